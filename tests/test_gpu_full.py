"""GPU parity at the five workloads' full sizes, in the launch configuration the
benchmark times (same call, same chunk). The oracle checks a sample of rows one by
one: the first and last rows of every head, chunk boundaries, causal rows < k, and
random rows."""
import numpy as np
import pytest
import torch

import paper_2106_06899_amd as tk
from paper_2106_06899_amd import workloads as wl
from oracle import topk_backward as bo
from tests import parity

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4"])
def test_attn_full_size(name):
    w = wl.WORKLOADS[name]
    _say(name, w.note)
    x = wl.make_inputs(w)
    out, idx, sc = parity.run_attn(w, x)
    rows = parity.sample_attn_rows(w, 160, seed=w.seed)
    rep = {}
    parity.check_attn(w, x, out, idx, rows=rows, report=rep)
    _say(name, "sampled rows ok", rep)
    # one whole head (every row of b = 0, h = H - 1) against the oracle as well
    head = np.stack([np.zeros(w.Lq, np.int64), np.full(w.Lq, w.H - 1), np.arange(w.Lq)], -1)
    rep_head = {}
    parity.check_attn(w, x, out, idx, rows=head, report=rep_head)
    _say(name, f"whole head {w.H - 1} ok", rep_head)
    # every row, not only the sampled ones, must carry exactly k_eff distinct valid indices
    g = idx.cpu().numpy()
    k_eff = np.minimum(w.k, np.arange(w.Lq) + 1) if w.causal else np.full(w.Lq, w.k)
    assert np.array_equal((g >= 0).sum(-1), np.broadcast_to(k_eff, g.shape[:-1]))
    srt = np.sort(np.where(g >= 0, g, -1 - np.arange(w.k)), axis=-1)
    assert not np.any(srt[..., 1:] == srt[..., :-1]), "duplicate index in a row"
    if w.causal:
        assert np.all(g <= np.arange(w.Lq)[:, None]), "a causal row selected a future key"
    assert torch.isfinite(out.float()).all()
    if w.planted:
        # generator sanity (not a parity criterion): a planted key scores about
        # |k|^2 = d above the noise, so most planted keys make the top-k
        pl = x["planted_idx"]
        kept = np.mean([np.isin(pl[0, h, i], g[0, h, i]).mean() for h in range(w.H) for i in range(0, w.Lq, 97)])
        _say(name, "fraction of planted keys kept", kept)
        assert kept > 0.8


def test_attn_causal_layer_shape_full_size():
    """The causal attention of the layer benchmark at its longest length: 12 heads of
    64, L 65536, k 128, chunk 1024 (rows below 12288 on the chunk-tile path, the rest
    fused), sampled rows of both parts against the oracle."""
    w = wl.WORKLOADS["c4"].scaled(B=1, H=12, Lq=65536, Lk=65536, d=64, k=128, chunk=1024,
                                  scale=float(np.float32(0.125)))
    assert tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, True, tk.TOPK_BF16) == 3
    _say("causal 12x65536", w)
    x = wl.make_inputs(w)
    out, idx, sc = parity.run_attn(w, x)
    rows = parity.sample_attn_rows(w, 120, seed=7)
    rep = {"fallback_rows": tk.last_fallback_rows()}
    parity.check_attn(w, x, out, idx, rows=rows, report=rep)
    _say("causal 12x65536 sampled rows ok", rep)
    g = idx.cpu().numpy()
    k_eff = np.minimum(w.k, np.arange(w.Lq) + 1)
    assert np.array_equal((g >= 0).sum(-1), np.broadcast_to(k_eff, g.shape[:-1]))
    assert np.all(g <= np.arange(w.Lq)[:, None]), "a causal row selected a future key"


def test_ffn_full_size():
    w = wl.WORKLOADS["c5"]
    _say("c5", w.note)
    x = wl.make_inputs(w)
    out, idx, sc = parity.run_ffn(w, x)
    rng = np.random.Generator(np.random.PCG64(w.seed))
    rows = np.unique(np.concatenate([[0, 1, w.chunk - 1, w.chunk, w.N - 1], rng.integers(0, w.N, 1100)]))
    assert rows.size >= 1024
    rep = {}
    parity.check_ffn(w, x, out, idx, rows=rows, report=rep)
    _say("c5", "sampled rows ok", rep)
    g = idx.cpu().numpy()
    assert np.all((g >= 0).sum(-1) == w.k)
    assert torch.isfinite(out.float()).all()


# ---------------------------------------------------------------- the paper's feed-forward shape
def _paper_ff_inputs(d_ff):
    """Inputs of the feed-forward benchmark (2^18 tokens = batch 512 x length 512,
    d_model 768) by the c5 recipe: X ~ N(0, 1), W1, W2 ~ N(0, 0.02^2), bf16."""
    w = wl.WORKLOADS["c5"].scaled(N=1 << 18, d_model=768, d_ff=d_ff, k=512, chunk=1 << 14)
    return w, wl.make_inputs(w)


@pytest.mark.parametrize("d_ff", [2048, 16384, 65536])
def test_ffn_paper_shape(d_ff):
    """The feed-forward benchmark of Section 3 (2^18 queries, d_model 768, k 512, token
    chunk 2^14) at three d_ff of its sweep: sampled rows against the oracle, every row
    with k distinct valid indices."""
    w, x = _paper_ff_inputs(d_ff)
    _say("paper FF", f"N {w.N} d_model {w.d_model} d_ff {d_ff} k {w.k} chunk {w.chunk}")
    out, idx, sc = parity.run_ffn(w, x)
    rng = np.random.Generator(np.random.PCG64(d_ff))
    C = w.chunk
    rows = np.unique(np.concatenate([[0, C - 1, C, w.N - C, w.N - 1], rng.integers(0, w.N, 250)]))
    rep = {"fallback_rows": tk.last_fallback_rows()}
    parity.check_ffn(w, x, out, idx, rows=rows, report=rep)
    _say("paper FF", d_ff, "sampled rows ok", rep)
    g = idx.cpu().numpy()
    assert np.all((g >= 0).sum(-1) == w.k) and np.all(g < d_ff)
    assert torch.isfinite(out.float()).all()


# ---------------------------------------------------------------- backward, full size
def _sample_keys(idx_head, Lk, rng, n):
    """Keys 0 and Lk - 1, the three most selected keys, and n random keys."""
    counts = np.bincount(idx_head[idx_head >= 0].ravel(), minlength=Lk)
    hot = np.argsort(-counts, kind="stable")[:3]
    return np.unique(np.concatenate([[0, Lk - 1], hot, rng.integers(0, Lk, n)]))


def _check_sample(name, got, ref, mag, dtype):
    """Each sampled row / key against its own reference (the rule of test_gpu_backward)."""
    return parity.check_grad_rows(name, got, ref, mag, dtype)


def _unselected_are_zero(idx, dk, dv, Lk):
    """Every key that no row selected gets exactly zero gradients (any size)."""
    counts = np.bincount(idx[idx >= 0].ravel(), minlength=Lk)
    cold = np.flatnonzero(counts == 0)
    assert not np.any(dk[cold]) and not np.any(dv[cold])
    return len(cold)


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_attn_backward_full_size(name):
    """The backward call bench.py --backward times, at the full workload: d_Q at
    sampled rows and d_K, d_V at sampled keys of three heads against the oracle's
    sampled backward (computed from the same cached index sets)."""
    w = wl.WORKLOADS[name]
    _say(name, "backward", w.note)
    x = wl.make_inputs(w)
    q, k, v = (parity.to_dev(x[n]) for n in ("Q", "K", "V"))
    _, idx, dots = tk.attn(q, k, v, w.k, w.chunk, w.causal, w.scale, debug=True)
    g = parity.grad_out((w.B, w.H, w.Lq, w.d), w.dtype, 5)
    dq, dk, dv = tk.attn_backward(q, k, v, idx, dots, parity.to_dev(g), w.scale)
    torch.cuda.synchronize()
    ix = idx.cpu().numpy()
    dq, dk, dv = (t.float().cpu().numpy() for t in (dq, dk, dv))
    assert np.isfinite(dq).all() and np.isfinite(dk).all() and np.isfinite(dv).all()
    rng = np.random.Generator(np.random.PCG64(w.seed + 1))
    heads = sorted({(0, 0), (w.B - 1, w.H - 1), (int(rng.integers(w.B)), int(rng.integers(w.H)))})
    C = w.chunk or w.Lq
    for b, h in heads:
        rows = np.unique(np.concatenate([[0, 1, C - 1, C, min(w.k - 1, w.Lq - 1), w.Lq - 1],
                                         rng.integers(0, w.Lq, 40)]))
        keys = _sample_keys(ix[b, h], w.Lk, rng, 24)
        (rq, rk, rv), (aq, ak, av) = bo.sampled_backward(x["Q"].values[b, h], x["K"].values[b, h],
                                                         x["V"].values[b, h], ix[b, h], g.values[b, h], rows, keys,
                                                         "softmax", w.scale, magnitudes=True)
        errs = (_check_sample("d_Q", dq[b, h][rows], rq, aq, w.dtype),
                _check_sample("d_K", dk[b, h][keys], rk, ak, w.dtype),
                _check_sample("d_V", dv[b, h][keys], rv, av, w.dtype))
        cold = _unselected_are_zero(ix[b, h], dk[b, h], dv[b, h], w.Lk)
        _say(name, f"head ({b},{h}) rows {len(rows)} keys {len(keys)} unselected keys {cold} errors", errs)


def test_ffn_backward_full_size():
    """The feed-forward backward at the full c5 workload: d_X at sampled rows and
    d_W1, d_W2 at sampled keys (hidden units) against the oracle's sampled backward."""
    w = wl.WORKLOADS["c5"]
    _say("c5", "backward", w.note)
    x = wl.make_inputs(w)
    a, b1, b2 = (parity.to_dev(x[n]) for n in ("X", "W1", "W2"))
    _, idx, dots = tk.ffn(a, b1, b2, w.k, w.chunk, debug=True)
    g = parity.grad_out((w.N, w.d_model), w.dtype, 5)
    dx, dw1, dw2 = tk.ffn_backward(a, b1, b2, idx, dots, parity.to_dev(g))
    torch.cuda.synchronize()
    ix = idx.cpu().numpy()
    dx, dw1, dw2 = (t.float().cpu().numpy() for t in (dx, dw1, dw2))
    assert np.isfinite(dx).all() and np.isfinite(dw1).all() and np.isfinite(dw2).all()
    rng = np.random.Generator(np.random.PCG64(w.seed + 1))
    rows = np.unique(np.concatenate([[0, 1, w.chunk - 1, w.chunk, w.N - 1], rng.integers(0, w.N, 40)]))
    keys = _sample_keys(ix, w.d_ff, rng, 16)
    (rx, r1, r2), (ax, a1, a2) = bo.sampled_backward(x["X"].values, x["W1"].values, x["W2"].values, ix, g.values,
                                                     rows, keys, "relu", magnitudes=True)
    errs = (_check_sample("d_X", dx[rows], rx, ax, w.dtype), _check_sample("d_W1", dw1[keys], r1, a1, w.dtype),
            _check_sample("d_W2", dw2[keys], r2, a2, w.dtype))
    cold = _unselected_are_zero(ix, dw1, dw2, w.d_ff)
    _say("c5", f"rows {len(rows)} keys {len(keys)} unselected keys {cold} errors", errs)
