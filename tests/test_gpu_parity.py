"""GPU parity of the HIP path against the fp64 oracle on small seeded cases.

Each case follows one workload's recipe at a size the oracle finishes in seconds
while still spanning several key tiles, several query blocks and ragged tails.
Every call goes through the C ABI via the binding (``paper_2106_06899_amd``).
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import paper_2106_06899_amd as tk
from paper_2106_06899_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tk.lib()
    yield


def test_mfma_lane_layout():
    """The fused scan assumes lane l, register v of the 32x32x16 bf16 MFMA holds output
    row 8*(v/4) + 4*(l/32) + v%4 and column l%32."""
    _say("mfma layout probe")
    rows, cols = tk.mfma_layout()
    torch.cuda.synchronize()
    rows, cols = rows.cpu().numpy(), cols.cpu().numpy()
    lanes = np.arange(64)[:, None]
    v = np.arange(16)[None, :]
    assert np.array_equal(rows, 8 * (v // 4) + 4 * (lanes // 32) + (v % 4))
    assert np.array_equal(cols, np.broadcast_to(lanes % 32, (64, 16)))


ATTN_CASES = {
    # name: (base workload, overrides)
    "c1_fp32_tile": ("c1", dict(Lq=300, Lk=777, chunk=100)),
    "c2_bf16_fused_all": ("c2", dict(B=2, H=3, Lq=200, Lk=512, chunk=128)),
    "c2_bf16_fused_all_ragged": ("c2", dict(B=1, H=2, Lq=130, Lk=333, chunk=64)),
    # every key a candidate and more than 512 of them: the select's long-list path
    "c2_bf16_fused_all_long_lists": ("c2", dict(B=1, H=2, Lq=150, Lk=1000, chunk=64)),
    "c3_bf16_fused_sample": ("c3", dict(H=2, Lq=300, Lk=9000, chunk=256)),
    "c3_bf16_fused_sample_k32": ("c3", dict(H=1, Lq=257, Lk=4600, k=32, chunk=1024)),
    "c4_bf16_causal_tile": ("c4", dict(B=1, H=2, Lq=600, Lk=600, chunk=256)),
    "c4_d128_fused_sample": ("c4", dict(B=1, H=1, Lq=200, Lk=17000, causal=False, chunk=128)),
    "c4_d128_fused_all": ("c4", dict(B=1, H=2, Lq=150, Lk=700, causal=False, chunk=64)),
    "bf16_tile_d96": ("c2", dict(B=1, H=2, Lq=70, Lk=300, d=96, k=40, chunk=32)),
    "fp32_causal_tile": ("c1", dict(Lq=200, Lk=260, causal=True, k=20, chunk=64)),
    # chunk-tile short-row select past 1024 keys: exact sampled rank (R > 96) and
    # the per-lane top-two threshold (R <= 96)
    "tile_sampled_exact_rank": ("c2", dict(B=1, H=1, Lq=90, Lk=1500, d=96, k=128, chunk=64)),
    "tile_sampled_top_two": ("c2", dict(B=1, H=1, Lq=90, Lk=6000, d=96, k=64, chunk=64, dtype=wl.F32)),
    # chunk-tile long-row select (workgroup per row, sampled blocks) and a causal
    # case whose rows cross 1024 keys
    "tile_long_rows": ("c2", dict(B=1, H=1, Lq=40, Lk=9500, d=96, k=300, chunk=40)),
    "c4_causal_long": ("c4", dict(B=1, H=1, Lq=2100, Lk=2100, chunk=1024)),
    # causal masks with Lk >= 256 k: rows below 1024 R on the chunk-tile path, the
    # rest on the fused path (path 3)
    "c3_causal_fused_k16": ("c3", dict(H=2, Lq=4500, Lk=4500, k=16, chunk=512, causal=True)),
    "c4_d128_causal_fused": ("c4", dict(B=1, H=1, Lq=8300, Lk=8300, k=32, chunk=1024)),
    "causal_fused_lq_below_lk": ("c3", dict(H=1, Lq=4000, Lk=8000, k=16, chunk=256, causal=True)),
    "causal_fused_lq_above_lk": ("c3", dict(H=1, Lq=6000, Lk=4200, k=16, chunk=1000, causal=True)),
    # filtered chunk-tile path (path 4): sampled thresholds, the tile GEMM keeps only
    # scores at or above them
    "filter_causal_d128_k128": ("c4", dict(B=1, H=2, Lq=3000, Lk=3000, chunk=512)),
    "filter_d96_k200": ("c2", dict(B=1, H=1, Lq=300, Lk=12000, d=96, k=200, chunk=128)),
    "filter_d32_k7_ragged": ("c2", dict(B=2, H=1, Lq=333, Lk=2601, d=32, k=7, chunk=100)),
    # the filtered path's scan at d = 128 with k > 256 (two 1024-word lists per row, the
    # larger select) under the causal mask: early rows keep every key (k_eff < k)
    "filter_causal_d128_k300": ("c4", dict(B=1, H=1, Lq=5000, Lk=5000, k=300, chunk=1000)),
    # a handful of rows of 563 samples each: the threshold kernel's loads (1024 samples
    # from each row's start) run past the last row into the padding after the samples
    "filter_d96_few_rows": ("c2", dict(B=1, H=1, Lq=3, Lk=9000, d=96, k=200, chunk=3)),
    "filter_d128_few_rows": ("c4", dict(B=1, H=1, Lq=2, Lk=9000, k=200, causal=False, chunk=2)),
}


@pytest.mark.parametrize("name", sorted(ATTN_CASES))
def test_attn_parity(name):
    base, kw = ATTN_CASES[name]
    w = wl.WORKLOADS[base].scaled(**kw)
    _say(name, w)
    x = wl.make_inputs(w)
    out, idx, sc = parity.run_attn(w, x)
    rep = {"fallback_rows": tk.last_fallback_rows()}
    parity.check_attn(w, x, out, idx, report=rep)
    _say(name, "ok", rep, "path", tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal,
                                                tk.TOPK_BF16 if w.dtype == wl.BF16 else tk.TOPK_F32))
    # debug scores are the raw fp32 scores of the selected keys, sorted descending
    s = sc.cpu().numpy()
    fin = np.isfinite(s)
    assert np.all(np.diff(np.where(fin, s, -np.inf), axis=-1)[fin[..., 1:]] <= 0)


FFN_CASES = {
    "c5_tile": dict(N=300, d_model=256, d_ff=4096, k=512, chunk=128),
    "c5_tile_small_k": dict(N=100, d_model=64, d_ff=2000, k=7, chunk=33),
    "ffn_fused_all": dict(N=260, d_model=64, d_ff=1000, k=64, chunk=100),
    # filtered chunk-tile path with k > 256 (2048-entry lists) and a workgroup threshold
    # over more than 1024 samples
    "ffn_filter_k300_wg_threshold": dict(N=200, d_model=128, d_ff=20000, k=300, chunk=64),
    "ffn_fused_sample": dict(N=130, d_model=128, d_ff=20000, k=100, chunk=0),
    # value matrices over 8 MiB: the gather runs in column slices of whole 128-byte
    # lines, each re-ordering the survivors by key index (eight slices with register
    # sorts of 128 and 512 entries; 4-byte elements; four 384-byte slices at d 768;
    # four 128-byte slices at d 256)
    "ffn_sliced_gather_k100": dict(N=150, d_model=512, d_ff=9000, k=100, chunk=64),
    "ffn_sliced_gather_k512": dict(N=70, d_model=1024, d_ff=5000, k=512, chunk=32),
    "ffn_sliced_gather_f32": dict(N=90, d_model=256, d_ff=9000, k=40, chunk=50, dtype=wl.F32),
    "ffn_sliced_gather_d768": dict(N=60, d_model=768, d_ff=6000, k=64, chunk=32),
    "ffn_sliced_gather_d256": dict(N=80, d_model=256, d_ff=20000, k=70, chunk=40),
}


@pytest.mark.parametrize("name", sorted(FFN_CASES))
def test_ffn_parity(name):
    w = wl.WORKLOADS["c5"].scaled(**FFN_CASES[name])
    _say(name, w)
    x = wl.make_inputs(w)
    out, idx, sc = parity.run_ffn(w, x)
    rep = {}
    parity.check_ffn(w, x, out, idx, report=rep)
    _say(name, "ok", rep, "path", tk.ffn_path(w.N, w.d_model, w.d_ff, w.k, w.chunk))


@pytest.mark.parametrize("name", ["ffn_sliced_gather_k100", "ffn_sliced_gather_f32", "ffn_sliced_gather_d768"])
def test_sliced_gather_plain_equals_debug(name):
    """The column-sliced gather gives the same bits whether or not the selection is written."""
    w = wl.WORKLOADS["c5"].scaled(**FFN_CASES[name])
    _say(name, w)
    x = wl.make_inputs(w)
    out_dbg, _, _ = parity.run_ffn(w, x)
    out = parity.run_ffn(w, x, debug=False)
    assert torch.equal(out, out_dbg)


@pytest.mark.parametrize("base,kw", [
    ("c2", dict(B=1, H=2, Lq=100, Lk=512)),                 # fused, all candidates
    ("c3", dict(H=1, Lq=150, Lk=9000)),                     # fused, sampled threshold
    ("c4", dict(B=1, H=1, Lq=100, Lk=300)),                 # chunk-tile, causal
])
def test_k1_returns_argmax_value_row_exactly(base, kw):
    """k = 1: the single survivor has softmax weight exactly 1, so the bf16 output is
    the value row of the best key, bit for bit."""
    w = wl.WORKLOADS[base].scaled(k=1, **kw)
    _say("k1", w)
    x = wl.make_inputs(w)
    out, idx, _ = parity.run_attn(w, x)
    parity.check_attn(w, x, out, idx)
    o = out.view(torch.int16).cpu().numpy()
    V = x["V"].bits.view(np.int16)
    g = idx.cpu().numpy()[..., 0]
    for b in range(w.B):
        for h in range(w.H):
            assert np.array_equal(o[b, h], V[b, h][g[b, h]])


@pytest.mark.parametrize("base,kw", [
    ("c1", dict(Lq=64, Lk=200, chunk=32)),
    ("c2", dict(B=1, H=1, Lq=64, Lk=256, chunk=64)),
    ("c4", dict(B=1, H=1, Lq=96, Lk=96, d=128, chunk=32)),
])
def test_k_equals_Lk_is_vanilla_attention(base, kw):
    """k = Lk: the GPU result equals dense softmax attention (Eq. 1 / Eq. 2) within tolerance."""
    w = wl.WORKLOADS[base].scaled(**kw)
    w = w.scaled(k=w.Lk)
    _say("k=Lk", w)
    x = wl.make_inputs(w)
    out, idx, _ = parity.run_attn(w, x)
    Q, K, V = (x[n].values.astype(np.float64) for n in ("Q", "K", "V"))
    S = np.einsum("bhid,bhjd->bhij", Q, K) * np.float64(np.float32(w.scale))
    if w.causal:
        S = np.where(np.tril(np.ones((w.Lq, w.Lk), bool))[None, None], S, -np.inf)
    P = np.exp(S - S.max(-1, keepdims=True))
    P /= P.sum(-1, keepdims=True)
    ref = P @ V
    got = out.float().cpu().numpy()
    err = np.abs(got - ref).max(-1) / np.abs(ref).max(-1)
    assert err.max() <= parity.RTOL[w.dtype], err.max()


@pytest.mark.parametrize("base,kw", [
    ("c2", dict(B=1, H=2, Lq=200, Lk=512)),
    ("c3", dict(H=1, Lq=300, Lk=9000)),
    ("c4", dict(B=1, H=1, Lq=300, Lk=300)),
    ("c1", dict(Lq=200, Lk=300)),
    ("c3", dict(H=1, Lq=4200, Lk=4200, k=16, causal=True)),
    ("c4", dict(B=1, H=1, Lq=2500, Lk=2500)),
])
def test_chunking_does_not_change_the_result(base, kw):
    """Query chunking is result-neutral: bit-identical outputs and indices for every C."""
    w = wl.WORKLOADS[base].scaled(**kw)
    x = wl.make_inputs(w)
    ref = None
    for C in (1, 7, 64, 256, w.Lq):
        _say("chunk", C, w)
        out, idx, sc = parity.run_attn(w, x, chunk=C)
        cur = (out.view(torch.int16 if w.dtype == wl.BF16 else torch.int32).cpu(), idx.cpu(), sc.cpu())
        if ref is None:
            ref = cur
            parity.check_attn(w, x, out, idx)
        else:
            for a, b in zip(ref, cur):
                assert torch.equal(a, b), f"chunk {C} differs"


def test_repeated_calls_are_bit_identical():
    w = wl.WORKLOADS["c3"].scaled(H=2, Lq=500, Lk=9000)
    _say("determinism", w)
    x = wl.make_inputs(w)
    a = parity.run_attn(w, x)
    b = parity.run_attn(w, x)
    for p, q in zip(a, b):
        assert torch.equal(p.cpu(), q.cpu())


@pytest.mark.parametrize("kw", [
    dict(B=1, H=1, Lq=1, Lk=1, k=1),
    dict(B=1, H=1, Lq=1, Lk=5, k=5),
    dict(B=1, H=3, Lq=5, Lk=63, k=10),
    dict(B=1, H=1, Lq=129, Lk=65, k=64),
    dict(B=2, H=1, Lq=33, Lk=1024, k=128),
])
def test_edge_shapes(kw):
    for base in ("c2", "c1"):
        w = wl.WORKLOADS[base].scaled(chunk=0, **kw)
        _say("edge", w)
        x = wl.make_inputs(w)
        out, idx, _ = parity.run_attn(w, x)
        parity.check_attn(w, x, out, idx)


def test_causal_rows_below_k_keep_every_valid_key():
    w = wl.WORKLOADS["c4"].scaled(B=1, H=1, Lq=300, Lk=300, k=128, chunk=100)
    _say("causal rows < k", w)
    x = wl.make_inputs(w)
    out, idx, _ = parity.run_attn(w, x)
    g = idx.cpu().numpy()[0, 0]
    for i in range(w.k):
        assert sorted(g[i][g[i] >= 0].tolist()) == list(range(i + 1))
        assert np.all(g[i][i + 1:] == -1)
    parity.check_attn(w, x, out, idx)


def _pad(a, n=8):
    a = np.asarray(a, dtype=np.float32)
    out = np.zeros(a.shape[:-1] + (max(n, a.shape[-1]),), np.float32)
    out[..., : a.shape[-1]] = a
    return out


@pytest.mark.parametrize("ex", json.load(open(os.path.join(HERE, "golden", "worked_examples.json")))["examples"],
                         ids=lambda e: e["name"])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_worked_examples_on_gpu(ex, dtype):
    """The hand-derived examples of Eq. 2-4 (features zero-padded to 8, exact in bf16)."""
    _say("worked example", ex["name"], dtype)
    Q, K, V = (torch.from_numpy(_pad(ex[n])).to("cuda", dtype) for n in ("Q", "K", "V"))
    if ex["activation"] == "relu":
        out, idx, _ = tk.ffn(Q, K, V, ex["k"], debug=True)
    else:
        out, idx, _ = tk.attn(Q[None, None], K[None, None], V[None, None], ex["k"], 0, ex.get("causal", False),
                              ex.get("scale", 1.0), debug=True)
        out, idx = out[0, 0], idx[0, 0]
    torch.cuda.synchronize()
    for i, want in enumerate(ex["selected"]):
        got = idx[i].cpu().numpy()
        assert got[got >= 0].tolist() == want
    want = np.array([[float(eval(v, {"__builtins__": {}}, {"exp": math.exp})) for v in row] for row in ex["out"]])
    got = out.float().cpu().numpy()[:, : want.shape[1]]
    tol = 1e-6 if dtype == torch.float32 else 1e-2
    np.testing.assert_allclose(got, want, rtol=tol, atol=tol)


def _planted(w: wl.Workload, alpha: np.ndarray, seed: int) -> dict:
    """Q = e0 + noise, K[j] = alpha[j] e0 + noise, V ~ N(0,1): score(i, j) is about
    alpha[j], so the test decides which keys win (stored in the workload's dtype)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    q = 0.3 * rng.standard_normal((w.B, w.H, w.Lq, w.d)).astype(np.float32)
    q[..., 0] = 1.0
    k = 0.3 * rng.standard_normal((w.B, w.H, w.Lk, w.d)).astype(np.float32)
    k[..., 0] = alpha.astype(np.float32)
    v = rng.standard_normal((w.B, w.H, w.Lk, w.d)).astype(np.float32)

    def t(a):
        if w.dtype == wl.F32:
            return wl.Tensor(a, None, wl.F32)
        bits = wl.f32_to_bf16_bits(a)
        return wl.Tensor(wl.bf16_bits_to_f32(bits), bits, wl.BF16)

    return {"Q": t(q), "K": t(k), "V": t(v)}


def test_fused_fallback_for_every_row():
    """Every key of the sampled tiles (1 in 8 at d = 64, k = 64) scores high, the rest
    lower: each row's threshold (the 20th largest of 48 sampled block maxima) keeps
    about 25 < k keys, so every row is recomputed by the fallback kernels, including
    more rows than the first fallback kernel takes (1024)."""
    w = wl.WORKLOADS["c3"].scaled(H=1, Lq=1200, Lk=6000, chunk=1024)
    assert tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal, tk.TOPK_BF16) == 1
    j = np.arange(w.Lk)
    alpha = np.where((j // 64) % 8 == 0, 10.0, 3.0)
    _say("fused fallback", w)
    x = _planted(w, alpha, 7)
    out, idx, _ = parity.run_attn(w, x)
    assert tk.last_fallback_rows() == w.Lq
    parity.check_attn(w, x, out, idx)


def test_tile_short_row_fallback():
    """Only 100 of the 1024 sampled keys score high (the rest of the sample lowest),
    so the per-lane top-two threshold keeps about 76 < k keys: every row goes to the
    short-row select's fallback list."""
    w = wl.WORKLOADS["c2"].scaled(B=1, H=1, Lq=120, Lk=2000, d=96, k=128, chunk=64)
    assert tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal, tk.TOPK_BF16) == 2
    alpha = np.full(w.Lk, 3.0)
    pos = (np.arange(1024) * w.Lk) // 1024
    alpha[pos] = -10.0
    alpha[pos[:100]] = 10.0
    _say("tile short-row fallback", w)
    x = _planted(w, alpha, 8)
    out, idx, _ = parity.run_attn(w, x)
    assert tk.last_fallback_rows() == w.Lq
    parity.check_attn(w, x, out, idx)


def test_filter_fallback_for_every_row():
    """Filtered chunk-tile path: every 16th key (the sampled ones) scores high, the rest
    lower, so each row's threshold keeps only about R < k keys: every row is
    recomputed by the fallback kernels, more rows than the first fallback kernel
    takes (1024)."""
    w = wl.WORKLOADS["c4"].scaled(B=1, H=1, Lq=1200, Lk=4000, causal=False, chunk=512)
    assert tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal, tk.TOPK_BF16) == 4
    alpha = np.where(np.arange(w.Lk) % 16 == 0, 10.0, 3.0)
    _say("filter fallback", w)
    x = _planted(w, alpha, 10)
    out, idx, _ = parity.run_attn(w, x)
    assert tk.last_fallback_rows() == w.Lq
    parity.check_attn(w, x, out, idx)


@pytest.mark.parametrize("d", [128, 96])
def test_filter_overflow_for_every_row(d):
    """Filtered path, the other way round: every 16th key (the sampled ones) scores low
    and the rest high, so each row's threshold lies below almost every key and its
    candidate lists overflow (more than 512 per half-wave list at d = 128, where the
    scan kernel appends them; more than 1024 per row list at d = 96, where the tile
    GEMM does): every row is recomputed by the fallback kernels."""
    w = wl.WORKLOADS["c4"].scaled(B=1, H=1, Lq=1100, Lk=4000, d=d, causal=False, chunk=512)
    assert tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal, tk.TOPK_BF16) == 4
    alpha = np.where(np.arange(w.Lk) % 16 == 0, 3.0, 10.0)
    _say("filter overflow", w)
    x = _planted(w, alpha, 11)
    out, idx, _ = parity.run_attn(w, x)
    assert tk.last_fallback_rows() == w.Lq
    parity.check_attn(w, x, out, idx)


def test_tile_long_row_fallback():
    """Rows over 8192 keys: 30 of the 1024 sampled keys score high, the rest of the
    sample lowest; the threshold (24th sampled key) keeps 24 < k keys, and the row is
    selected by the multi-pass radix select from the tile row."""
    w = wl.WORKLOADS["c2"].scaled(B=1, H=1, Lq=60, Lk=17000, d=96, k=32, chunk=64, dtype=wl.F32)
    assert tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal, tk.TOPK_F32) == 2
    alpha = np.full(w.Lk, 3.0)
    s = np.arange(1024)
    pos = 32 * ((s >> 5) * w.Lk // 1024) + (s & 31)
    alpha[pos] = -10.0
    alpha[pos[:30]] = 10.0
    _say("tile long-row fallback", w)
    x = _planted(w, alpha, 9)
    out, idx, _ = parity.run_attn(w, x)
    assert tk.last_fallback_rows() == w.Lq
    parity.check_attn(w, x, out, idx)


@pytest.mark.parametrize("base,kw,path", [
    ("c3", dict(H=2, Lq=700, Lk=9000, chunk=128), 1),                                  # fused
    ("c2", dict(B=1, H=2, Lq=300, Lk=1500, d=96, k=40, chunk=64), 2),                # chunk-tile
    ("c4", dict(B=1, H=2, Lq=2500, Lk=2500, chunk=256), 4),                          # filtered chunk-tile
    ("c3", dict(H=2, Lq=4200, Lk=4200, k=16, chunk=512, causal=True), 3),            # split by rows
])
def test_one_chunk_per_pass_is_bit_identical(base, kw, path):
    """A memory budget below one chunk runs every chunk in a pass of its own (the
    paper's sequential query chunking); the result is the default budget's, bit for bit."""
    w = wl.WORKLOADS[base].scaled(**kw)
    dt = tk.TOPK_BF16 if w.dtype == wl.BF16 else tk.TOPK_F32
    assert tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal, dt) == path
    _say("one chunk per pass", path, w)
    x = wl.make_inputs(w)
    ref = parity.run_attn(w, x)
    tk.set_memory_budget(1)
    try:
        got = parity.run_attn(w, x)
    finally:
        tk.set_memory_budget(0)
    def bits(t):  # compare floating-point outputs bit for bit (NaN-safe)
        t = t.cpu()
        return t.view(torch.int32) if t.dtype == torch.float32 else t.view(torch.int16) \
            if t.dtype == torch.bfloat16 else t

    for a, b in zip(ref, got):
        assert torch.equal(bits(a), bits(b))
    parity.check_attn(w, x, got[0], got[1])


# Ties: every score of a row equal (Q = 0), so the total order (score desc, index asc)
# keeps the k lowest valid key indices, in increasing order; and scores confined to a
# narrow band (Q scaled down), where the keys of the candidates share their top bits
# and differ only low in the score or in the index.
TIE_CASES = [
    ("c3", dict(H=2, Lq=300, Lk=6000, chunk=256), 1),        # fused path, sampled threshold
    ("c2", dict(B=1, H=2, Lq=200, Lk=512, chunk=128), 1),     # fused path, every key a candidate
    ("c4", dict(B=1, H=2, Lq=300, Lk=4096, chunk=128), 4),    # filtered chunk-tile path (causal)
    ("c5", dict(N=200, d_model=256, d_ff=3000, k=256, chunk=64), 4),  # filtered chunk-tile (FFN)
    ("c1", dict(Lq=200, Lk=700, chunk=64), 2),                # chunk-tile path, fp32
]


@pytest.mark.parametrize("base,kw,path", TIE_CASES)
@pytest.mark.parametrize("band", [0.0, 1e-3])
def test_ties_keep_the_lowest_indices(base, kw, path, band):
    w = wl.WORKLOADS[base].scaled(**kw)
    _say("ties", band, w)
    x = wl.make_inputs(w)
    qn = "Q" if w.kind == "attn" else "X"
    x[qn] = wl._store((x[qn].values * np.float32(band)).astype(np.float32), w.dtype)
    if w.kind == "attn":
        assert tk.attn_path(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, w.causal,
                            tk.TOPK_BF16 if w.dtype == wl.BF16 else tk.TOPK_F32) == path
        out, idx, sc = parity.run_attn(w, x)
        rep = {}
        parity.check_attn(w, x, out, idx, report=rep)
    else:
        assert tk.ffn_path(w.N, w.d_model, w.d_ff, w.k, w.chunk) == path
        out, idx, sc = parity.run_ffn(w, x)
        rep = {}
        parity.check_ffn(w, x, out, idx, report=rep)
    _say("ties", band, "ok", rep)
    if band == 0.0:  # all scores 0: the lowest valid indices, ascending
        g = idx.cpu().numpy().reshape(-1, w.k)
        L = w.Lq if w.kind == "attn" else w.N
        rows = np.arange(g.shape[0]) % L
        nvalid = np.minimum(rows + 1, w.Lk) if (w.kind == "attn" and w.causal) else np.full(g.shape[0], w.Lk if w.kind == "attn" else w.d_ff)
        k_eff = np.minimum(w.k, nvalid)
        want = np.where(np.arange(w.k)[None, :] < k_eff[:, None], np.arange(w.k)[None, :], -1)
        assert np.array_equal(g, want), f"first bad row {int(np.argmax(np.any(g != want, axis=1)))}"
        assert np.all(sc.cpu().numpy().reshape(-1, w.k)[want >= 0] == 0.0)
