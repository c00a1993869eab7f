"""GPU parity of query chunking with the top-k disabled (the paper's comparison
baseline, Section 2.2 "Query chunking"): ``topk_attn_dense`` against the oracle at
k = Lk, where Eq. 4 keeps every valid key and reduces to Eq. 1 (with the Eq. 2 mask).
Outputs must agree per row to 2e-2 (bf16) in the row max norm. Small cases with
ragged tails and both feature sizes check every row; the paper's long-sequence
point, L = 65536 (d = 64), is checked on sampled rows."""
import numpy as np
import pytest
import torch

import paper_2106_06899_amd as tk
from oracle import topk_oracle as o
from paper_2106_06899_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu


def _dense(w, x, chunk=None):
    q, k, v = (parity.to_dev(x[n]) for n in ("Q", "K", "V"))
    out = tk.attn_dense(q, k, v, w.chunk if chunk is None else chunk, w.causal, w.scale)
    torch.cuda.synchronize()
    return out


def _check_rows(w, x, out, rows):
    Q, K, V = (x[n].values for n in ("Q", "K", "V"))
    ref = o.oracle_attn_rows(Q, K, V, w.Lk, w.causal, w.scale, rows)
    g = out.float().cpu().numpy().astype(np.float64)[rows[:, 0], rows[:, 1], rows[:, 2]]
    # softmax weights sum to one, so the ratio's floor is 1e-6 max|V|
    ratio = o.output_rel_errors(g, ref["out"], np.ones((len(rows), 1)), float(np.abs(V).max()))
    assert np.all(ratio <= parity.RTOL[w.dtype]), \
        f"output error {ratio.max():.3e} at row {rows[int(np.argmax(ratio))].tolist()}"
    return float(ratio.max())


def _all_rows(w):
    return np.stack(np.meshgrid(np.arange(w.B), np.arange(w.H), np.arange(w.Lq), indexing="ij"), -1).reshape(-1, 3)


CASES = {
    "d64": dict(B=1, H=2, Lq=300, Lk=700, d=64, chunk=128, causal=False),
    "d64_causal": dict(B=2, H=1, Lq=450, Lk=450, d=64, chunk=200, causal=True),
    "d128": dict(B=1, H=2, Lq=200, Lk=333, d=128, chunk=64, causal=False),
    "d128_causal": dict(B=1, H=1, Lq=260, Lk=260, d=128, chunk=1000, causal=True),
    "lq_above_lk_causal": dict(B=1, H=1, Lq=200, Lk=70, d=64, chunk=64, causal=True),
    "single_key": dict(B=1, H=1, Lq=5, Lk=1, d=64, chunk=2, causal=False),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_dense_matches_eq1(name):
    kw = dict(CASES[name])
    w = wl.WORKLOADS["c2"].scaled(k=kw["Lk"], scale=float(np.float32(1 / np.sqrt(kw["d"]))), **kw)
    x = wl.make_inputs(w)
    out = _dense(w, x)
    _check_rows(w, x, out, _all_rows(w))


def test_dense_chunk_size_does_not_change_the_result():
    w = wl.WORKLOADS["c2"].scaled(B=1, H=2, Lq=520, Lk=520, k=520, chunk=0, causal=True)
    x = wl.make_inputs(w)
    ref = _dense(w, x, 520).view(torch.int16)
    for C in (1, 7, 64, 128, 300):
        assert torch.equal(_dense(w, x, C).view(torch.int16), ref), f"chunk {C}"


def test_topk_attn_with_k_equal_lk_above_the_select_limit_is_dense():
    w = wl.WORKLOADS["c2"].scaled(B=1, H=1, Lq=256, Lk=3000, k=3000, chunk=128)
    x = wl.make_inputs(w)
    q, k, v = (parity.to_dev(x[n]) for n in ("Q", "K", "V"))
    a = tk.attn(q, k, v, 3000, 128, False, w.scale)
    b = tk.attn_dense(q, k, v, 128, False, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    _check_rows(w, x, a, parity.sample_attn_rows(w, 24, seed=4))


@pytest.mark.parametrize("causal", [False, True])
def test_dense_at_the_paper_length_65536(causal):
    """The single-layer benchmark's longest input (L = 65536, heads of 64): sampled
    rows, including the first and last rows and chunk boundaries, against Eq. 1."""
    w = wl.WORKLOADS["c2"].scaled(B=1, H=2, Lq=65536, Lk=65536, k=65536, chunk=1024, causal=causal)
    x = wl.make_inputs(w)
    out = _dense(w, x)
    err = _check_rows(w, x, out, parity.sample_attn_rows(w, 40, seed=5))
    print(f"L=65536 causal={causal}: max row error {err:.3e}")
