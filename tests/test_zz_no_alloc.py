"""GPU test of topk_attn_noalloc (the entry point whose workspace is the library's
fixed device scratch): through the C ABI, its output equals topk_attn's bit for bit
on two calls in a row, the second smaller than the first, and a call whose single
query chunk does not fit the scratch is refused before any launch."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2106_06899_amd as tk
from paper_2106_06899_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu


def _call(fn, q, k, v, out, w):
    rc = fn(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk,
            int(w.causal), w.scale, tk.TOPK_BF16 if w.dtype == wl.BF16 else tk.TOPK_F32,
            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    return rc


def _compare(w):
    L = tk.lib()
    x = wl.make_inputs(w)
    q, k, v = (parity.to_dev(x[n]) for n in ("Q", "K", "V"))
    print(f"no-alloc case: {w.note} B={w.B} H={w.H} Lq={w.Lq} Lk={w.Lk} k={w.k} chunk={w.chunk}", flush=True)
    ref = torch.empty_like(q)
    got = torch.full_like(q, float("nan"))
    assert tk.lib().topk_attn_workspace_bytes(w.B, w.H, w.Lq, w.Lk, w.d, w.k, w.chunk, int(w.causal),
                                              tk.TOPK_BF16 if w.dtype == wl.BF16 else tk.TOPK_F32) > 0
    tk._raise(_call(L.topk_attn, q, k, v, ref, w))
    tk._raise(_call(L.topk_attn_noalloc, q, k, v, got, w))
    torch.cuda.synchronize()
    a = got.view(torch.int16 if got.dtype == torch.bfloat16 else torch.int32).cpu().numpy()
    b = ref.view(torch.int16 if ref.dtype == torch.bfloat16 else torch.int32).cpu().numpy()
    assert np.array_equal(a, b), f"no-alloc output differs from topk_attn in {int((a != b).sum())} elements"
    # and the existing entry point's output is itself right: sampled rows against the oracle
    rows = parity.sample_attn_rows(w, 48, seed=3)
    idx = parity.run_attn(w, x)[1]
    parity.check_attn(w, x, ref, idx, rows=rows)


def test_noalloc_matches_topk_attn_on_two_calls_second_smaller():
    assert tk.lib().topk_noalloc_scratch_bytes() == 128 << 20
    big = wl.WORKLOADS["c3"].scaled(H=3, Lq=8192, Lk=8192, chunk=512)       # fused path, several passes
    small = wl.WORKLOADS["c2"].scaled(B=1, H=2, Lq=300, Lk=300, chunk=64)   # every key a candidate
    _compare(big)
    _compare(small)


def test_noalloc_chunk_tile_path_and_refusal():
    _compare(wl.WORKLOADS["c4"].scaled(B=1, H=2, Lq=1500, Lk=1500, chunk=256))   # causal, chunk-tile rows
    L = tk.lib()
    # one chunk of a 2^20-key head needs far more than the scratch: refused, nothing launched
    x = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    rc = L.topk_attn_noalloc(x.data_ptr(), x.data_ptr(), x.data_ptr(), x.data_ptr(), 1, 1, 4096, 1 << 20, 64, 64,
                             4096, 0, 0.125, tk.TOPK_BF16, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == -5, rc
    assert "fixed device scratch" in L.topk_last_error().decode()
