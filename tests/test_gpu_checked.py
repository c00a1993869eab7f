"""GPU test of the checked build (libtopk_check.so, compiled with TOPK_CHECK_INDICES):
on each forward path it returns the same output bits as libtopk.so, its finalize sees
no selected index outside the value matrix (topk_debug_bad_indices() == 0), and its
calls, which wait for their stream, report no asynchronous kernel error."""
import ctypes

import pytest
import torch

import paper_2106_06899_amd as tk
from paper_2106_06899_amd import build as b
from paper_2106_06899_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu

_CHECK = None


def _checked():
    global _CHECK
    if _CHECK is None:
        L = ctypes.CDLL(b.LIB_CHECK)
        i64, vp, i32, f32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_float
        L.topk_attn.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i64, i32, f32, i32, vp]
        L.topk_ffn.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, i64, i32, vp]
        L.topk_attn.restype = L.topk_ffn.restype = i32
        L.topk_debug_bad_indices.restype = i64
        L.topk_last_error.restype = ctypes.c_char_p
        _CHECK = L
    return _CHECK


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


CASES = {
    "fused_all_keys": ("c2", dict(B=1, H=2, Lq=300, Lk=512, chunk=128)),
    "fused_sampled": ("c3", dict(H=2, Lq=700, Lk=9000, chunk=256)),
    "chunk_tile_causal": ("c4", dict(B=1, H=2, Lq=400, Lk=400, chunk=128)),
    "filtered_causal": ("c4", dict(B=1, H=1, Lq=512, Lk=6000, causal=False, chunk=256)),
    "fp32": ("c1", dict(Lq=300, Lk=500, chunk=100)),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_checked_build_attention(name):
    base, kw = CASES[name]
    w = wl.WORKLOADS[base].scaled(**kw)
    x = wl.make_inputs(w)
    q, k, v = (parity.to_dev(x[n]) for n in ("Q", "K", "V"))
    ref = tk.attn(q, k, v, w.k, w.chunk, w.causal, w.scale)
    got = torch.empty_like(q)
    L = _checked()
    dt = tk.TOPK_BF16 if w.dtype == wl.BF16 else tk.TOPK_F32
    rc = L.topk_attn(q.data_ptr(), k.data_ptr(), v.data_ptr(), got.data_ptr(), w.B, w.H, w.Lq, w.Lk, w.d, w.k,
                     w.chunk, int(w.causal), w.scale, dt, _stream())
    assert rc == 0, L.topk_last_error().decode()
    torch.cuda.synchronize()
    assert L.topk_debug_bad_indices() == 0
    view = torch.int16 if q.dtype == torch.bfloat16 else torch.int32
    assert torch.equal(got.view(view), ref.view(view))


def test_checked_build_ffn_and_the_normal_build_hook():
    w = wl.WORKLOADS["c5"].scaled(N=200, d_model=256, d_ff=3000, k=256, chunk=64)
    x = wl.make_inputs(w)
    a, w1, w2 = (parity.to_dev(x[n]) for n in ("X", "W1", "W2"))
    ref = tk.ffn(a, w1, w2, w.k, w.chunk)
    got = torch.empty_like(a)
    L = _checked()
    rc = L.topk_ffn(a.data_ptr(), w1.data_ptr(), w2.data_ptr(), got.data_ptr(), w.N, w.d_model, w.d_ff, w.k,
                    w.chunk, tk.TOPK_BF16, _stream())
    assert rc == 0, L.topk_last_error().decode()
    torch.cuda.synchronize()
    assert L.topk_debug_bad_indices() == 0
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16))
    tk.lib().topk_debug_bad_indices.restype = ctypes.c_int64
    assert tk.lib().topk_debug_bad_indices() == -1
