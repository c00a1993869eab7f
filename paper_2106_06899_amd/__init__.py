"""MI355X (gfx950) top-k attention -- Python binding of ``libtopk.so``.

Argument marshalling only: every step of the computation runs in the HIP kernels
of ``libtopk.so`` (built from ``csrc/`` by ``paper_2106_06899_amd.build``). There
is no CPU or PyTorch fallback; if the library is missing the calls raise.

* ``attn(q, k, v, topk, chunk, causal, scale)`` -> top-k attention (Eq. 4, softmax)
* ``ffn(x, w1, w2, topk, chunk)``               -> top-k feed-forward (Eq. 3 + Eq. 4, ReLU)

Tensors live on the GPU (PyTorch provides device memory and the stream); the
work is enqueued on ``torch.cuda.current_stream()``. The workspace is a PyTorch
byte tensor registered with ``topk_set_workspace`` for the duration of the call,
so PyTorch's memory statistics include it.
"""
from __future__ import annotations

import ctypes
import math
import os

__all__ = ["attn", "attn_dense", "scan_ablation", "probe_mfma", "ffn", "attn_workspace_bytes", "ffn_workspace_bytes", "attn_path", "ffn_path",
           "mfma_layout", "lib", "TopkError", "LIB_PATH", "profile_begin", "profile_end", "STAGES",
           "attn_backward", "ffn_backward", "set_backward_lists", "set_memory_budget", "last_fallback_rows"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtopk.so")

TOPK_F32, TOPK_BF16 = 0, 1
MAX_SELECT_K = 2048  # largest k the select handles (k = Lk above it runs attn_dense)
TOPK_LISTS_AUTO, TOPK_LISTS_BUCKET, TOPK_LISTS_ATOMIC = 0, 1, 2
_STATUS = {0: "OK", -1: "TOPK_E_INVAL", -2: "TOPK_E_NULL", -3: "TOPK_E_ALIGN", -4: "TOPK_E_UNSUPPORTED",
           -5: "TOPK_E_NOMEM", -6: "TOPK_E_HIP"}

_lib = None


class TopkError(RuntimeError):
    """A non-OK status from libtopk; ``status`` holds the code."""

    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load ``libtopk.so`` (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2106_06899_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    i64, vp, i32, f32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    attn_args = [vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i64, i32, f32, i32, vp]
    ffn_args = [vp, vp, vp, vp, i64, i64, i64, i64, i64, i32, vp]
    sigs = {
        "topk_attn": (attn_args, i32),
        "topk_attn_noalloc": (attn_args, i32),
        "topk_attn_dense": ([vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, f32, i32, vp], i32),
        "topk_noalloc_scratch_bytes": ([], ctypes.c_size_t),
        "topk_attn_debug": (attn_args + [vp, vp], i32),
        "topk_ffn": (ffn_args, i32),
        "topk_ffn_debug": (ffn_args + [vp, vp], i32),
        "topk_attn_with_cache": (attn_args + [vp, vp], i32),
        "topk_ffn_with_cache": (ffn_args + [vp, vp], i32),
        "topk_attn_workspace_bytes": ([i64] * 7 + [i32, i32], ctypes.c_size_t),
        "topk_ffn_workspace_bytes": ([i64] * 5 + [i32], ctypes.c_size_t),
        "topk_set_workspace": ([vp, ctypes.c_size_t], i32),
        "topk_last_error": ([], ctypes.c_char_p),
        "topk_last_fallback_rows": ([], i64),
        "topk_set_backward_lists": ([i32], i32),
        "topk_set_memory_budget": ([ctypes.c_size_t], i32),
        "topk_attn_backward": ([vp] * 9 + [i64] * 6 + [ctypes.c_float, i32, vp], i32),
        "topk_ffn_backward": ([vp] * 9 + [i64] * 4 + [i32, vp], i32),
        "topk_attn_backward_workspace_bytes": ([i64] * 6 + [i32], ctypes.c_size_t),
        "topk_ffn_backward_workspace_bytes": ([i64] * 4 + [i32], ctypes.c_size_t),
        "topk_attn_path": ([i64] * 7 + [i32, i32], i32),
        "topk_ffn_path": ([i64] * 5 + [i32], i32),
        "topk_selftest_mfma_layout": ([vp, vp, vp], i32),
        "topk_scan_ablation": ([vp, vp] + [i64] * 7 + [i32, vp], i32),
        "topk_probe_mfma": ([ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), vp], i32),
        "topk_profile_begin": ([], i32),
        "topk_profile_end": ([ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), i32], i32),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def _raise(rc: int):
    if rc != 0:
        raise TopkError(rc, lib().topk_last_error().decode())


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return TOPK_F32
    if t.dtype == torch.bfloat16:
        return TOPK_BF16
    raise TypeError(f"unsupported dtype {t.dtype}: use torch.float32 or torch.bfloat16")


def _check(t, name, ndim, dtype, device):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got {tuple(t.shape)}")
    if t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _stream_ptr(device):
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _with_workspace(nbytes: int, device, fn):
    import torch
    ws = torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)
    L = lib()
    _raise(L.topk_set_workspace(ctypes.c_void_p(ws.data_ptr()), int(nbytes)))
    try:
        _raise(fn())
    finally:
        L.topk_set_workspace(None, 0)
    return ws  # caller keeps it until the call is enqueued (stream-ordered reuse is safe)


def attn_workspace_bytes(B, H, Lq, Lk, d, k, chunk=0, causal=False, dtype=TOPK_BF16) -> int:
    return int(lib().topk_attn_workspace_bytes(B, H, Lq, Lk, d, k, chunk, int(causal), dtype))


def ffn_workspace_bytes(N, d_model, d_ff, k, chunk=0, dtype=TOPK_BF16) -> int:
    return int(lib().topk_ffn_workspace_bytes(N, d_model, d_ff, k, chunk, dtype))


def attn_path(B, H, Lq, Lk, d, k, chunk=0, causal=False, dtype=TOPK_BF16) -> int:
    """1 = fused score+filter path, 2 = chunk-tile path (negative: invalid arguments)."""
    return int(lib().topk_attn_path(B, H, Lq, Lk, d, k, chunk, int(causal), dtype))


def ffn_path(N, d_model, d_ff, k, chunk=0, dtype=TOPK_BF16) -> int:
    return int(lib().topk_ffn_path(N, d_model, d_ff, k, chunk, dtype))


def attn(q, k, v, topk: int, chunk: int = 0, causal: bool = False, scale: float | None = None,
         debug: bool = False, cache: bool = False):
    """Top-k attention over [B, H, L, d] tensors; returns out (and idx, scores if debug
    or cache).

    ``scale`` is the softmax temperature 1/lambda of Eq. 1 (default 1/sqrt(d)).
    ``debug`` also returns the selected indices (int32 [B, H, Lq, topk], -1 pads) and
    their raw fp32 scores (-inf pads), ordered by (score desc, index asc), and records
    the fallback row count (the call waits for the stream). ``cache`` returns the same
    two tensors, the backward pass's input-checkpointing cache, without waiting.
    """
    import torch
    device = q.device
    _check(q, "q", 4, q.dtype, device)
    _check(k, "k", 4, q.dtype, device)
    _check(v, "v", 4, q.dtype, device)
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    if tuple(k.shape) != (B, H, Lk, d) or tuple(v.shape) != (B, H, Lk, d):
        raise ValueError(f"shape mismatch q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")
    dt = _dtype_code(q)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if topk == Lk and topk > MAX_SELECT_K and not (debug or cache):
        return attn_dense(q, k, v, chunk, causal, scale)
    out = torch.empty_like(q)
    idx = torch.empty((B, H, Lq, topk), dtype=torch.int32, device=device) if debug or cache else None
    sc = torch.empty((B, H, Lq, topk), dtype=torch.float32, device=device) if debug or cache else None
    L = lib()
    nbytes = L.topk_attn_workspace_bytes(B, H, Lq, Lk, d, topk, chunk, int(causal), dt)
    if nbytes == 0:  # invalid arguments: let the call report why
        _raise(L.topk_attn(None, None, None, None, B, H, Lq, Lk, d, topk, chunk, int(causal), scale, dt, None))
    args = (q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, Lq, Lk, d, topk, chunk, int(causal),
            float(scale), dt, _stream_ptr(device))
    if debug or cache:
        fn = L.topk_attn_debug if debug else L.topk_attn_with_cache
        _with_workspace(nbytes, device, lambda: fn(*args, idx.data_ptr(), sc.data_ptr()))
        return out, idx, sc
    _with_workspace(nbytes, device, lambda: L.topk_attn(*args))
    return out


def scan_ablation(q, k, topk: int, chunk: int = 0, score_only: bool = False):
    """Measurement hook: only the fused path's score kernel of an attention call
    (``score_only``: the score-core ablation without the filter); time it with
    profile_begin / profile_end (stage "score")."""
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    _raise(lib().topk_scan_ablation(q.data_ptr(), k.data_ptr(), B, H, Lq, Lk, d, topk, chunk, int(score_only),
                                    _stream_ptr(q.device)))


def probe_mfma():
    """(sustained bf16 MFMA TFLOP/s, shader clock MHz) of the current device."""
    t, c = ctypes.c_double(), ctypes.c_double()
    import torch
    _raise(lib().topk_probe_mfma(ctypes.byref(t), ctypes.byref(c), _stream_ptr(torch.device("cuda", torch.cuda.current_device()))))
    return t.value, c.value


def attn_dense(q, k, v, chunk: int = 0, causal: bool = False, scale: float | None = None):
    """Query chunking with the top-k disabled (the paper's comparison baseline): every
    valid key contributes through the softmax of Eq. 1 (k = Lk). bf16, d = 64 or 128;
    no workspace."""
    import torch
    device = q.device
    _check(q, "q", 4, q.dtype, device)
    _check(k, "k", 4, q.dtype, device)
    _check(v, "v", 4, q.dtype, device)
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    if tuple(k.shape) != (B, H, Lk, d) or tuple(v.shape) != (B, H, Lk, d):
        raise ValueError(f"shape mismatch q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")
    dt = _dtype_code(q)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = torch.empty_like(q)
    _raise(lib().topk_attn_dense(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, Lq, Lk, d, chunk,
                                 int(causal), float(scale), dt, _stream_ptr(device)))
    return out


def ffn(x, w1, w2, topk: int, chunk: int = 0, debug: bool = False, cache: bool = False):
    """Top-k feed-forward layer: x [N, d_model], w1/w2 [d_ff, d_model] (row j = key/value j).
    ``debug`` / ``cache`` as for ``attn``."""
    import torch
    device = x.device
    _check(x, "x", 2, x.dtype, device)
    _check(w1, "w1", 2, x.dtype, device)
    _check(w2, "w2", 2, x.dtype, device)
    N, dm = x.shape
    dff = w1.shape[0]
    if tuple(w1.shape) != (dff, dm) or tuple(w2.shape) != (dff, dm):
        raise ValueError(f"shape mismatch x {tuple(x.shape)} w1 {tuple(w1.shape)} w2 {tuple(w2.shape)}")
    dt = _dtype_code(x)
    out = torch.empty_like(x)
    idx = torch.empty((N, topk), dtype=torch.int32, device=device) if debug or cache else None
    sc = torch.empty((N, topk), dtype=torch.float32, device=device) if debug or cache else None
    L = lib()
    nbytes = L.topk_ffn_workspace_bytes(N, dm, dff, topk, chunk, dt)
    if nbytes == 0:
        _raise(L.topk_ffn(None, None, None, None, N, dm, dff, topk, chunk, dt, None))
    args = (x.data_ptr(), w1.data_ptr(), w2.data_ptr(), out.data_ptr(), N, dm, dff, topk, chunk, dt,
            _stream_ptr(device))
    if debug or cache:
        fn = L.topk_ffn_debug if debug else L.topk_ffn_with_cache
        _with_workspace(nbytes, device, lambda: fn(*args, idx.data_ptr(), sc.data_ptr()))
        return out, idx, sc
    _with_workspace(nbytes, device, lambda: L.topk_ffn(*args))
    return out


def attn_backward(q, k, v, idx, dots, d_out, scale: float | None = None):
    """Gradients (d_q, d_k, d_v) of top-k attention from the forward's cache: idx and
    dots are what ``attn(..., debug=True)`` returns (selected keys, their raw scores).
    Input checkpointing (Section 2.2): no Lq x Lk matrix is formed."""
    import torch
    device = q.device
    _check(q, "q", 4, q.dtype, device)
    _check(k, "k", 4, q.dtype, device)
    _check(v, "v", 4, q.dtype, device)
    _check(d_out, "d_out", 4, q.dtype, device)
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    topk = idx.shape[-1]
    if tuple(k.shape) != (B, H, Lk, d) or tuple(v.shape) != (B, H, Lk, d) or tuple(d_out.shape) != (B, H, Lq, d):
        raise ValueError("shape mismatch")
    if idx.dtype != torch.int32 or dots.dtype != torch.float32 or tuple(idx.shape) != (B, H, Lq, topk) \
            or tuple(dots.shape) != (B, H, Lq, topk) or not idx.is_contiguous() or not dots.is_contiguous():
        raise ValueError("idx (int32) and dots (float32) must be contiguous [B, H, Lq, k]")
    dt = _dtype_code(q)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    L = lib()
    nbytes = L.topk_attn_backward_workspace_bytes(B, H, Lq, Lk, d, topk, dt)
    args = (q.data_ptr(), k.data_ptr(), v.data_ptr(), idx.data_ptr(), dots.data_ptr(), d_out.data_ptr(),
            dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), B, H, Lq, Lk, d, topk, float(scale), dt, _stream_ptr(device))
    if nbytes == 0:
        _raise(L.topk_attn_backward(*args))
    _with_workspace(nbytes, device, lambda: L.topk_attn_backward(*args))
    return dq, dk, dv


def ffn_backward(x, w1, w2, idx, dots, d_out):
    """Gradients (d_x, d_w1, d_w2) of the top-k feed-forward layer from the forward's
    cache (idx, dots as ``ffn(..., debug=True)`` returns them)."""
    import torch
    device = x.device
    for t, n in ((x, "x"), (w1, "w1"), (w2, "w2"), (d_out, "d_out")):
        _check(t, n, 2, x.dtype, device)
    N, dm = x.shape
    dff = w1.shape[0]
    topk = idx.shape[-1]
    if tuple(w1.shape) != (dff, dm) or tuple(w2.shape) != (dff, dm) or tuple(d_out.shape) != (N, dm):
        raise ValueError("shape mismatch")
    if idx.dtype != torch.int32 or dots.dtype != torch.float32 or tuple(idx.shape) != (N, topk) \
            or tuple(dots.shape) != (N, topk) or not idx.is_contiguous() or not dots.is_contiguous():
        raise ValueError("idx (int32) and dots (float32) must be contiguous [N, k]")
    dt = _dtype_code(x)
    dx, dw1, dw2 = torch.empty_like(x), torch.empty_like(w1), torch.empty_like(w2)
    L = lib()
    nbytes = L.topk_ffn_backward_workspace_bytes(N, dm, dff, topk, dt)
    args = (x.data_ptr(), w1.data_ptr(), w2.data_ptr(), idx.data_ptr(), dots.data_ptr(), d_out.data_ptr(),
            dx.data_ptr(), dw1.data_ptr(), dw2.data_ptr(), N, dm, dff, topk, dt, _stream_ptr(device))
    if nbytes == 0:
        _raise(L.topk_ffn_backward(*args))
    _with_workspace(nbytes, device, lambda: L.topk_ffn_backward(*args))
    return dx, dw1, dw2


STAGES = ("score", "select", "redo", "finalize", "backward")


def profile_begin():
    """Start per-stage HIP-event timing of this thread's calls (see topk_profile_begin)."""
    _raise(lib().topk_profile_begin())


def profile_end():
    """Stop timing; return {stage: (total_ms, launches)} over the calls since profile_begin."""
    ms = (ctypes.c_double * len(STAGES))()
    n = (ctypes.c_int64 * len(STAGES))()
    _raise(lib().topk_profile_end(ms, n, len(STAGES)))
    return {s: (ms[i], n[i]) for i, s in enumerate(STAGES)}


def set_memory_budget(nbytes: int) -> None:
    """Most workspace a forward call sizes for itself (process-wide; 0 = 8 GiB). A small
    budget runs the query chunks in more passes (one chunk per pass at the limit)."""
    _raise(lib().topk_set_memory_budget(int(nbytes)))


def set_backward_lists(mode: int) -> None:
    """How backward calls group the selected pairs by key (process-wide):
    TOPK_LISTS_AUTO, TOPK_LISTS_BUCKET (stable bucket sort) or TOPK_LISTS_ATOMIC."""
    _raise(lib().topk_set_backward_lists(int(mode)))


def last_fallback_rows() -> int:
    """Rows the last debug call on this thread selected through a fallback path (-1: none / failed)."""
    return int(lib().topk_last_fallback_rows())


def mfma_layout(device="cuda"):
    """(rows, cols) int32 [64, 16]: output row / column held by lane l, register v of
    the bf16 32x32x16 MFMA the fused scan uses (test hook)."""
    import torch
    rows = torch.full((64, 16), -1, dtype=torch.int32, device=device)
    cols = torch.full((64, 16), -1, dtype=torch.int32, device=device)
    _raise(lib().topk_selftest_mfma_layout(ctypes.c_void_p(rows.data_ptr()), ctypes.c_void_p(cols.data_ptr()),
                                           _stream_ptr(torch.device(device))))
    return rows, cols
