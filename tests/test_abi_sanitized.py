"""CPU test of the C ABI's host code under AddressSanitizer and
UndefinedBehaviorSanitizer: ``libtopk_san.so`` (host code instrumented, device code
unchanged) is loaded in a child process with the sanitizer runtime preloaded, and
every argument check and planning entry point is driven over valid, boundary and
invalid arguments. None of these calls reaches the GPU (invalid calls return before
any HIP call; planning is host arithmetic), so the test runs without one. Any
sanitizer report aborts the child and fails the test."""
import os
import subprocess
import sys
import textwrap

import pytest

from paper_2106_06899_amd import build as b

CHILD = textwrap.dedent(r"""
    import ctypes, sys
    L = ctypes.CDLL(sys.argv[1])
    i64, vp, i32, f32, sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    attn = [vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i64, i32, f32, i32, vp]
    sigs = {"topk_attn": (attn, i32), "topk_attn_debug": (attn + [vp, vp], i32),
            "topk_attn_noalloc": (attn, i32),
            "topk_attn_dense": ([vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i32, f32, i32, vp], i32),
            "topk_ffn": ([vp, vp, vp, vp, i64, i64, i64, i64, i64, i32, vp], i32),
            "topk_attn_workspace_bytes": ([i64] * 7 + [i32, i32], sz),
            "topk_ffn_workspace_bytes": ([i64] * 5 + [i32], sz),
            "topk_attn_path": ([i64] * 7 + [i32, i32], i32), "topk_ffn_path": ([i64] * 5 + [i32], i32),
            "topk_attn_backward_workspace_bytes": ([i64] * 6 + [i32], sz),
            "topk_ffn_backward_workspace_bytes": ([i64] * 4 + [i32], sz),
            "topk_set_workspace": ([vp, sz], i32), "topk_set_memory_budget": ([sz], i32),
            "topk_last_error": ([], ctypes.c_char_p), "topk_noalloc_scratch_bytes": ([], sz)}
    for n, (a, r) in sigs.items():
        f = getattr(L, n); f.argtypes = a; f.restype = r
    FAKE = 0x10000
    calls = 0
    # planning over a grid of shapes, both dtypes, causal or not
    for (B, H, Lq, Lk, d) in [(1, 1, 1, 1, 8), (2, 3, 77, 129, 64), (1, 16, 32768, 32768, 64),
                              (4, 16, 8192, 8192, 128), (1, 12, 65536, 65536, 64), (1, 1, 5, 1 << 20, 1024)]:
        for k in sorted({1, min(7, Lk), min(64, Lk), min(128, Lk), min(512, Lk), min(2048, Lk), Lk}):
            for chunk in (0, 1, 7, 1024):
                for causal in (0, 1):
                    for dt in (0, 1):
                        L.topk_attn_workspace_bytes(B, H, Lq, Lk, d, k, chunk, causal, dt)
                        L.topk_attn_path(B, H, Lq, Lk, d, k, chunk, causal, dt)
                        calls += 2
            L.topk_attn_backward_workspace_bytes(B, H, Lq, Lk, d, min(k, 2048), 1)
    for (N, dm, dff) in [(1, 8, 1), (16384, 1024, 65536), (1 << 18, 768, 65536), (100, 96, 3000)]:
        for k in sorted({1, min(512, dff), dff}):
            for chunk in (0, 3, 16384):
                for dt in (0, 1):
                    L.topk_ffn_workspace_bytes(N, dm, dff, k, chunk, dt)
                    L.topk_ffn_path(N, dm, dff, k, chunk, dt)
                    calls += 2
        L.topk_ffn_backward_workspace_bytes(N, dm, dff, min(512, dff), 1)
    # invalid arguments: each returns before any HIP call, with a message
    bad = [dict(B=0), dict(H=-1), dict(Lq=0), dict(Lk=0), dict(d=0), dict(d=7), dict(d=2048), dict(k=0),
           dict(k=200), dict(chunk=-1), dict(causal=2), dict(scale=0.0), dict(scale=float("inf")),
           dict(scale=float("nan")), dict(dtype=5), dict(Q=0), dict(out=0), dict(Q=FAKE + 2)]
    for kw in bad:
        a = dict(Q=FAKE, K=FAKE, V=FAKE, out=FAKE, B=1, H=2, Lq=64, Lk=128, d=64, k=8, chunk=0, causal=0,
                 scale=0.125, dtype=1)
        a.update(kw)
        args = (a["Q"], a["K"], a["V"], a["out"], a["B"], a["H"], a["Lq"], a["Lk"], a["d"], a["k"], a["chunk"],
                a["causal"], a["scale"], a["dtype"], None)
        for fn in (L.topk_attn, L.topk_attn_noalloc):
            rc = fn(*args)
            assert rc < 0, (kw, rc)
            assert L.topk_last_error(), kw
            calls += 1
        rc = L.topk_attn_debug(*args, None, None)
        assert rc < 0, (kw, rc)
    assert L.topk_attn_dense(FAKE, FAKE, FAKE, FAKE, 1, 1, 64, 64, 96, 0, 0, 0.125, 1, None) == -4
    assert L.topk_set_workspace(None, 16) == -2 and L.topk_set_workspace(FAKE + 8, 16) == -3
    assert L.topk_set_workspace(None, 0) == 0
    assert L.topk_set_memory_budget(1 << 30) == 0 and L.topk_set_memory_budget(0) == 0
    assert L.topk_noalloc_scratch_bytes() == 128 << 20
    print("sanitized ABI calls:", calls)
""")


def test_host_code_under_sanitizers():
    rt = b.sanitizer_runtime()
    if rt is None:
        pytest.skip("no AddressSanitizer runtime in this ROCm install")
    if not os.path.exists(b.LIB_SAN):
        b.build(variants=("san",))
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", CHILD, b.LIB_SAN], env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, f"sanitized run failed ({r.returncode}):\n{r.stdout[-3000:]}\n{r.stderr[-6000:]}"
    assert "sanitized ABI calls:" in r.stdout
