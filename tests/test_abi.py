"""CPU tests of the C-ABI library: it loads, exports every declared symbol, validates
arguments synchronously (no GPU needed: invalid calls return before any HIP call),
and its host-side planning (path choice, workspace sizing) behaves as documented."""
import ctypes
import os
import re

import pytest

import paper_2106_06899_amd as tk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "topk_attn.h")

E_INVAL, E_NULL, E_ALIGN, E_UNSUPPORTED = -1, -2, -3, -4
FAKE = 0x10000  # aligned, never dereferenced: every call below fails validation first


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(topk_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 10
    L = ctypes.CDLL(tk.LIB_PATH)
    for n in names:
        assert hasattr(L, n), f"libtopk.so does not export {n}"


def _attn(**kw):
    a = dict(Q=FAKE, K=FAKE, V=FAKE, out=FAKE, B=1, H=2, Lq=64, Lk=128, d=64, k=8, chunk=0, causal=0,
             scale=0.125, dtype=1)
    a.update(kw)
    L = tk.lib()
    return L.topk_attn(a["Q"], a["K"], a["V"], a["out"], a["B"], a["H"], a["Lq"], a["Lk"], a["d"], a["k"],
                       a["chunk"], a["causal"], a["scale"], a["dtype"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(k=0), E_INVAL), (dict(k=129), E_INVAL), (dict(B=0), E_INVAL), (dict(Lq=0), E_INVAL),
    (dict(Lk=0), E_INVAL), (dict(d=0), E_INVAL), (dict(chunk=-1), E_INVAL), (dict(causal=2), E_INVAL),
    (dict(scale=0.0), E_INVAL), (dict(scale=-1.0), E_INVAL), (dict(scale=float("nan")), E_INVAL),
    (dict(scale=float("inf")), E_INVAL), (dict(dtype=7), E_INVAL),
    (dict(Q=None), E_NULL), (dict(out=None), E_NULL), (dict(V=None), E_NULL),
    (dict(K=FAKE + 8), E_ALIGN), (dict(out=FAKE + 4), E_ALIGN),
    (dict(d=60), E_UNSUPPORTED), (dict(d=2048), E_UNSUPPORTED), (dict(Lk=10000, k=5000), E_UNSUPPORTED),
])
def test_attn_validation(kw, code):
    assert _attn(**kw) == code
    msg = tk.lib().topk_last_error().decode()
    assert msg, "a failing call must leave a message"


def test_ffn_validation():
    L = tk.lib()
    assert L.topk_ffn(FAKE, FAKE, FAKE, FAKE, 16, 64, 128, 0, 0, 1, None) == E_INVAL
    assert L.topk_ffn(FAKE, FAKE, FAKE, FAKE, 16, 64, 128, 129, 0, 1, None) == E_INVAL
    assert L.topk_ffn(None, FAKE, FAKE, FAKE, 16, 64, 128, 8, 0, 1, None) == E_NULL
    assert L.topk_ffn(FAKE, FAKE, FAKE, FAKE, 16, 63, 128, 8, 0, 1, None) == E_UNSUPPORTED
    assert L.topk_ffn_debug(FAKE, FAKE, FAKE, FAKE, 16, 64, 128, 8, -3, 1, None, None, None) == E_INVAL


def test_set_workspace_validation():
    L = tk.lib()
    assert L.topk_set_workspace(None, 16) == E_NULL
    assert L.topk_set_workspace(ctypes.c_void_p(FAKE + 64), 1024) == E_ALIGN
    assert L.topk_set_workspace(None, 0) == 0


def test_path_choice_for_the_five_workloads():
    # c1 fp32 -> chunk-tile; c2 short rows -> fused (every key a candidate);
    # c3 long rows -> fused (sampled threshold); c4 causal -> filtered chunk-tile; c5 FFN k 512 -> chunk-tile
    assert tk.attn_path(1, 1, 1024, 1024, 64, 32, 256, False, tk.TOPK_F32) == 2
    assert tk.attn_path(8, 12, 512, 512, 64, 64, 512, False, tk.TOPK_BF16) == 1
    assert tk.attn_path(1, 16, 32768, 32768, 64, 64, 1024, False, tk.TOPK_BF16) == 1
    assert tk.attn_path(4, 16, 8192, 8192, 128, 128, 1024, True, tk.TOPK_BF16) == 4
    assert tk.ffn_path(16384, 1024, 65536, 512, 1024, tk.TOPK_BF16) == 4
    assert tk.attn_path(1, 1, 10, 10, 64, 0) == E_INVAL


def test_workspace_is_linear_in_length_and_capped():
    """Per-chunk working memory does not depend on L for the fused path (O(C*k) per
    chunk); total workspace grows linearly with the number of chunks until the
    budget caps the chunks in flight."""
    sizes = [tk.attn_workspace_bytes(1, 16, L, L, 64, 64, 1024, False, tk.TOPK_BF16) for L in
             (16384, 32768, 65536, 131072)]
    assert all(s > 0 for s in sizes)
    assert sizes[1] <= 2.2 * sizes[0]
    assert max(sizes) <= (8 << 30) + (64 << 20)
    tile = [tk.attn_workspace_bytes(1, 1, L, L, 64, 32, 256, False, tk.TOPK_F32) for L in (1024, 2048, 4096)]
    # chunk-tile path: one chunk costs O(C * Lk); the whole call O(L^2) until capped
    assert tile[1] > tile[0]
    assert tk.attn_workspace_bytes(1, 1, 10, 10, 64, 0) == 0
    assert tk.ffn_workspace_bytes(16384, 1024, 65536, 512, 1024) <= (8 << 30) + (64 << 20)


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU; asking for more exits with a message before touching a GPU."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def test_backward_list_modes():
    """The list-mode setting is validated; the bucket sort needs more workspace than
    atomic counters (a stage entry per pair and the tile counts) and refuses heads of
    more than 2^19 keys, which the automatic mode gives to atomic counters."""
    L = tk.lib()
    assert L.topk_set_backward_lists(3) == E_INVAL
    assert L.topk_set_backward_lists(-1) == E_INVAL
    shape = (1, 4, 4096, 8192, 64, 64, 1)
    try:
        tk.set_backward_lists(tk.TOPK_LISTS_ATOMIC)
        atomic = L.topk_attn_backward_workspace_bytes(*shape)
        tk.set_backward_lists(tk.TOPK_LISTS_BUCKET)
        bucket = L.topk_attn_backward_workspace_bytes(*shape)
        assert bucket > atomic > 0
        pairs = 4 * 4096 * 64
        assert bucket - atomic >= pairs * 4  # 8-byte stage entries instead of 4-byte places
        big = (1, 1, 16, (1 << 19) + 1, 8, 4, 1)
        assert L.topk_attn_backward_workspace_bytes(*big) == 0  # bucket sort refuses
        tk.set_backward_lists(tk.TOPK_LISTS_AUTO)
        assert L.topk_attn_backward_workspace_bytes(*shape) == bucket
        assert L.topk_attn_backward_workspace_bytes(*big) > 0
    finally:
        tk.set_backward_lists(tk.TOPK_LISTS_AUTO)


def test_memory_budget_bounds_the_workspace():
    """The budget caps the workspace a call sizes for itself; at a budget below one
    chunk's needs one chunk runs per pass, and 0 restores the default."""
    L = tk.lib()
    shape = (1, 4, 8192, 8192, 64, 64, 512, 0, 1)
    default = L.topk_attn_workspace_bytes(*shape)
    try:
        tk.set_memory_budget(1)
        one = L.topk_attn_workspace_bytes(*shape)
        tk.set_memory_budget(64 << 20)
        mid = L.topk_attn_workspace_bytes(*shape)
        assert 0 < one < mid <= default
        assert mid <= (64 << 20) + one  # the budget plus at most the fixed part
    finally:
        tk.set_memory_budget(0)
    assert L.topk_attn_workspace_bytes(*shape) == default


def test_causal_split_path():
    """Causal masks with long keys take the fused path for rows from 1024 R on and the
    chunk-tile path below (reported as 3); short keys stay on the chunk-tile path."""
    assert tk.attn_path(1, 12, 65536, 65536, 64, 128, 1024, True, tk.TOPK_BF16) == 3
    assert tk.attn_path(1, 1, 4500, 4500, 64, 16, 512, True, tk.TOPK_BF16) == 3
    assert tk.attn_path(1, 1, 3000, 4500, 64, 16, 512, True, tk.TOPK_BF16) == 4  # every row below 1024 R: filtered tiles
    assert tk.attn_path(4, 16, 8192, 8192, 128, 128, 1024, True, tk.TOPK_BF16) == 4  # Lk < 256 k: filtered tiles
    assert tk.attn_path(1, 1, 4500, 4500, 64, 16, 512, True, tk.TOPK_F32) == 2
    assert tk.attn_workspace_bytes(1, 12, 65536, 65536, 64, 128, 1024, True) > 0
