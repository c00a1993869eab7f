"""Linear memory (Section 2.2): the memory a call needs beyond its inputs and output
is the workspace the library reports, and it grows at most linearly with the
sequence length. Measured with PyTorch's allocator, which holds the workspace (the
binding allocates it as a PyTorch tensor for the duration of the call)."""
import numpy as np
import pytest
import torch

import paper_2106_06899_amd as tk
from paper_2106_06899_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tk.lib()
    yield


def test_peak_memory_linear_in_length():
    dev = torch.device("cuda:0")
    # lengths on one path (the fused path; shorter rows take the chunk-tile paths,
    # whose workspace per row differs)
    lengths = (8192, 16384, 32768, 65536)
    extra = {}
    for L in lengths:
        w = wl.WORKLOADS["c3"].scaled(H=4, Lq=L, Lk=L)
        _say("memory", w)
        assert tk.attn_path(w.B, w.H, L, L, w.d, w.k, w.chunk, w.causal) == 1
        x = wl.make_inputs(w)
        q, k, v = (parity.to_dev(x[n]) for n in ("Q", "K", "V"))
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated(dev)  # everything alive before the call, Q, K, V included
        torch.cuda.reset_peak_memory_stats(dev)
        out = tk.attn(q, k, v, w.k, w.chunk, w.causal, w.scale)
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated(dev)
        ws = tk.attn_workspace_bytes(w.B, w.H, L, L, w.d, w.k, w.chunk, w.causal)
        extra[L] = peak - base - out.numel() * out.element_size()
        _say("L", L, "beyond inputs and output", extra[L], "workspace", ws)
        # the workspace is the call's only allocation besides its output (allocator
        # granularity: 2 MiB)
        assert ws <= extra[L] <= ws + (2 << 20)
        del q, k, v, out
    for a, b in zip(lengths, lengths[1:]):
        assert extra[b] <= 2.2 * extra[a], f"memory grew {extra[b] / extra[a]:.2f}x from L {a} to {b}"
