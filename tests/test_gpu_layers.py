"""GPU parity of the PyTorch layers over libtopk (autograd functions, the multi-head
attention layer, the feed-forward layer) against the fp64 oracles.

The multi-head layer is checked step by step: its projections (PyTorch GEMMs)
against fp64 products; its heads, on the projected q, k, v the layer computed, with
the same acceptance rules as every top-k attention test (index sets equal up to
near ties, outputs within tolerance); its output and every gradient against the
layer oracle evaluated on those projections and the validated index sets."""
import math

import numpy as np
import pytest
import torch

import paper_2106_06899_amd as tk
from oracle import topk_backward as bo
from oracle import topk_mha as mo
from paper_2106_06899_amd import layers
from paper_2106_06899_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu

RTOL = {wl.F32: 1e-5, wl.BF16: 2e-2}  # layer outputs and gradients
TORCH = {wl.F32: torch.float32, wl.BF16: torch.bfloat16}


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tk.lib()
    yield


def _tensor(a, dtype):
    """numpy fp32 -> device tensor in dtype, and its exact values as fp64."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH[dtype]).cuda()
    return t, t.float().cpu().numpy().astype(np.float64)


def _rows_close(name, got, ref, rtol):
    g = np.asarray(got, np.float64).reshape(-1, np.shape(got)[-1])
    r = np.asarray(ref, np.float64).reshape(-1, np.shape(ref)[-1])
    err = np.abs(g - r).max(axis=1) / max(float(np.abs(r).max()), 1e-30)
    assert np.all(err <= rtol), f"{name}: error {err.max():.3e} > {rtol} at row {int(np.argmax(err))}"
    return float(err.max())


def test_attention_function_equals_direct_calls():
    """The autograd function's output and gradients are the library calls' own (bit for bit)."""
    w = wl.WORKLOADS["c3"].scaled(H=2, Lq=300, Lk=2000, chunk=128)
    x = wl.make_inputs(w)
    q, k, v = (parity.to_dev(x[n]).requires_grad_() for n in ("Q", "K", "V"))
    g = parity.to_dev(parity.grad_out((w.B, w.H, w.Lq, w.d), w.dtype, 90))
    out = layers.topk_attention(q, k, v, w.k, w.chunk, w.causal, w.scale)
    out.backward(g)
    o2, idx, dots = tk.attn(q.detach(), k.detach(), v.detach(), w.k, w.chunk, w.causal, w.scale, debug=True)
    d2 = tk.attn_backward(q.detach(), k.detach(), v.detach(), idx, dots, g, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(out, o2)
    for a, b in zip((q.grad, k.grad, v.grad), d2):
        assert torch.equal(a, b)


def test_ffn_function_equals_direct_calls():
    w = wl.WORKLOADS["c5"].scaled(N=200, d_model=256, d_ff=3000, k=64, chunk=64)
    x = wl.make_inputs(w)
    a, b1, b2 = (parity.to_dev(x[n]).requires_grad_() for n in ("X", "W1", "W2"))
    g = parity.to_dev(parity.grad_out((w.N, w.d_model), w.dtype, 91))
    out = layers.topk_feed_forward(a, b1, b2, w.k, w.chunk)
    out.backward(g)
    o2, idx, dots = tk.ffn(a.detach(), b1.detach(), b2.detach(), w.k, w.chunk, debug=True)
    d2 = tk.ffn_backward(a.detach(), b1.detach(), b2.detach(), idx, dots, g)
    torch.cuda.synchronize()
    assert torch.equal(out, o2)
    for t, r in zip((a.grad, b1.grad, b2.grad), d2):
        assert torch.equal(t, r)


MHA_CASES = {
    # d_head 64, bf16, non-causal, L <= 1024: the heads take the fused path
    "bf16_fused": dict(dtype=wl.BF16, B=2, L=300, H=2, dh=64, k=16, chunk=64, causal=False),
    # causal heads (chunk-tile path), ragged chunks
    "bf16_causal": dict(dtype=wl.BF16, B=1, L=333, H=3, dh=64, k=32, chunk=128, causal=True),
    "fp32_causal": dict(dtype=wl.F32, B=2, L=200, H=2, dh=32, k=8, chunk=48, causal=True),
    # BERT-base shape (d_model 768, 12 heads of 64, k 128), bidirectional (fused heads,
    # every key a candidate) and causal (chunk-tile heads)
    "bf16_bert_base": dict(dtype=wl.BF16, B=1, L=1024, H=12, dh=64, k=128, chunk=256, causal=False),
    "bf16_bert_base_causal": dict(dtype=wl.BF16, B=1, L=2048, H=12, dh=64, k=128, chunk=1024, causal=True),
}


@pytest.mark.parametrize("name", sorted(MHA_CASES))
def test_multihead_layer_parity(name):
    c = MHA_CASES[name]
    dt, B, L, H, dh, kk = c["dtype"], c["B"], c["L"], c["H"], c["dh"], c["k"]
    dm = H * dh
    _say(name, c)
    rng = np.random.Generator(np.random.PCG64(300))
    X, Xv = _tensor(rng.standard_normal((B, L, dm)), dt)
    layer = layers.TopkMultiheadAttention(dm, H, kk, c["chunk"], c["causal"], device="cuda", dtype=TORCH[dt])
    ws = {}
    with torch.no_grad():
        for name_p, shape, sd in (("qkv.weight", (3 * dm, dm), dm ** -0.5), ("qkv.bias", (3 * dm,), 0.1),
                                  ("out.weight", (dm, dm), dm ** -0.5), ("out.bias", (dm,), 0.1)):
            t, v = _tensor(sd * rng.standard_normal(shape), dt)
            dict(layer.named_parameters())[name_p].copy_(t)
            ws[name_p] = v
    X.requires_grad_()
    G, Gv = _tensor(rng.standard_normal((B, L, dm)), dt)
    Y = layer(X)
    Y.backward(G)
    # the projections the heads saw (the same GEMM, recomputed), and the heads' index sets
    with torch.no_grad():
        p = layer.qkv(X).view(B, L, 3, H, dh).permute(2, 0, 3, 1, 4)
        q, k, v = (p[t].contiguous() for t in range(3))
        out_h, idx, _ = tk.attn(q, k, v, kk, c["chunk"], c["causal"], layer.scale, debug=True)
    torch.cuda.synchronize()
    qkv = tuple(t.float().cpu().numpy().astype(np.float64) for t in (q, k, v))
    ref_qkv = mo.projections(Xv, ws["qkv.weight"], ws["qkv.bias"], H)
    errs = {"proj": max(_rows_close("projection", a, b, RTOL[dt]) for a, b in zip(qkv, ref_qkv))}
    w = wl.WORKLOADS["c2"].scaled(B=B, H=H, Lq=L, Lk=L, d=dh, k=kk, chunk=c["chunk"], causal=c["causal"],
                                  scale=layer.scale, dtype=dt)
    heads = {n: wl.Tensor(a.astype(np.float32), None, dt) for n, a in zip(("Q", "K", "V"), qkv)}
    parity.check_attn(w, heads, out_h, idx)  # index sets up to near ties, head outputs
    ix = idx.cpu().numpy()
    args = (Xv, ws["qkv.weight"], ws["qkv.bias"], ws["out.weight"], ws["out.bias"], H)
    Yr, _ = mo.mha_forward(*args, kk, c["chunk"], c["causal"], layer.scale, top_idx=ix, qkv=qkv)
    errs["Y"] = _rows_close("layer output", Y.detach().float().cpu().numpy(), Yr, RTOL[dt])
    ref = mo.mha_backward(*args, ix, Gv, layer.scale, qkv=qkv)
    got = (X.grad, layer.qkv.weight.grad, layer.qkv.bias.grad, layer.out.weight.grad, layer.out.bias.grad)
    for n, a, b in zip(("dX", "dWqkv", "dbqkv", "dWo", "dbo"), got, ref):
        a = a.float().cpu().numpy()
        errs[n] = _rows_close(n, a.reshape(-1, a.shape[-1]) if a.ndim > 1 else a[None], b if b.ndim > 1 else b[None],
                              RTOL[dt])
    _say(name, "ok", errs)


def test_feed_forward_layer_parity():
    """TopkFeedForward on [2, 150, 256] bf16 tokens, d_ff 2000, k 64: output against the
    oracle on validated index sets, gradients against the backward oracle."""
    dt = wl.BF16
    rng = np.random.Generator(np.random.PCG64(301))
    dm, dff, kk, C = 256, 2000, 64, 128
    layer = layers.TopkFeedForward(dm, dff, kk, C, device="cuda", dtype=torch.bfloat16)
    with torch.no_grad():
        t1, W1 = _tensor(0.05 * rng.standard_normal((dff, dm)), dt)
        t2, W2 = _tensor(0.05 * rng.standard_normal((dff, dm)), dt)
        layer.w1.copy_(t1)
        layer.w2.copy_(t2)
    X, Xv = _tensor(rng.standard_normal((2, 150, dm)), dt)
    X.requires_grad_()
    G, Gv = _tensor(rng.standard_normal((2, 150, dm)), dt)
    Y = layer(X)
    Y.backward(G)
    with torch.no_grad():
        out, idx, _ = tk.ffn(X.detach().reshape(-1, dm), layer.w1, layer.w2, kk, C, debug=True)
    torch.cuda.synchronize()
    w = wl.WORKLOADS["c5"].scaled(N=300, d_model=dm, d_ff=dff, k=kk, chunk=C)
    xs = {"X": wl.Tensor(Xv.reshape(-1, dm).astype(np.float32), None, dt), "W1": wl.Tensor(W1.astype(np.float32), None, dt),
          "W2": wl.Tensor(W2.astype(np.float32), None, dt)}
    parity.check_ffn(w, xs, out, idx)
    assert torch.equal(Y.detach().reshape(-1, dm), out)
    ref, mag = bo.oracle_ffn_backward(Xv.reshape(-1, dm), W1, W2, idx.cpu().numpy(), Gv.reshape(-1, dm), chunk=C,
                                      magnitudes=True)
    got = (X.grad.reshape(-1, dm), layer.w1.grad, layer.w2.grad)
    errs = {n: parity.check_grad_rows(n, a, b, m, wl.BF16) for n, a, b, m in zip(("dX", "dW1", "dW2"), got, ref, mag)}
    _say("ffn layer ok", errs)
