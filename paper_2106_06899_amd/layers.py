"""PyTorch layers over libtopk: top-k attention as a drop-in multi-head attention
layer (Section 2.1 with Eq. 4 per head) and the top-k feed-forward layer (Eq. 3),
each with a backward pass by input checkpointing (Section 2.2): the forward keeps
only its inputs and the selected keys with their raw scores, the backward calls
``topk_attn_backward`` / ``topk_ffn_backward``.

The projections around the attention are plain GEMMs left to PyTorch (rocBLAS);
every top-k step runs in libtopk's kernels.
"""
from __future__ import annotations

import math

import torch

from . import attn, attn_backward, attn_dense, ffn, ffn_backward


class TopkAttentionFunction(torch.autograd.Function):
    """out = top-k attention(q, k, v) over [B, H, L, d] tensors, differentiable in
    q, k and v. The selection itself carries no gradient (the index set is piecewise
    constant in the inputs)."""

    @staticmethod
    def forward(ctx, q, k, v, topk: int, chunk: int, causal: bool, scale: float):
        out, idx, dots = attn(q, k, v, topk, chunk, causal, scale, cache=True)
        ctx.save_for_backward(q, k, v, idx, dots)
        ctx.scale = scale
        return out

    @staticmethod
    def backward(ctx, d_out):
        q, k, v, idx, dots = ctx.saved_tensors
        dq, dk, dv = attn_backward(q, k, v, idx, dots, d_out.contiguous(), ctx.scale)
        return dq, dk, dv, None, None, None, None


class TopkFFNFunction(torch.autograd.Function):
    """out = top-k feed-forward layer(x) with keys w1 and values w2 (Eq. 3, ReLU after
    the selection), differentiable in x, w1 and w2."""

    @staticmethod
    def forward(ctx, x, w1, w2, topk: int, chunk: int):
        out, idx, dots = ffn(x, w1, w2, topk, chunk, cache=True)
        ctx.save_for_backward(x, w1, w2, idx, dots)
        return out

    @staticmethod
    def backward(ctx, d_out):
        x, w1, w2, idx, dots = ctx.saved_tensors
        dx, dw1, dw2 = ffn_backward(x, w1, w2, idx, dots, d_out.contiguous())
        return dx, dw1, dw2, None, None


def topk_attention(q, k, v, topk: int, chunk: int = 0, causal: bool = False, scale: float | None = None):
    """Differentiable top-k attention over contiguous [B, H, L, d] tensors."""
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    return TopkAttentionFunction.apply(q, k, v, int(topk), int(chunk), bool(causal), float(scale))


def dense_attention(q, k, v, chunk: int = 0, causal: bool = False, scale: float | None = None):
    """Query chunking with the top-k disabled (every valid key, Eq. 1): the paper's
    comparison baseline. Forward only (no backward is provided for it)."""
    if torch.is_grad_enabled() and (q.requires_grad or k.requires_grad or v.requires_grad):
        raise RuntimeError("dense_attention has no backward pass; call it under torch.no_grad()")
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    return attn_dense(q, k, v, int(chunk), bool(causal), float(scale))


def topk_feed_forward(x, w1, w2, topk: int, chunk: int = 0):
    """Differentiable top-k feed-forward layer: x [N, d_model], w1 / w2 [d_ff, d_model]."""
    return TopkFFNFunction.apply(x, w1, w2, int(topk), int(chunk))


class TopkMultiheadAttention(torch.nn.Module):
    """Multi-head self-attention whose heads use top-k attention: a drop-in for a
    BERT-style attention block on batch-first input x [B, L, d_model].

    [q | k | v] = x W_qkv^T + b_qkv, head h takes columns h*d_h .. (h+1)*d_h - 1 of
    each; every head runs top-k attention (temperature 1/sqrt(d_h) unless given);
    y = concat(heads) W_o^T + b_o. With topk=None the heads keep every key (query
    chunking without top-k, the paper's baseline; forward only)."""

    def __init__(self, d_model: int, n_heads: int, topk: int, chunk: int = 1024, causal: bool = False,
                 bias: bool = True, scale: float | None = None, device=None, dtype=torch.bfloat16):
        super().__init__()
        if d_model % n_heads:
            raise ValueError(f"d_model {d_model} is not a multiple of n_heads {n_heads}")
        self.d_model, self.n_heads, self.topk, self.chunk, self.causal = d_model, n_heads, topk, chunk, causal
        self.d_head = d_model // n_heads
        self.scale = 1.0 / math.sqrt(self.d_head) if scale is None else float(scale)
        kw = dict(device=device, dtype=dtype)
        self.qkv = torch.nn.Linear(d_model, 3 * d_model, bias=bias, **kw)
        self.out = torch.nn.Linear(d_model, d_model, bias=bias, **kw)

    def forward(self, x):
        B, L, D = x.shape
        p = self.qkv(x).view(B, L, 3, self.n_heads, self.d_head).permute(2, 0, 3, 1, 4)
        q, k, v = (p[t].contiguous() for t in range(3))
        if self.topk is None:
            o = dense_attention(q, k, v, self.chunk, self.causal, self.scale)
        else:
            o = topk_attention(q, k, v, self.topk, self.chunk, self.causal, self.scale)
        return self.out(o.permute(0, 2, 1, 3).reshape(B, L, D))


class TopkFeedForward(torch.nn.Module):
    """The feed-forward sub-layer cast as attention (Eq. 3): keys are the rows of w1,
    values the rows of w2 (both [d_ff, d_model]); each token keeps its top-k hidden
    units, ReLU after the selection. Input [..., d_model]."""

    def __init__(self, d_model: int, d_ff: int, topk: int, chunk: int = 1024, device=None,
                 dtype=torch.bfloat16):
        super().__init__()
        self.topk, self.chunk = topk, chunk
        kw = dict(device=device, dtype=dtype)
        self.w1 = torch.nn.Parameter(torch.empty(d_ff, d_model, **kw))
        self.w2 = torch.nn.Parameter(torch.empty(d_ff, d_model, **kw))
        torch.nn.init.normal_(self.w1, std=d_model ** -0.5)
        torch.nn.init.normal_(self.w2, std=d_ff ** -0.5)

    def forward(self, x):
        shape = x.shape
        y = topk_feed_forward(x.reshape(-1, shape[-1]).contiguous(), self.w1, self.w2, self.topk, self.chunk)
        return y.reshape(shape)
