"""fp64 CPU oracle of a multi-head attention layer whose heads use top-k attention
(Section 2.1, multi-head attention; Section 2.2, Eq. 4 per head), forward and
backward (the backward of each head by input checkpointing, Section 2.2).

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. It shares no code with
the HIP library or its Python binding.

The layer, for X [B, L, d_model] and H heads of size d_h = d_model / H:
  [Q | K | V] = X W_qkv^T + b_qkv            (W_qkv [3 d_model, d_model])
  head h takes columns h d_h .. (h + 1) d_h - 1 of each of Q, K, V;
  O_h = top-k attention(Q_h, K_h, V_h)        (Eq. 4, temperature `scale`)
  Y = concat_h(O_h) W_o^T + b_o               (W_o [d_model, d_model]).
The paper's formula has no biases; zero biases give it. Every input is upcast to
float64.
"""
from __future__ import annotations

import numpy as np

from oracle import topk_backward as bwd
from oracle import topk_oracle as fwd


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def split_heads(Y, H):
    """[B, L, H d_h] -> [B, H, L, d_h]."""
    B, L, D = Y.shape
    return Y.reshape(B, L, H, D // H).transpose(0, 2, 1, 3)


def merge_heads(O):
    """[B, H, L, d_h] -> [B, L, H d_h]."""
    B, H, L, dh = O.shape
    return O.transpose(0, 2, 1, 3).reshape(B, L, H * dh)


def projections(X, Wqkv, bqkv, H):
    """Q, K, V as [B, H, L, d_h] each."""
    X, Wqkv, bqkv = _f64(X), _f64(Wqkv), _f64(bqkv)
    dm = X.shape[-1]
    P = X @ Wqkv.T + bqkv
    return tuple(split_heads(P[..., t * dm:(t + 1) * dm], H) for t in range(3))


def mha_forward(X, Wqkv, bqkv, Wo, bo, H, k, chunk, causal, scale, top_idx=None, qkv=None):
    """Y [B, L, d_model] and the per-head index sets [B, H, L, k]. With ``top_idx``
    given, the heads use those index sets (scores recomputed in fp64) instead of
    selecting their own; with ``qkv`` given (three [B, H, L, d_h] arrays, e.g. the
    projections as a lower-precision GEMM rounded them), the heads attend over those."""
    Q, K, V = projections(X, Wqkv, bqkv, H) if qkv is None else tuple(_f64(t) for t in qkv)
    if top_idx is None:
        r = fwd.oracle_attn(Q, K, V, k, chunk, causal, scale)
        O, top_idx = r["out"], r["idx"]
    else:
        B, Hh, L, dh = Q.shape
        O = np.zeros_like(Q)
        for b in range(B):
            for h in range(Hh):
                O[b, h], _ = fwd.from_indices(Q[b, h], K[b, h], V[b, h], top_idx[b, h], "softmax", scale)
    Y = merge_heads(O) @ _f64(Wo).T + _f64(bo)
    return Y, top_idx


def mha_backward(X, Wqkv, bqkv, Wo, bo, H, top_idx, dY, scale, qkv=None):
    """Gradients (dX, dWqkv, dbqkv, dWo, dbo) of the layer for the index sets
    ``top_idx`` and the output gradient dY: the output projection's gradients, each
    head's backward by input checkpointing (oracle_attn_backward), then the
    projections' gradients. ``qkv`` as for mha_forward."""
    X, dY, Wqkv, Wo = _f64(X), _f64(dY), _f64(Wqkv), _f64(Wo)
    B, L, dm = X.shape
    Q, K, V = projections(X, Wqkv, bqkv, H) if qkv is None else tuple(_f64(t) for t in qkv)
    O = np.zeros_like(Q)
    for b in range(B):
        for h in range(H):
            O[b, h], _ = fwd.from_indices(Q[b, h], K[b, h], V[b, h], top_idx[b, h], "softmax", scale)
    Om = merge_heads(O)
    dWo = dY.reshape(-1, dm).T @ Om.reshape(-1, dm)
    dbo = dY.reshape(-1, dm).sum(axis=0)
    dO = split_heads(dY @ Wo, H)
    dQ, dK, dV = bwd.oracle_attn_backward(Q, K, V, top_idx, dO, scale)
    dP = np.concatenate([merge_heads(dQ), merge_heads(dK), merge_heads(dV)], axis=-1)  # [B, L, 3 d_model]
    dWqkv = dP.reshape(-1, 3 * dm).T @ X.reshape(-1, dm)
    dbqkv = dP.reshape(-1, 3 * dm).sum(axis=0)
    dX = dP @ Wqkv
    return dX, dWqkv, dbqkv, dWo, dbo
