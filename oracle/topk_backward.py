"""fp64 CPU oracle of the backward pass of top-k attention and of the top-k
feed-forward layer, with input checkpointing (Section 2.2, "Input checkpointing",
and the backward pseudo-code that follows it).

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The product path (the
HIP library and its Python binding) never calls it, and this module shares no
code with that path.

The forward pass caches only its inputs and, per query row, the selected keys
(``top_indices``) and their raw scores (``top_dots``). Given the gradient of the
loss with respect to the output (``d_out``), the backward pass of one query chunk
takes these steps, in the paper's order:

1. ``d_top_actv[r, m] = d_out[r] . V[top_indices[r, m]]`` -- the value-row dot
   products at the selected positions only;
2. ``top_actv = activation(top_dots)``, recomputed: the softmax with temperature
   over the survivors (Eq. 1, Eq. 4), or ReLU (Eq. 3);
3. ``d_top_dots``: the activation backpropagated on the ``[C, k]`` survivors. For
   the softmax ``w = softmax(scale * s)``: ``scale * w * (g - sum_m w_m g_m)``;
   for ReLU: ``g * [s > 0]`` (zero at s = 0);
4. ``actv = matrix(top_actv, top_indices)``; ``d_V = actv^T d_out``;
5. ``d_dots = matrix(d_top_dots, top_indices)``; ``d_Q = d_dots K``;
   ``d_K = d_dots^T Q``.

Padding entries (index -1, rows with fewer than k valid keys) carry no weight and no
gradient. Keys and values shared by several chunks accumulate their gradients over
the chunks. The feed-forward layer is the same with X as the queries, W1 as the
keys, W2 as the values, ReLU, and no temperature.

Every input is upcast exactly to float64.
"""
from __future__ import annotations

import numpy as np

from oracle import topk_oracle as fwd


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def selected_dots(Qc: np.ndarray, K: np.ndarray, top_idx: np.ndarray) -> np.ndarray:
    """Raw scores q_r . K[top_idx[r, m]] in fp64 (what the forward caches as top_dots);
    -inf at padding entries."""
    Qc, K = _f64(Qc), _f64(K)
    safe = np.where(top_idx >= 0, top_idx, 0)
    d = np.einsum("rt,rmt->rm", Qc, K[safe])
    return np.where(top_idx >= 0, d, -np.inf)


def activation_backward(top_dots: np.ndarray, d_top_actv: np.ndarray, valid: np.ndarray, activation: str,
                        scale: float):
    """Steps 2-3: recompute the survivors' activation and backpropagate through it.
    Returns (top_actv, d_top_dots), both [R, k], zero at padding entries."""
    if activation == "softmax":
        w = fwd.softmax_over_survivors(np.where(valid, top_dots, -np.inf), scale)
        w = np.where(valid, w, 0.0)
        g = np.where(valid, d_top_actv, 0.0)
        inner = np.sum(w * g, axis=1, keepdims=True)
        d = np.float64(np.float32(scale)) * w * (g - inner)
    elif activation == "relu":
        s = np.where(valid, top_dots, 0.0)
        w = np.where(valid, np.maximum(s, 0.0), 0.0)
        d = np.where(valid & (s > 0), d_top_actv, 0.0)
    else:
        raise ValueError(activation)
    return w, np.where(valid, d, 0.0)


def chunk_backward(Qc, K, V, top_idx, d_out, activation, scale=1.0, top_dots=None):
    """Backward pass of one query chunk (Section 2.2 backward pseudo-code).

    Qc [C, d], K and V [Lk, d], top_idx [C, k] (-1 pads), d_out [C, d]. top_dots
    defaults to the exact fp64 scores of the selected keys. Returns
    (d_Qc [C, d], d_K [Lk, d], d_V [Lk, d])."""
    Qc, K, V, d_out = _f64(Qc), _f64(K), _f64(V), _f64(d_out)
    Lk = K.shape[0]
    valid = top_idx >= 0
    if top_dots is None:
        top_dots = selected_dots(Qc, K, top_idx)
    safe = np.where(valid, top_idx, 0)
    # 1. value-row dot products at the selected positions
    d_top_actv = np.where(valid, np.einsum("rt,rmt->rm", d_out, V[safe]), 0.0)
    # 2-3. recompute the activation and backpropagate through it
    top_actv, d_top_dots = activation_backward(_f64(top_dots), d_top_actv, valid, activation, scale)
    # 4. d_V = actv^T d_out
    actv = fwd.scatter_dense(top_actv, top_idx, Lk)
    d_V = actv.T @ d_out
    # 5. d_Q = d_dots K, d_K = d_dots^T Q
    d_dots = fwd.scatter_dense(d_top_dots, top_idx, Lk)
    d_Q = d_dots @ K
    d_K = d_dots.T @ Qc
    return d_Q, d_K, d_V


def oracle_attn_backward(Q, K, V, top_idx, d_out, scale, chunk=None):
    """Gradients of top-k attention over [B, H, L, d] inputs for the index sets
    top_idx [B, H, Lq, k], chunk by chunk (input checkpointing). Returns fp64
    (d_Q [B, H, Lq, d], d_K [B, H, Lk, d], d_V [B, H, Lk, d])."""
    Q, K, V, d_out = _f64(Q), _f64(K), _f64(V), _f64(d_out)
    B, H, Lq, d = Q.shape
    C = Lq if not chunk else chunk
    dQ = np.zeros_like(Q)
    dK = np.zeros_like(K)
    dV = np.zeros_like(V)
    for b in range(B):
        for h in range(H):
            for c0 in range(0, Lq, C):
                c1 = min(c0 + C, Lq)
                gq, gk, gv = chunk_backward(Q[b, h, c0:c1], K[b, h], V[b, h], top_idx[b, h, c0:c1],
                                            d_out[b, h, c0:c1], "softmax", scale)
                dQ[b, h, c0:c1] = gq
                dK[b, h] += gk
                dV[b, h] += gv
    return dQ, dK, dV


def oracle_ffn_backward(X, W1, W2, top_idx, d_out, chunk=None):
    """Gradients of the top-k feed-forward layer (keys W1, values W2, ReLU) for the
    index sets top_idx [N, k]. Returns fp64 (d_X [N, dm], d_W1 [dff, dm], d_W2 [dff, dm])."""
    X, W1, W2, d_out = _f64(X), _f64(W1), _f64(W2), _f64(d_out)
    N = X.shape[0]
    C = N if not chunk else chunk
    dX = np.zeros_like(X)
    dW1 = np.zeros_like(W1)
    dW2 = np.zeros_like(W2)
    for c0 in range(0, N, C):
        c1 = min(c0 + C, N)
        gx, g1, g2 = chunk_backward(X[c0:c1], W1, W2, top_idx[c0:c1], d_out[c0:c1], "relu")
        dX[c0:c1] = gx
        dW1 += g1
        dW2 += g2
    return dX, dW1, dW2


def row_terms(Qr, K, V, top_idx_r, d_out_r, activation, scale=1.0):
    """Steps 1-3 for a set of rows: (top_actv, d_top_dots), each [R, k], from the
    rows' queries Qr [R, d], index sets top_idx_r [R, k] and output gradients d_out_r."""
    Qr, d_out_r = _f64(Qr), _f64(d_out_r)
    valid = top_idx_r >= 0
    safe = np.where(valid, top_idx_r, 0)
    top_dots = selected_dots(Qr, K, top_idx_r)
    d_top_actv = np.where(valid, np.einsum("rt,rmt->rm", d_out_r, _f64(V[safe])), 0.0)
    return activation_backward(top_dots, d_top_actv, valid, activation, scale)


def sampled_backward(Q, K, V, top_idx, d_out, rows, keys, activation, scale=1.0, batch=64):
    """The gradients of one head at a sample of rows and keys, for checks at sizes
    where the dense [Lq, Lk] matrices of chunk_backward do not fit: Q [Lq, d],
    K and V [Lk, d], top_idx [Lq, k], d_out [Lq, d].

    Step 5 restricted to rows: d_Q[r] = sum_m d_top_dots[r, m] K[top_idx[r, m]];
    steps 4-5 restricted to keys: d_K[j] = sum over the (r, m) with top_idx[r, m] = j
    of d_top_dots[r, m] Q[r], and d_V[j] the same with top_actv[r, m] d_out[r]. Rows
    go through steps 1-3 `batch` at a time. Returns fp64 (d_Q [len(rows), d],
    d_K [len(keys), d], d_V [len(keys), d]), keys taken in increasing order."""
    rows = np.asarray(rows, dtype=np.int64)
    keys = np.unique(np.asarray(keys, dtype=np.int64))
    k, d = top_idx.shape[1], Q.shape[1]
    dQ = np.zeros((len(rows), d))
    for b0 in range(0, len(rows), batch):
        rb = rows[b0:b0 + batch]
        _, dd = row_terms(Q[rb], K, V, top_idx[rb], d_out[rb], activation, scale)
        safe = np.where(top_idx[rb] >= 0, top_idx[rb], 0)
        dQ[b0:b0 + batch] = np.einsum("rm,rmt->rt", dd, _f64(K[safe]))
    sel_rows = np.unique(np.flatnonzero(np.isin(top_idx.ravel(), keys)) // k)  # rows that chose a sampled key
    dK = np.zeros((len(keys), d))
    dV = np.zeros((len(keys), d))
    for b0 in range(0, len(sel_rows), batch):
        rb = sel_rows[b0:b0 + batch]
        actv, dd = row_terms(Q[rb], K, V, top_idx[rb], d_out[rb], activation, scale)
        a, m = np.nonzero(np.isin(top_idx[rb], keys))
        n = np.searchsorted(keys, top_idx[rb][a, m])
        np.add.at(dK, n, dd[a, m, None] * _f64(Q[rb][a]))
        np.add.at(dV, n, actv[a, m, None] * _f64(d_out[rb][a]))
    return dQ, dK, dV
