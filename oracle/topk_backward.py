"""fp64 CPU oracle of the gradients of top-k attention and of the top-k feed-forward
layer, with input checkpointing (Section 2.2, "Input checkpointing").

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The product path (the
HIP library and its Python binding) never calls it, and this module shares no
code with that path.

Input checkpointing keeps only the inputs and, per query row, the survivor set S_i
(the selected keys); everything else is recomputed. For fixed survivor sets the
output of a row is o_i = sum_{j in S_i} w_ij v_j with w_ij a function of the
survivors' scores s_ij = q_i . k_j, so the gradients follow from the chain rule.
With g_i = dL/do_i:

* dL/dv_j = sum over the rows i that selected j of w_ij g_i;
* a_ij = dL/dw_ij = g_i . v_j for every survivor;
* softmax weights (temperature ``scale``): dL/ds_ij = scale * w_ij * (a_ij - sum_{m in
  S_i} w_im a_im); ReLU weights: dL/ds_ij = a_ij if s_ij > 0, else 0 (0 at s = 0);
* dL/dq_i = sum_{j in S_i} dL/ds_ij k_j, and dL/dk_j = sum over the rows i that
  selected j of dL/ds_ij q_i.

The selection itself is piecewise constant in the inputs and carries no gradient.
Padding entries (index -1, causal rows with fewer than k valid keys) carry no weight
and no gradient; keys that no row selected get zero gradients. The feed-forward
layer is the same with X as the queries, W1 as the keys, W2 as the values, ReLU and
no temperature.

Every input is upcast exactly to float64.
"""
from __future__ import annotations

import numpy as np

from oracle.topk_oracle import selected_scores, weights


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def score_grads(top, a, valid, activation, scale):
    """Weights w [R, k] of the survivors (scores ``top``) and dL/ds [R, k], given
    a = dL/dw; both zero at padding entries."""
    if activation == "softmax":
        w = np.where(valid, weights(np.where(valid, top, -np.inf), "softmax", scale), 0.0)
        a = np.where(valid, a, 0.0)
        mean = np.sum(w * a, axis=1, keepdims=True)
        ds = np.float64(np.float32(scale)) * w * (a - mean)
    elif activation == "relu":
        s = np.where(valid, top, 0.0)
        w = np.where(valid, np.maximum(s, 0.0), 0.0)
        ds = np.where(valid & (s > 0), a, 0.0)
    else:
        raise ValueError(activation)
    return w, np.where(valid, ds, 0.0)


def row_terms(Qr, K, V, idx, G, activation, scale=1.0):
    """Per-survivor terms of rows Qr [R, d] with survivor sets idx [R, k] and output
    gradients G [R, dv]: the weights w and dL/ds, each [R, k], from fp64 scores."""
    valid = idx >= 0
    safe = np.where(valid, idx, 0)
    a = np.where(valid, np.einsum("rt,rmt->rm", _f64(G), _f64(V)[safe]), 0.0)
    return score_grads(selected_scores(Qr, K, idx), a, valid, activation, scale)


def row_term_magnitudes(Qr, K, V, idx, G, activation, scale=1.0):
    """Per-survivor bounds |dL/ds| <= b of rows Qr [R, d], [R, k]: the chain of
    row_terms with every sum taken over absolute values (a_ij replaced by
    sum_t |g_it| |v_jt|, the softmax centring by a sum of absolute terms)."""
    valid = idx >= 0
    safe = np.where(valid, idx, 0)
    a_abs = np.where(valid, np.einsum("rt,rmt->rm", np.abs(_f64(G)), np.abs(_f64(V)[safe])), 0.0)
    top = selected_scores(Qr, K, idx)
    if activation == "softmax":
        w = np.where(valid, weights(np.where(valid, top, -np.inf), "softmax", scale), 0.0)
        mean = np.sum(w * a_abs, axis=1, keepdims=True)
        b = np.float64(np.float32(scale)) * w * (a_abs + mean)
    else:
        b = np.where(valid & (np.where(valid, top, 0.0) > 0), a_abs, 0.0)
    return np.where(valid, b, 0.0)


def head_backward(Qh, Kh, Vh, idx, G, activation, scale=1.0, chunk=None, magnitudes=False):
    """Gradients of one head (Q [Lq, d], K and V [Lk, *], survivor sets idx [Lq, k],
    output gradients G [Lq, dv]), ``chunk`` rows at a time. Returns fp64
    (dQ [Lq, d], dK [Lk, d], dV [Lk, dv]).

    With ``magnitudes`` it also returns the same sums taken over the absolute values of
    their terms, with the per-survivor bound b of row_term_magnitudes in place of
    dL/ds (sum b |k|, sum b |q|, sum |w| |g|): the scale against which rounding in sums
    of terms of mixed signs is judged."""
    Qh, Kh, Vh, G = _f64(Qh), _f64(Kh), _f64(Vh), _f64(G)
    Lq = Qh.shape[0]
    C = Lq if not chunk else int(chunk)
    dQ = np.zeros_like(Qh)
    dK = np.zeros_like(Kh)
    dV = np.zeros_like(Vh)
    mags = (np.zeros_like(Qh), np.zeros_like(Kh), np.zeros_like(Vh)) if magnitudes else None
    for c0 in range(0, Lq, C):
        r = np.arange(c0, min(c0 + C, Lq))
        w, ds = row_terms(Qh[r], Kh, Vh, idx[r], G[r], activation, scale)
        valid = idx[r] >= 0
        safe = np.where(valid, idx[r], 0)
        dQ[r] = np.einsum("rm,rmt->rt", ds, Kh[safe])
        rr, mm = np.nonzero(valid)
        np.add.at(dK, idx[r][rr, mm], ds[rr, mm, None] * Qh[r][rr])
        np.add.at(dV, idx[r][rr, mm], w[rr, mm, None] * G[r][rr])
        if magnitudes:
            bnd = row_term_magnitudes(Qh[r], Kh, Vh, idx[r], G[r], activation, scale)
            mags[0][r] = np.einsum("rm,rmt->rt", bnd, np.abs(Kh[safe]))
            np.add.at(mags[1], idx[r][rr, mm], bnd[rr, mm, None] * np.abs(Qh[r][rr]))
            np.add.at(mags[2], idx[r][rr, mm], np.abs(w[rr, mm, None] * G[r][rr]))
    return ((dQ, dK, dV), mags) if magnitudes else (dQ, dK, dV)


def oracle_attn_backward(Q, K, V, top_idx, d_out, scale, chunk=None, magnitudes=False):
    """Gradients of top-k attention over [B, H, L, d] inputs for the survivor sets
    top_idx [B, H, Lq, k]. Returns fp64 (d_Q, d_K, d_V) shaped like Q, K, V (and, with
    ``magnitudes``, their sums of absolute terms, see head_backward)."""
    B, H = Q.shape[:2]
    out = [np.zeros(Q.shape), np.zeros(K.shape), np.zeros(V.shape)]
    mags = [np.zeros(Q.shape), np.zeros(K.shape), np.zeros(V.shape)]
    for b in range(B):
        for h in range(H):
            r = head_backward(Q[b, h], K[b, h], V[b, h], top_idx[b, h], d_out[b, h], "softmax", scale, chunk,
                              magnitudes)
            grads, m = r if magnitudes else (r, None)
            for t in range(3):
                out[t][b, h] = grads[t]
                if magnitudes:
                    mags[t][b, h] = m[t]
    return (tuple(out), tuple(mags)) if magnitudes else tuple(out)


def oracle_ffn_backward(X, W1, W2, top_idx, d_out, chunk=None, magnitudes=False):
    """Gradients of the top-k feed-forward layer (keys W1, values W2, ReLU) for the
    survivor sets top_idx [N, k]. Returns fp64 (d_X [N, dm], d_W1, d_W2 [dff, dm])
    (and, with ``magnitudes``, their sums of absolute terms)."""
    return head_backward(X, W1, W2, top_idx, d_out, "relu", 1.0, chunk, magnitudes)


def sampled_backward(Q, K, V, top_idx, d_out, rows, keys, activation, scale=1.0, batch=64, magnitudes=False):
    """The gradients of one head at chosen rows and keys, for checks at sizes where a
    whole head is too slow: Q [Lq, d], K and V [Lk, *], top_idx [Lq, k], d_out [Lq, dv].

    dQ at the chosen rows; dK and dV at the chosen keys, summed over every row that
    selected them. Rows go through the per-survivor terms ``batch`` at a time.
    Returns fp64 (d_Q [len(rows), d], d_K [len(keys), d], d_V [len(keys), dv]), keys
    in increasing order (and, with ``magnitudes``, their sums of absolute terms)."""
    rows = np.asarray(rows, dtype=np.int64)
    keys = np.unique(np.asarray(keys, dtype=np.int64))
    k, d = top_idx.shape[1], Q.shape[1]
    dQ = np.zeros((len(rows), d))
    aQ = np.zeros((len(rows), d))
    for b0 in range(0, len(rows), batch):
        rb = rows[b0:b0 + batch]
        _, ds = row_terms(Q[rb], K, V, top_idx[rb], d_out[rb], activation, scale)
        safe = np.where(top_idx[rb] >= 0, top_idx[rb], 0)
        dQ[b0:b0 + batch] = np.einsum("rm,rmt->rt", ds, _f64(K[safe]))
        if magnitudes:
            bnd = row_term_magnitudes(Q[rb], K, V, top_idx[rb], d_out[rb], activation, scale)
            aQ[b0:b0 + batch] = np.einsum("rm,rmt->rt", bnd, np.abs(_f64(K[safe])))
    chose = np.unique(np.flatnonzero(np.isin(top_idx.ravel(), keys)) // k)  # rows that selected a chosen key
    dK = np.zeros((len(keys), d))
    dV = np.zeros((len(keys), V.shape[1]))
    aK = np.zeros_like(dK)
    aV = np.zeros_like(dV)
    for b0 in range(0, len(chose), batch):
        rb = chose[b0:b0 + batch]
        w, ds = row_terms(Q[rb], K, V, top_idx[rb], d_out[rb], activation, scale)
        a, m = np.nonzero(np.isin(top_idx[rb], keys))
        n = np.searchsorted(keys, top_idx[rb][a, m])
        tk_ = ds[a, m, None] * _f64(Q[rb][a])
        tv_ = w[a, m, None] * _f64(d_out[rb][a])
        np.add.at(dK, n, tk_)
        np.add.at(dV, n, tv_)
        if magnitudes:
            bnd = row_term_magnitudes(Q[rb], K, V, top_idx[rb], d_out[rb], activation, scale)
            np.add.at(aK, n, bnd[a, m, None] * np.abs(_f64(Q[rb][a])))
            np.add.at(aV, n, np.abs(tv_))
    return ((dQ, dK, dV), (aQ, aK, aV)) if magnitudes else (dQ, dK, dV)
