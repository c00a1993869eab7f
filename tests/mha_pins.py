"""Pins of the multi-head layer oracle against things other than itself: central
finite differences of the layer with the index sets held fixed, and, at k = L, the
textbook dense multi-head attention (projections, softmax attention per head,
output projection) written out with explicit per-head loops."""
from __future__ import annotations

import math

import numpy as np

from oracle import topk_oracle as fwd


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _close(a, b, tol, what):
    err = float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


def _weights(rng, dm, scale_w=0.4):
    return (scale_w * rng.standard_normal((3 * dm, dm)), 0.1 * rng.standard_normal(3 * dm),
            scale_w * rng.standard_normal((dm, dm)), 0.1 * rng.standard_normal(dm))


def pin_mha_dense_at_full_k(mo):
    """k = L: the layer equals dense multi-head attention (Section 2.1) computed with
    per-head loops over explicit projection column blocks."""
    rng = _rng(201)
    B, L, H, dh = 2, 7, 3, 4
    dm = H * dh
    X = rng.standard_normal((B, L, dm))
    Wqkv, bqkv, Wo, bo = _weights(rng, dm)
    scale = 1 / math.sqrt(dh)
    Y, _ = mo.mha_forward(X, Wqkv, bqkv, Wo, bo, H, L, 3, False, scale)
    ref = np.zeros((B, L, dm))
    for b in range(B):
        heads = []
        for h in range(H):
            cols = slice(h * dh, (h + 1) * dh)
            q = X[b] @ Wqkv[0 * dm:1 * dm][cols].T + bqkv[0 * dm:1 * dm][cols]
            k = X[b] @ Wqkv[1 * dm:2 * dm][cols].T + bqkv[1 * dm:2 * dm][cols]
            v = X[b] @ Wqkv[2 * dm:3 * dm][cols].T + bqkv[2 * dm:3 * dm][cols]
            s = scale * (q @ k.T)
            p = np.exp(s - s.max(axis=1, keepdims=True))
            p /= p.sum(axis=1, keepdims=True)
            heads.append(p @ v)
        ref[b] = np.concatenate(heads, axis=1) @ Wo.T + bo
    _close(Y, ref, 1e-12, "layer at k = L vs dense multi-head attention")


def pin_mha_backward_finite_differences(mo):
    """The layer's gradients (input, both weights, both biases) equal central
    differences of its forward with the index sets held fixed (causal, k < L, no
    near ties in the pin data)."""
    rng = _rng(202)
    B, L, H, dh, k = 1, 6, 2, 3, 3
    dm = H * dh
    X = rng.standard_normal((B, L, dm))
    Wqkv, bqkv, Wo, bo = _weights(rng, dm)
    G = rng.standard_normal((B, L, dm))
    scale = 0.6
    Y, idx = mo.mha_forward(X, Wqkv, bqkv, Wo, bo, H, k, 2, True, scale)
    Q, K, V = mo.projections(X, Wqkv, bqkv, H)
    for b in range(B):
        for h in range(H):
            r = fwd.oracle_attn(Q[b:b + 1, h:h + 1], K[b:b + 1, h:h + 1], V[b:b + 1, h:h + 1], k, 0, True, scale)
            has_next = np.isfinite(r["sigma_k1"])
            assert np.all(r["sigma_k"][has_next] - r["sigma_k1"][has_next] > 1e-3), "near tie in pin data"
    grads = mo.mha_backward(X, Wqkv, bqkv, Wo, bo, H, idx, G, scale)
    params = [X, Wqkv, bqkv, Wo, bo]

    def loss():
        y, _ = mo.mha_forward(*params[:5], H, k, 2, True, scale, top_idx=idx)
        return float(np.sum(y * G))

    h = 1e-6
    for n, (p, g) in enumerate(zip(params, grads)):
        num = np.zeros_like(p)
        it = np.nditer(p, flags=["multi_index"])
        for _ in it:
            ix = it.multi_index
            old = p[ix]
            p[ix] = old + h
            fp = loss()
            p[ix] = old - h
            fm = loss()
            p[ix] = old
            num[ix] = (fp - fm) / (2 * h)
        _close(g, num, 1e-6, f"gradient {('dX', 'dWqkv', 'dbqkv', 'dWo', 'dbo')[n]} vs finite differences")


ALL_PINS = [v for kname, v in sorted(globals().items()) if kname.startswith("pin_")]
