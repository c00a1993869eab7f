"""Pins of the fp64 backward oracle against things other than itself.

Each ``pin_*`` takes the backward-oracle module and raises AssertionError when it
disagrees with central finite differences of the forward definition, with the
textbook dense gradients of Eq. 1 / Eq. 3 (the k = Lk fixed point), with the k = 1
closed form, or with chunk invariance. ``test_oracle_backward.py`` also runs them
against copies of the oracle with a planted mistake and checks that some pin fails.
"""
from __future__ import annotations

import math

import numpy as np

from oracle import topk_oracle as fwd


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _close(a, b, tol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


def _numeric_grad(f, arrays, h=1e-6):
    """Central differences of the scalar f(*arrays) w.r.t. every element of every array."""
    grads = []
    for a in arrays:
        g = np.zeros_like(a)
        it = np.nditer(a, flags=["multi_index"])
        for _ in it:
            ix = it.multi_index
            old = a[ix]
            a[ix] = old + h
            fp = f(*arrays)
            a[ix] = old - h
            fm = f(*arrays)
            a[ix] = old
            g[ix] = (fp - fm) / (2 * h)
        grads.append(g)
    return grads


def _attn_loss(idx, G, scale):
    # the forward on a FIXED index set, contracted with G: d(loss)/d(out) = G
    def f(Q, K, V):
        out, _ = fwd.from_indices(Q, K, V, idx, "softmax", scale)
        return float(np.sum(out * G))
    return f


def pin_bwd_attention_vs_finite_differences(bo):
    """Gradients w.r.t. Q, K, V equal central differences of the forward definition
    (index sets held fixed: no near-ties, so the selection is locally constant),
    with and without the causal mask."""
    rng = _rng(101)
    Lq, Lk, d, k = 6, 8, 4, 3
    scale = float(np.float32(0.7))
    for causal in (False, True):
        Q = rng.standard_normal((1, 1, Lq, d))
        K = rng.standard_normal((1, 1, Lk, d))
        V = rng.standard_normal((1, 1, Lk, d))
        G = rng.standard_normal((1, 1, Lq, d))
        r = fwd.oracle_attn(Q, K, V, k, 4, causal, scale)
        idx = r["idx"]
        has_next = np.isfinite(r["sigma_k1"])  # rows that have a (k+1)-th key
        assert np.all(r["sigma_k"][has_next] - r["sigma_k1"][has_next] > 1e-3), "near tie in pin data"
        dQ, dK, dV = bo.oracle_attn_backward(Q, K, V, idx, G, scale, chunk=4)
        q, kk, v = Q[0, 0].copy(), K[0, 0].copy(), V[0, 0].copy()
        nQ, nK, nV = _numeric_grad(_attn_loss(idx[0, 0], G[0, 0], scale), [q, kk, v])
        _close(dQ[0, 0], nQ, 1e-7, f"dQ vs finite differences (causal={causal})")
        _close(dK[0, 0], nK, 1e-7, f"dK vs finite differences (causal={causal})")
        _close(dV[0, 0], nV, 1e-7, f"dV vs finite differences (causal={causal})")


def pin_bwd_ffn_vs_finite_differences(bo):
    """Feed-forward gradients w.r.t. X, W1, W2 equal central differences of the
    forward definition; the selected sets include negative scores (ReLU gives them
    weight and gradient 0)."""
    rng = _rng(102)
    N, dm, dff, k = 5, 4, 9, 5
    X = rng.standard_normal((N, dm))
    W1 = rng.standard_normal((dff, dm))
    W2 = rng.standard_normal((dff, dm))
    G = rng.standard_normal((N, dm))
    r = fwd.oracle_ffn(X, W1, W2, k, 0)
    idx = r["idx"]
    top = fwd.selected_scores(X, W1, idx)
    assert np.any(top < -1e-3) and np.all(np.abs(top) > 1e-3), "pin data must select negative scores, none near 0"
    assert np.all(r["sigma_k"] - r["sigma_k1"] > 1e-3), "near tie in pin data"  # k < d_ff: every row has one

    def f(x, w1, w2):
        out, _ = fwd.from_indices(x, w1, w2, idx, "relu")
        return float(np.sum(out * G))

    dX, dW1, dW2 = bo.oracle_ffn_backward(X, W1, W2, idx, G)
    nX, n1, n2 = _numeric_grad(f, [X.copy(), W1.copy(), W2.copy()])
    _close(dX, nX, 1e-7, "dX vs finite differences")
    _close(dW1, n1, 1e-7, "dW1 vs finite differences")
    _close(dW2, n2, 1e-7, "dW2 vs finite differences")


def pin_bwd_full_k_is_dense_attention_gradient(bo):
    """k = Lk: the gradients are the textbook gradients of Eq. 1 written densely:
    P = softmax(scale S); dV = P^T G; dS = P * (G V^T - rowsum(P * G V^T)); dQ = scale dS K;
    dK = scale dS^T Q."""
    rng = _rng(103)
    L, d = 12, 5
    scale = float(np.float32(1 / math.sqrt(d)))
    Q, K, V, G = (rng.standard_normal((1, 1, L, d)) for _ in range(4))
    r = fwd.oracle_attn(Q, K, V, L, 5, False, scale)
    dQ, dK, dV = bo.oracle_attn_backward(Q, K, V, r["idx"], G, scale, chunk=5)
    q, kk, v, g = Q[0, 0], K[0, 0], V[0, 0], G[0, 0]
    S = q @ kk.T
    P = np.exp(scale * (S - S.max(axis=1, keepdims=True)))
    P /= P.sum(axis=1, keepdims=True)
    dP = g @ v.T
    dS = P * (dP - np.sum(dP * P, axis=1, keepdims=True))
    _close(dV[0, 0], P.T @ g, 1e-12, "dV (k = Lk)")
    _close(dQ[0, 0], scale * dS @ kk, 1e-12, "dQ (k = Lk)")
    _close(dK[0, 0], scale * dS.T @ q, 1e-12, "dK (k = Lk)")


def pin_bwd_full_k_is_dense_ffn_gradient(bo):
    """k = d_ff: the gradients of the dense ReLU feed-forward layer (Eq. 3):
    A = X W1^T, H = relu(A), out = H W2; dW2 = H^T G; dA = (G W2^T) * [A > 0];
    dX = dA W1; dW1 = dA^T X."""
    rng = _rng(104)
    N, dm, dff = 7, 4, 10
    X, G = rng.standard_normal((N, dm)), rng.standard_normal((N, dm))
    W1, W2 = rng.standard_normal((dff, dm)), rng.standard_normal((dff, dm))
    r = fwd.oracle_ffn(X, W1, W2, dff, 3)
    dX, dW1, dW2 = bo.oracle_ffn_backward(X, W1, W2, r["idx"], G, chunk=3)
    A = X @ W1.T
    Hh = np.maximum(A, 0.0)
    dA = (G @ W2.T) * (A > 0)
    _close(dW2, Hh.T @ G, 1e-12, "dW2 (k = d_ff)")
    _close(dX, dA @ W1, 1e-12, "dX (k = d_ff)")
    _close(dW1, dA.T @ X, 1e-12, "dW1 (k = d_ff)")


def pin_bwd_k1_closed_form(bo):
    """k = 1: the lone survivor has softmax weight 1 whatever its score, so d_Q = d_K = 0
    and d_V of key j is the sum of d_out over the rows that selected j."""
    rng = _rng(105)
    L, d = 9, 3
    Q, K, V, G = (rng.standard_normal((1, 1, L, d)) for _ in range(4))
    r = fwd.oracle_attn(Q, K, V, 1, 4, False, 0.5)
    dQ, dK, dV = bo.oracle_attn_backward(Q, K, V, r["idx"], G, 0.5, chunk=4)
    _close(dQ, np.zeros_like(dQ), 0.0, "dQ (k = 1)")
    _close(dK, np.zeros_like(dK), 0.0, "dK (k = 1)")
    ref = np.zeros((L, d))
    for i in range(L):
        ref[r["idx"][0, 0, i, 0]] += G[0, 0, i]
    _close(dV[0, 0], ref, 1e-15, "dV (k = 1)")


def pin_bwd_chunk_invariance_and_padding(bo):
    """The gradients do not depend on the chunk size; causal rows with fewer than k
    keys (-1 padded index sets) contribute only through their valid keys."""
    rng = _rng(106)
    B, H, L, d, k = 1, 2, 11, 4, 5
    Q, K, V, G = (rng.standard_normal((B, H, L, d)) for _ in range(4))
    r = fwd.oracle_attn(Q, K, V, k, 0, True, 0.6)
    assert np.any(r["idx"] < 0), "pin data must hold padded rows"
    ref = bo.oracle_attn_backward(Q, K, V, r["idx"], G, 0.6)
    for C in (1, 3, 7):
        got = bo.oracle_attn_backward(Q, K, V, r["idx"], G, 0.6, chunk=C)
        for a, b, n in zip(got, ref, ("dQ", "dK", "dV")):
            _close(a, b, 1e-12, f"{n} with chunk {C}")
    # keys j > i never receive gradient from causal row i: the last key only from the last row
    dQ, dK, dV = ref
    sel_last = np.any(r["idx"][0, :, :, :] == L - 1, axis=-1)
    assert sel_last[:, : L - 1].sum() == 0



def pin_bwd_sampled_equals_full(bo):
    """The sampled backward (per-row steps, then sums restricted to chosen rows and
    keys) equals the full chunked backward at those rows and keys, for the softmax
    (causal, with padded rows) and for ReLU."""
    rng = _rng(107)
    L, d, k = 40, 6, 5
    Q, K, V, G = (rng.standard_normal((1, 1, L, d)) for _ in range(4))
    r = fwd.oracle_attn(Q, K, V, k, 8, True, 0.4)
    full = bo.oracle_attn_backward(Q, K, V, r["idx"], G, 0.4, chunk=8)
    rows, keys = np.array([0, 3, 17, 39]), np.array([0, 1, 20, 39])
    got = bo.sampled_backward(Q[0, 0], K[0, 0], V[0, 0], r["idx"][0, 0], G[0, 0], rows, keys, "softmax", 0.4)
    _close(got[0], full[0][0, 0][rows], 1e-12, "sampled dQ")
    _close(got[1], full[1][0, 0][keys], 1e-12, "sampled dK")
    _close(got[2], full[2][0, 0][keys], 1e-12, "sampled dV")
    N, dff = 30, 50
    X, Gx = rng.standard_normal((N, d)), rng.standard_normal((N, d))
    W1, W2 = rng.standard_normal((dff, d)), rng.standard_normal((dff, d))
    rf = fwd.oracle_ffn(X, W1, W2, 7, 0)
    fullf = bo.oracle_ffn_backward(X, W1, W2, rf["idx"], Gx, chunk=9)
    rows, keys = np.array([1, 29]), np.arange(0, dff, 7)
    got = bo.sampled_backward(X, W1, W2, rf["idx"], Gx, rows, keys, "relu")
    _close(got[0], fullf[0][rows], 1e-12, "sampled dX")
    _close(got[1], fullf[1][keys], 1e-12, "sampled dW1")
    _close(got[2], fullf[2][keys], 1e-12, "sampled dW2")


def pin_bwd_magnitudes_bound_the_gradients(bo):
    """The sums of absolute terms bound the gradients elementwise (triangle inequality),
    equal them where every term has one sign (d_V with non-negative d_out: softmax
    weights are non-negative), and the sampled form returns the same sums."""
    rng = _rng(108)
    L, d, k = 30, 4, 5
    Q, K, V = (rng.standard_normal((1, 1, L, d)) for _ in range(3))
    G = np.abs(rng.standard_normal((1, 1, L, d)))
    r = fwd.oracle_attn(Q, K, V, k, 0, True, 0.5)
    grads, mags = bo.oracle_attn_backward(Q, K, V, r["idx"], G, 0.5, chunk=7, magnitudes=True)
    for gr, mg, n in zip(grads, mags, ("dQ", "dK", "dV")):
        assert np.all(np.abs(gr) <= mg + 1e-12), f"{n}: |gradient| above its magnitude"
    _close(grads[2], mags[2], 1e-12, "dV with d_out >= 0 equals its magnitude")
    assert np.any(mags[0] > np.abs(grads[0]) + 1e-6), "dQ terms of mixed sign must show in the magnitude"
    rows, keys = np.array([2, 17, 29]), np.array([0, 5, 28])
    sg, sm = bo.sampled_backward(Q[0, 0], K[0, 0], V[0, 0], r["idx"][0, 0], G[0, 0], rows, keys, "softmax", 0.5,
                                 magnitudes=True)
    _close(sm[0], mags[0][0, 0][rows], 1e-12, "sampled dQ magnitude")
    _close(sm[1], mags[1][0, 0][keys], 1e-12, "sampled dK magnitude")
    _close(sm[2], mags[2][0, 0][keys], 1e-12, "sampled dV magnitude")


ALL_PINS = [v for kname, v in sorted(globals().items()) if kname.startswith("pin_")]
