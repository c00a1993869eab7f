"""Pins of the fp64 oracle against things other than itself.

Each ``pin_*`` function takes the oracle module and raises AssertionError when the
oracle disagrees with brute force, a closed form, or an invariant fixed by the paper.
They are plain functions so that ``test_oracle.py`` can also run them against
copies of the oracle with a planted mistake and check that some pin fails.
"""
from __future__ import annotations

import math

import numpy as np

from oracle import brute


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _close(a, b, tol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


# ---------------------------------------------------------------- scores (Eq. 4, Eq. 2)
def pin_scores_vs_loops(o):
    """Chunk score tile vs explicit loops, with and without the causal mask."""
    rng = _rng(11)
    Q = rng.standard_normal((6, 5))
    K = rng.standard_normal((9, 5))
    for causal, row0 in ((False, 0), (True, 0), (True, 2)):
        got = o.scores(Q, K, o.valid_lengths(row0 + np.arange(6), 9, causal))
        ref = brute.scores(Q.tolist(), K.tolist(), causal, rows=range(row0, row0 + 6))
        for r in range(6):
            for j in range(9):
                if ref[r][j] is None:
                    assert got[r, j] == -np.inf, f"masked entry ({r},{j}) not -inf"
                else:
                    assert abs(got[r, j] - ref[r][j]) <= 1e-12, f"score ({r},{j})"


# ---------------------------------------------------------------- selection (Eq. 4)
def _tie_rows(rng, R, Lk):
    # small integers -> many exact ties, including at the k-th place
    return rng.integers(-3, 4, size=(R, Lk)).astype(np.float64)


def pin_selection_vs_subsets(o):
    """Row-wise top-k == the unique k-subset preceding all others, every k, with ties."""
    rng = _rng(12)
    for Lk in (1, 2, 5, 8):
        S = _tie_rows(rng, 6, Lk)
        for causal in (False, True):
            dots = S.copy()
            if causal:
                for r in range(dots.shape[0]):
                    dots[r, r + 1:] = -np.inf
            for k in range(1, Lk + 1):
                idx, top, k_eff, sk, sk1 = o.select(dots.copy(), k)
                for r in range(dots.shape[0]):
                    row = [None if not np.isfinite(v) else float(v) for v in dots[r]]
                    want = brute.topk_subset(row, k)
                    got = idx[r][idx[r] >= 0]
                    assert sorted(got.tolist()) == want, f"Lk={Lk} k={k} causal={causal} row {r}"
                    assert k_eff[r] == len(want)
                    # order (score desc, index asc) and the reported scores
                    order = sorted(want, key=lambda j: (-row[j], j))
                    assert got.tolist() == order, f"order Lk={Lk} k={k} row {r}"
                    assert np.all(top[r][:len(want)] == [row[j] for j in order])
                    assert sk[r] == row[order[-1]]
                    rest = sorted((j for j in range(Lk) if row[j] is not None and j not in want),
                                  key=lambda j: (-row[j], j))
                    if rest:
                        assert sk1[r] == row[rest[0]], "sigma_k+1"
                    else:
                        assert np.isnan(sk1[r]), "sigma_k+1 must be NaN when all keys are kept"


def pin_k1_is_argmax_row(o):
    """k = 1: softmax of a single survivor is exactly 1, so out = V[argmax] (ties -> low j)."""
    rng = _rng(13)
    Q = rng.integers(-2, 3, size=(16, 3)).astype(np.float64)
    K = rng.integers(-2, 3, size=(7, 3)).astype(np.float64)
    V = rng.standard_normal((7, 4))
    r = o.topk_rows(Q, K, V, 1, np.full(16, 7), "softmax", scale=0.37)
    S = Q @ K.T
    for i in range(16):
        j = int(np.flatnonzero(S[i] == S[i].max())[0])
        assert r["idx"][i, 0] == j
        assert np.array_equal(r["out"][i], V[j]), "k=1 must return the value row exactly"


# ---------------------------------------------------------------- softmax + sum (Eq. 1, 2, 4)
def _vanilla(Q, K, V, scale, causal=False):
    """Eq. 1 / Eq. 2 written independently: row-softmax(scale * QK^T + B) V."""
    out = np.zeros((Q.shape[0], V.shape[1]))
    for i in range(Q.shape[0]):
        n = i + 1 if causal else K.shape[0]
        logits = np.array([scale * float(Q[i] @ K[j]) for j in range(n)])
        p = np.exp(logits - logits.max())
        p /= p.sum()
        out[i] = p @ V[:n]
    return out


def pin_full_k_is_vanilla_attention(o):
    """k = Lk: top-k attention is exactly Eq. 1 (to 1e-6, in fact to rounding)."""
    rng = _rng(14)
    B, H, L, d = 1, 2, 40, 8
    Q = rng.standard_normal((B, H, L, d))
    K = rng.standard_normal((B, H, L, d))
    V = rng.standard_normal((B, H, L, d))
    scale = float(np.float32(1 / math.sqrt(d)))
    r = o.oracle_attn(Q, K, V, L, 16, False, scale)
    for h in range(H):
        _close(r["out"][0, h], _vanilla(Q[0, h], K[0, h], V[0, h], scale), 1e-6, "k=Lk vs Eq. 1")
        _close(r["out"][0, h], _vanilla(Q[0, h], K[0, h], V[0, h], scale), 1e-12, "k=Lk vs Eq. 1 (fp64)")


def pin_causal_short_rows_are_vanilla_causal(o):
    """Causal rows i < k keep all i+1 valid keys: equal to Eq. 2 with the causal mask."""
    rng = _rng(15)
    L, d, k = 24, 6, 10
    Q, K, V = (rng.standard_normal((1, 1, L, d)) for _ in range(3))
    r = o.oracle_attn(Q, K, V, k, 5, True, 0.5)
    ref = _vanilla(Q[0, 0], K[0, 0], V[0, 0], 0.5, causal=True)
    _close(r["out"][0, 0, :k], ref[:k], 1e-12, "causal rows < k vs Eq. 2")
    assert np.all(r["k_eff"][0, 0] == np.minimum(k, np.arange(L) + 1))
    assert np.all(r["idx"][0, 0, 0, 1:] == -1)


def pin_brute_force_attention(o):
    """Whole forward pass vs the brute-force loops (softmax, causal or not, ties)."""
    rng = _rng(16)
    sc = float(np.float32(0.7))        # the oracle uses the float32 value of the temperature
    for causal in (False, True):
        for k in (1, 2, 3, 5, 6):
            Q = rng.integers(-2, 3, size=(6, 3)).astype(np.float64)
            K = rng.integers(-2, 3, size=(6, 3)).astype(np.float64)
            V = rng.standard_normal((6, 4))
            want, subs = brute.attention(Q.tolist(), K.tolist(), V.tolist(), k, sc, causal)
            got = o.oracle_attn(Q[None, None], K[None, None], V[None, None], k, 4, causal, sc)
            _close(got["out"][0, 0], want, 1e-12, f"brute attention k={k} causal={causal}")
            for i, sub in enumerate(subs):
                g = got["idx"][0, 0, i]
                assert sorted(g[g >= 0].tolist()) == sub


# ---------------------------------------------------------------- feed-forward (Eq. 3 + Eq. 4)
def pin_ffn_full_k_is_dense_relu_ffn(o):
    """k = d_ff: the top-k FFN is the plain ReLU(X W1^T) W2 of Eq. 3."""
    rng = _rng(17)
    X = rng.standard_normal((20, 8))
    W1 = rng.standard_normal((30, 8))
    W2 = rng.standard_normal((30, 8))
    r = o.oracle_ffn(X, W1, W2, 30, 7)
    dense = np.zeros((20, 8))
    for i in range(20):
        for j in range(30):
            h = max(float(X[i] @ W1[j]), 0.0)
            dense[i] += h * W2[j]
    _close(r["out"], dense, 1e-12, "k=d_ff vs Eq. 3")


def pin_ffn_brute_and_k1(o):
    """FFN vs brute force (ReLU after selection) and the k = 1 closed form."""
    rng = _rng(18)
    X = rng.integers(-2, 3, size=(9, 3)).astype(np.float64)
    W1 = rng.integers(-2, 3, size=(7, 3)).astype(np.float64)
    W2 = rng.standard_normal((7, 5))
    for k in (1, 2, 4, 7):
        want, subs = brute.attention(X.tolist(), W1.tolist(), W2.tolist(), k, 1.0, False, "relu")
        got = o.oracle_ffn(X, W1, W2, k, 4)
        _close(got["out"], want, 1e-12, f"brute ffn k={k}")
        for i, sub in enumerate(subs):
            assert sorted(got["idx"][i].tolist()) == sub
    S = X @ W1.T
    got = o.oracle_ffn(X, W1, W2, 1, 0)
    for i in range(9):
        j = int(np.flatnonzero(S[i] == S[i].max())[0])
        _close(got["out"][i], max(S[i, j], 0.0) * W2[j], 1e-12, "ffn k=1")


def pin_ffn_homogeneity(o):
    """ReLU is positively homogeneous: out(2X) = 2 out(X), same selected set."""
    rng = _rng(19)
    X = rng.standard_normal((12, 6))
    W1 = rng.standard_normal((25, 6))
    W2 = rng.standard_normal((25, 6))
    a = o.oracle_ffn(X, W1, W2, 5, 0)
    b = o.oracle_ffn(2 * X, W1, W2, 5, 0)
    assert np.array_equal(a["idx"], b["idx"])
    _close(b["out"], 2 * a["out"], 1e-12, "homogeneity")


# ---------------------------------------------------------------- invariants (Section 2.2)
def pin_chunk_invariance(o):
    """Query chunking does not change the function: same sets, same outputs, any C."""
    rng = _rng(20)
    L, d = 48, 8
    Q, K, V = (rng.standard_normal((2, 1, L, d)) for _ in range(3))
    for causal in (False, True):
        ref = o.oracle_attn(Q, K, V, 6, L, causal, 0.3)
        for C in (1, 7, 16, L):
            r = o.oracle_attn(Q, K, V, 6, C, causal, 0.3)
            assert np.array_equal(r["idx"], ref["idx"]), f"chunk {C}"
            _close(r["out"], ref["out"], 1e-12, f"chunk {C}")


def pin_permutation_equivariance(o):
    """Keys are an unordered set: permuting K and V rows together permutes the indices
    and leaves the output unchanged; permuting queries permutes the output rows."""
    rng = _rng(21)
    L, d, k = 40, 6, 7
    Q, K, V = (rng.standard_normal((1, 1, L, d)) for _ in range(3))
    base = o.oracle_attn(Q, K, V, k, 0, False, 0.4)
    perm = rng.permutation(L)
    inv = np.argsort(perm)
    r = o.oracle_attn(Q, K[:, :, perm], V[:, :, perm], k, 0, False, 0.4)
    _close(r["out"], base["out"], 1e-12, "key permutation")
    assert np.array_equal(np.sort(perm[r["idx"][0, 0]], axis=1), np.sort(base["idx"][0, 0], axis=1))
    qp = rng.permutation(L)
    r2 = o.oracle_attn(Q[:, :, qp], K, V, k, 0, False, 0.4)
    _close(r2["out"][0, 0], base["out"][0, 0][qp], 1e-12, "query permutation")
    del inv


def pin_heads_independent_and_future_keys(o):
    """Heads do not interact (Section 2.1), and under the causal mask row i ignores keys j > i."""
    rng = _rng(22)
    L, d, k = 30, 5, 4
    Q, K, V = (rng.standard_normal((1, 3, L, d)) for _ in range(3))
    base = o.oracle_attn(Q, K, V, k, 8, True, 0.6)
    K2, V2 = K.copy(), V.copy()
    K2[0, 1] = rng.standard_normal((L, d))
    V2[0, 1] = rng.standard_normal((L, d))
    r = o.oracle_attn(Q, K2, V2, k, 8, True, 0.6)
    for h in (0, 2):
        _close(r["out"][0, h], base["out"][0, h], 0.0, "other heads unchanged")
    i = 11
    K3, V3 = K.copy(), V.copy()
    K3[0, 0, i + 1:] = 10 * rng.standard_normal((L - i - 1, d))
    V3[0, 0, i + 1:] = rng.standard_normal((L - i - 1, d))
    r3 = o.oracle_attn(Q, K3, V3, k, 8, True, 0.6)
    _close(r3["out"][0, 0, :i + 1], base["out"][0, 0, :i + 1], 1e-12, "future keys ignored")


def pin_from_indices_matches(o):
    """Steps 4-6 on the oracle's own sets reproduce its outputs (acceptance-rule helper)."""
    rng = _rng(23)
    L, d, k = 33, 7, 5
    Q, K, V = (rng.standard_normal((1, 1, L, d)) for _ in range(3))
    for causal in (False, True):
        r = o.oracle_attn(Q, K, V, k, 0, causal, 0.8)
        out, w = o.from_indices(Q[0, 0], K[0, 0], V[0, 0], r["idx"][0, 0], "softmax", 0.8)
        _close(out, r["out"][0, 0], 1e-12, "from_indices")
        _close(w.sum(axis=1), np.ones(L), 1e-12, "softmax weights sum to 1")


# ---------------------------------------------------------------- the row-subset variants (Eq. 4, Eq. 2)
def pin_selected_scores_vs_loops(o):
    """Scores of given (row, key) pairs vs explicit loops; -1 pads give -inf."""
    rng = _rng(24)
    Q = rng.standard_normal((5, 4))
    K = rng.standard_normal((11, 4))
    idx = rng.integers(-1, 11, size=(5, 6))
    got = o.selected_scores(Q, K, idx)
    for r in range(5):
        for m in range(6):
            j = int(idx[r, m])
            if j < 0:
                assert got[r, m] == -np.inf
            else:
                assert abs(got[r, m] - brute.dot(Q[r], K[j])) <= 1e-12, f"pair ({r}, {j})"


def pin_rows_variants_match_whole_calls(o):
    """oracle_attn_rows on rows drawn across heads and chunk boundaries, shuffled and with
    repeats, returns exactly what the whole call gives at those rows, in the order asked
    (causal rows take their own position for the mask); the same for oracle_ffn_rows.
    Run with a small row batch so that one (b, h) group spans several batches."""
    rng = _rng(25)
    B, H, L, d, k = 2, 2, 37, 5, 6
    Q, K, V = (rng.standard_normal((B, H, L, d)) for _ in range(3))
    grid = np.stack(np.meshgrid(np.arange(B), np.arange(H), np.arange(L), indexing="ij"), -1).reshape(-1, 3)
    rows = np.concatenate([grid[rng.permutation(len(grid))[:90]], grid[[0, 5, 37, 40]]])
    saved = o.ROW_BATCH
    o.ROW_BATCH = 7
    try:
        for causal in (False, True):
            full = o.oracle_attn(Q, K, V, k, 8, causal, 0.45)
            got = o.oracle_attn_rows(Q, K, V, k, causal, 0.45, rows)
            at = (rows[:, 0], rows[:, 1], rows[:, 2])
            assert np.array_equal(got["idx"], full["idx"][at]), f"rows idx (causal={causal})"
            assert np.array_equal(got["k_eff"], full["k_eff"][at]), f"rows k_eff (causal={causal})"
            _close(got["out"], full["out"][at], 1e-12, f"rows out (causal={causal})")
            _close(np.nan_to_num(got["sigma_k1"], nan=7.0), np.nan_to_num(full["sigma_k1"][at], nan=7.0), 1e-12,
                   "rows sigma_k1")
        X = rng.standard_normal((29, d))
        W1, W2 = rng.standard_normal((23, d)), rng.standard_normal((23, d))
        full = o.oracle_ffn(X, W1, W2, 4, 6)
        trow = np.concatenate([rng.permutation(29), [3, 3, 28]])
        got = o.oracle_ffn_rows(X, W1, W2, 4, trow)
        assert np.array_equal(got["idx"], full["idx"][trow]), "ffn rows idx"
        _close(got["out"], full["out"][trow], 1e-12, "ffn rows out")
    finally:
        o.ROW_BATCH = saved


# ---------------------------------------------------------------- the output acceptance metric
def pin_output_rel_errors_rejects_wrong_rows(o):
    """The per-row output ratio (row max-norm error over row max-norm reference, with a
    floor only for zero-weight rows): exact rows give 0; a row moved by 2.5e-2 of its
    largest entry fails the bf16 bound 2e-2 and one moved by 2e-5 fails the fp32 bound
    1e-5, in that row only; a single wrong element is enough; a feed-forward row whose
    survivors all score <= 0 (zero weights, zero reference) fails for any non-zero output
    and passes for zero."""
    rng = _rng(26)
    R, dv = 6, 9
    ref = rng.standard_normal((R, dv))
    w = np.abs(rng.standard_normal((R, 4)))
    vmax = 3.0
    assert np.all(o.output_rel_errors(ref.copy(), ref, w, vmax) == 0.0)
    for rel, rtol in ((2.5e-2, 2e-2), (2e-5, 1e-5)):
        g = ref.copy()
        r, t = 2, int(np.argmax(np.abs(ref[2])))
        g[r, t] += rel * np.max(np.abs(ref[r]))
        ratio = o.output_rel_errors(g, ref, w, vmax)
        assert ratio.shape == (R,)
        assert ratio[r] > rtol and abs(ratio[r] - rel) <= 1e-9 * rel, f"perturbed row ratio {ratio[r]}"
        assert np.all(np.delete(ratio, r) == 0.0), "only the perturbed row may fail"
        g = ref.copy()
        g[4, 7] = ref[4, 7] + 0.4 * rel * np.max(np.abs(ref[4]))   # a smaller move passes
        assert o.output_rel_errors(g, ref, w, vmax)[4] <= rtol
    # zero-weight row (all survivors <= 0 under ReLU): reference 0, floor 0
    ref0 = ref.copy()
    ref0[1] = 0.0
    w0 = w.copy()
    w0[1] = 0.0
    g = ref0.copy()
    assert o.output_rel_errors(g, ref0, w0, vmax)[1] == 0.0
    g[1, 3] = 1e-3
    assert o.output_rel_errors(g, ref0, w0, vmax)[1] > 1.0
    # near-zero reference with weights: the floor (1e-6 max|V| sum|w|) keeps the ratio finite
    ref1 = ref.copy()
    ref1[5] = 1e-12
    g = ref1.copy()
    g[5] += 1e-9
    fl = 1e-6 * vmax * np.sum(np.abs(w[5]))
    assert abs(o.output_rel_errors(g, ref1, w, vmax)[5] - 1e-9 / fl) <= 1e-9 * (1e-9 / fl)


ALL_PINS = [v for kname, v in sorted(globals().items()) if kname.startswith("pin_")]
