"""fp64 CPU oracle of top-k attention (Eq. 4) and of the top-k feed-forward layer (Eq. 3 + Eq. 4).

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The product path (the
HIP library and its Python binding) never calls it, and this module shares no
code with that path.

What is computed is the definition itself, row by row. For one head with keys
k_j and values v_j (j = 0 .. Lk-1) and a query row q_i:

* valid keys: every key, or only j <= i under the causal mask (Eq. 2: the masked
  entries get -inf, so they can never be among the largest);
* scores: s_ij = q_i . k_j (the dot products of Eq. 4, before any temperature);
* survivors S_i: the k_eff = min(k, number of valid keys) valid keys that come first
  when the keys are ordered by score, highest first (Eq. 4 keeps the k largest
  entries of each row);
* weights: the softmax of scale * s_ij over the survivors only (Eq. 1 with its
  temperature, applied to the row that Eq. 4 left), or, for the feed-forward
  layer, w_ij = max(s_ij, 0) (Eq. 3);
* output: o_i = sum over j in S_i of w_ij v_j.

Query chunking (Section 2.2) bounds how many rows are processed at once; each row
depends only on its own query and on all keys and values, so the chunk size does not
change any result. Here it only sets how many rows are scored together.

Readings of points the paper leaves open (the same on the GPU side):

* the temperature ``scale`` (= 1/lambda of Eq. 1) multiplies scores inside the
  softmax only; selection uses the raw score, and the value used is the float32
  number the caller passes, upcast to fp64;
* non-selected entries are excluded from the softmax (-inf), not set to zero;
* equal scores are ordered by the lower key index first;
* a causal row with fewer than k valid keys keeps all of them (k_eff = i + 1);
  index outputs are padded with -1 and score outputs with -inf;
* the feed-forward layer has no bias and no temperature, and ReLU is applied to the
  survivors, so a selected negative score stays selected with weight 0.

Every input is upcast exactly to float64 (bf16 and fp32 values are representable).
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# --------------------------------------------------------------------------- valid keys (Eq. 2)
def valid_lengths(i, Lk: int, causal: bool) -> np.ndarray:
    """Number of valid keys of query rows with absolute indices ``i`` (array): keys
    0 .. n-1 are valid, n = min(i + 1, Lk) under the causal mask (top-left aligned,
    0-based), n = Lk otherwise."""
    i = np.asarray(i, dtype=np.int64)
    return np.minimum(i + 1, Lk) if causal else np.full(i.shape, Lk, dtype=np.int64)


# --------------------------------------------------------------------------- scores (Eq. 4)
def scores(Qr, K, n_valid) -> np.ndarray:
    """fp64 scores s[r, j] = Qr[r] . K[j] of query rows Qr [R, d] against every key
    K [Lk, d]; -inf where key j is not valid for row r (j >= n_valid[r])."""
    s = _f64(Qr) @ _f64(K).T
    j = np.arange(s.shape[1])
    s[j[None, :] >= np.asarray(n_valid)[:, None]] = -np.inf
    return s


def selected_scores(Qr, K, idx) -> np.ndarray:
    """fp64 scores Qr[r] . K[idx[r, m]] of given (row, key) pairs; -inf where idx = -1."""
    valid = idx >= 0
    s = np.einsum("rt,rmt->rm", _f64(Qr), _f64(K)[np.where(valid, idx, 0)])
    return np.where(valid, s, -np.inf)


# --------------------------------------------------------------------------- survivors (Eq. 4)
def select(S: np.ndarray, k: int):
    """The survivors of each row of the score matrix S [R, Lk] (-inf = invalid key).

    A row's survivors are its k_eff = min(k, #valid) valid keys that come first in the
    order (score desc, index asc). With t the k-th largest entry of the row, they are
    every key scoring above t plus, among the keys scoring exactly t, the ones with the
    lowest indices (np.partition finds t).

    Returns ``idx`` [R, k] int64 in that order (-1 pads), ``top`` [R, k] their scores
    (-inf pads), ``k_eff`` [R], ``sigma_k`` (the last survivor's score) and
    ``sigma_k1`` (the best non-survivor's score; NaN when every valid key survives).
    """
    R, Lk = S.shape
    if not 1 <= k <= Lk:
        raise ValueError("need 1 <= k <= Lk")
    valid = S > -np.inf
    n_valid = valid.sum(axis=1)
    k_eff = np.minimum(k, n_valid)
    if k < Lk:
        part = -np.partition(-S, (k - 1, k), axis=1)
        t, t_next = part[:, k - 1], part[:, k]
    else:
        t, t_next = S.min(axis=1), np.full(R, -np.inf)
    above = S > t[:, None]
    at_t = (S == t[:, None]) & valid
    room = k_eff - above.sum(axis=1)
    keep = above | (at_t & (np.cumsum(at_t, axis=1) <= room[:, None]))
    assert np.array_equal(keep.sum(axis=1), k_eff)

    # the kept keys of each row in index order, then sorted by (score desc, index asc);
    # pads (index -1, score -inf) go last
    rows, cols = np.nonzero(keep)
    slot = np.arange(rows.size) - np.repeat(np.cumsum(k_eff) - k_eff, k_eff)
    idx = np.full((R, k), -1, dtype=np.int64)
    top = np.full((R, k), -np.inf)
    idx[rows, slot] = cols
    top[rows, slot] = S[rows, cols]
    order = np.lexsort((np.where(idx < 0, Lk, idx), -top), axis=1)
    idx = np.take_along_axis(idx, order, axis=1)
    top = np.take_along_axis(top, order, axis=1)
    sigma_k = top[np.arange(R), k_eff - 1]
    sigma_k1 = np.where(n_valid > k, t_next, np.nan)
    return idx, top, k_eff, sigma_k, sigma_k1


# --------------------------------------------------------------------------- weights (Eq. 1, Eq. 3)
def softmax_weights(top: np.ndarray, scale: float) -> np.ndarray:
    """Softmax of ``scale * score`` over each row's survivors (Eq. 1 with temperature
    1/scale, restricted to the survivors of Eq. 4); pads (-inf) get weight 0."""
    z = np.float64(np.float32(scale)) * top
    m = np.max(z, axis=1, keepdims=True)
    e = np.where(np.isfinite(top), np.exp(z - m), 0.0)
    return e / e.sum(axis=1, keepdims=True)


def relu_weights(top: np.ndarray) -> np.ndarray:
    """ReLU of each survivor's score (Eq. 3); pads get weight 0."""
    return np.where(np.isfinite(top), np.maximum(top, 0.0), 0.0)


def weights(top, activation: str, scale: float = 1.0) -> np.ndarray:
    if activation == "softmax":
        return softmax_weights(top, scale)
    if activation == "relu":
        return relu_weights(top)
    raise ValueError(activation)


# --------------------------------------------------------------------------- output
def weighted_sum(w: np.ndarray, idx: np.ndarray, V) -> np.ndarray:
    """o[r] = sum_m w[r, m] V[idx[r, m]] over the survivors (pads skipped)."""
    V = _f64(V)
    valid = idx >= 0
    rows = V[np.where(valid, idx, 0)]                  # [R, k, dv]
    return np.einsum("rm,rmt->rt", np.where(valid, w, 0.0), rows)


# --------------------------------------------------------------------------- rows of one head
def topk_rows(Qr, K, V, k, n_valid, activation, scale=1.0):
    """The definition for query rows Qr [R, d] of one head with keys K and values V
    [Lk, *]: row r may use keys 0 .. n_valid[r]-1.

    Returns a dict: ``out`` [R, dv] fp64, ``idx`` [R, k], ``top`` [R, k] raw scores,
    ``k_eff``, ``sigma_k``, ``sigma_k1`` (see ``select``)."""
    S = scores(Qr, K, n_valid)
    idx, top, k_eff, sk, sk1 = select(S, k)
    del S
    out = weighted_sum(weights(top, activation, scale), idx, V)
    return {"out": out, "idx": idx, "top": top, "k_eff": k_eff, "sigma_k": sk, "sigma_k1": sk1}


# --------------------------------------------------------------------------- whole calls
def _stack(parts, shape_prefix):
    return {key: np.concatenate([p[key] for p in parts], axis=0).reshape(shape_prefix + parts[0][key].shape[1:])
            for key in parts[0]}


def oracle_attn(Q, K, V, k, chunk, causal, scale):
    """Top-k attention over [B, H, L, d] inputs; ``chunk`` rows of a head at a time
    (0 or None: the whole head). Outputs have shape [B, H, Lq, ...]."""
    B, H, Lq, _ = Q.shape
    Lk = K.shape[2]
    C = Lq if chunk in (0, None) else int(chunk)
    res = []
    for b in range(B):
        for h in range(H):
            for c0 in range(0, Lq, C):
                i = np.arange(c0, min(c0 + C, Lq))
                res.append(topk_rows(Q[b, h, i], K[b, h], V[b, h], k, valid_lengths(i, Lk, causal), "softmax",
                                     scale))
    return _stack(res, (B, H, Lq))


def oracle_ffn(X, W1, W2, k, chunk):
    """Top-k feed-forward layer: the keys are the rows of W1, the values the rows of
    W2, ReLU weights, no temperature (Eq. 3 through Eq. 4); ``chunk`` tokens at a time.
    Outputs [N, ...]."""
    N, d_ff = X.shape[0], W1.shape[0]
    C = N if chunk in (0, None) else int(chunk)
    res = [topk_rows(X[c0:c0 + C], W1, W2, k, np.full(min(C, N - c0), d_ff), "relu") for c0 in range(0, N, C)]
    return _stack(res, (N,))


ROW_BATCH = 1024  # rows scored together by the *_rows functions (bounds the [rows, Lk] score matrix)


def oracle_attn_rows(Q, K, V, k, causal, scale, rows):
    """The oracle on chosen query rows; ``rows`` is an int array [R, 3] of (b, h, i).
    Results are returned in the order of ``rows``."""
    rows = np.asarray(rows, dtype=np.int64)
    Lk = K.shape[2]
    out = {}
    for (b, h) in sorted({(int(r[0]), int(r[1])) for r in rows}):
        same = np.nonzero((rows[:, 0] == b) & (rows[:, 1] == h))[0]
        for s0 in range(0, same.size, ROW_BATCH):
            pos = same[s0:s0 + ROW_BATCH]
            i = rows[pos, 2]
            r = topk_rows(Q[b, h][i], K[b, h], V[b, h], k, valid_lengths(i, Lk, causal), "softmax", scale)
            for key, val in r.items():
                if key not in out:
                    out[key] = np.empty((rows.shape[0],) + val.shape[1:], dtype=val.dtype)
                out[key][pos] = val
    return out


def oracle_ffn_rows(X, W1, W2, k, rows):
    """The feed-forward oracle on chosen token rows (int array [R]), in that order."""
    rows = np.asarray(rows, dtype=np.int64)
    parts = [topk_rows(X[rows[s0:s0 + ROW_BATCH]], W1, W2, k, np.full(rows[s0:s0 + ROW_BATCH].size, W1.shape[0]),
                       "relu") for s0 in range(0, rows.size, ROW_BATCH)]
    return _stack(parts, (rows.size,))


# --------------------------------------------------------------------------- given index sets
def from_indices(Qr, K, V, idx, activation, scale=1.0):
    """Weights and output for GIVEN survivor sets (e.g. the ones the GPU selected):
    Qr [R, d] query rows, idx [R, k] (-1 pads). Scores of the given keys are
    recomputed in fp64. Returns ``out`` [R, dv] and the weights ``w`` [R, k]."""
    w = weights(selected_scores(Qr, K, idx), activation, scale)
    return weighted_sum(w, idx, V), w


# --------------------------------------------------------------------------- acceptance rules
def check_index_sets(g_idx, t_idx, sigma_k, sigma_k1, k_eff, scores_of, valid_of, rel=1e-5):
    """Index-set acceptance: the sets must be equal except among near-tied keys.

    g_idx, t_idx: [R, k] candidate and oracle index sets (-1 pads). ``scores_of(r, js)``
    returns the oracle's fp64 scores of keys ``js`` for row r; ``valid_of(r, js)``
    says whether keys are valid (in range and unmasked) for row r.
    A row passes iff G has exactly k_eff distinct valid keys and every key in the
    symmetric difference of G and T scores within delta = rel * max(|sigma_k|,
    |sigma_{k+1}|) of sigma_k. Returns (n_bad, n_tie_rows, first_bad_row_or_None).
    """
    n_bad = 0
    n_tie = 0
    first = None
    for r in range(g_idx.shape[0]):
        g = g_idx[r][g_idx[r] >= 0]
        t = t_idx[r][t_idx[r] >= 0]
        ok = (g.size == k_eff[r] and np.unique(g).size == g.size and bool(np.all(valid_of(r, g))))
        if ok:
            diff = np.setxor1d(g, t)
            if diff.size:
                n_tie += 1
                s1 = sigma_k1[r]
                scale_ = max(abs(sigma_k[r]), abs(s1) if np.isfinite(s1) else 0.0)
                delta = rel * scale_
                ok = bool(np.all(np.abs(scores_of(r, diff) - sigma_k[r]) < delta))
        if not ok:
            n_bad += 1
            if first is None:
                first = r
    return n_bad, n_tie, first


def output_rel_errors(out_gpu, out_ref, w_ref, v_absmax):
    """Per-row error ratio  max_t |o_gpu - o_ref| / max(max_t |o_ref|, floor).

    floor = 1e-6 * max|V| * sum_j |w_j| keeps rows whose reference output is (near)
    zero, e.g. a feed-forward row whose survivors all have negative scores, from
    dividing by zero. A row passes when its ratio is <= rtol.
    """
    out_gpu = np.asarray(out_gpu, dtype=np.float64)
    err = np.max(np.abs(out_gpu - out_ref), axis=1)
    ref = np.max(np.abs(out_ref), axis=1)
    floor = 1e-6 * v_absmax * np.sum(np.abs(w_ref), axis=1)
    return err / np.maximum(ref, np.maximum(floor, 1e-300))
