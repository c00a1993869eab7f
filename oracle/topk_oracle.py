"""fp64 CPU oracle of top-k attention (Eq. 4) and of the top-k feed-forward layer (Eq. 3 + Eq. 4).

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The product path (the
HIP library and its Python binding) never calls it, and this module shares no
code with that path.

It follows the forward pass of the paper's pseudo-code (Section 2.2, "Improving
efficiency through top-k attention") for one query chunk at a time, in the order
the paper gives the steps:

1. ``dots = Q_C K^T``                         -- the chunk's score tile (Eq. 4);
2. masked entries set to -inf                   -- the binary mask B of Eq. 2 (causal);
3. ``top_dots, top_indices = row_wise_topk``    -- keep each row's k largest entries;
4. ``top_actv = activation(top_dots)``          -- softmax over the k survivors (Eq. 1
   with temperature) or ReLU (Eq. 3);
5. ``actv = matrix(top_actv, top_indices)``     -- scatter into a dense zero matrix;
6. ``out = actv V``                             -- dense product.

Query chunking (Section 2.2, "Query chunking") only bounds memory; each chunk is
computed from ``Q_C, K, V`` alone, so the result does not depend on the chunk size.

Readings of points the paper leaves open:

* selection uses the raw score ``q.k``; the temperature ``scale`` (= 1/lambda of
  Eq. 1) multiplies scores only inside the softmax, and is the float32 value the
  caller passes, upcast to fp64;
* the softmax runs over the k survivors only (non-selected entries are masked out,
  i.e. -inf, not zero);
* ties are broken by the lower key index: rows are ordered by (score desc, index asc);
* causal rows with fewer than k valid keys (key j valid iff j <= i, 0-based) keep
  all of them (k_eff = min(k, i + 1)); padding indices are -1;
* the feed-forward layer has no bias and no temperature; ReLU is applied after the
  selection, so negative survivors stay selected with weight 0.

Every input is upcast exactly to float64 (bf16 and fp32 values are representable).
"""
from __future__ import annotations

import numpy as np


# --------------------------------------------------------------------------- step 1-2
def chunk_scores(Qc: np.ndarray, K: np.ndarray, row0: int | None = None, causal: bool = False) -> np.ndarray:
    """The chunk's score tile ``dots = Q_C K^T`` in fp64 (Eq. 4), with the Eq. 2 mask.

    Qc: [C, d] queries of the chunk, K: [Lk, d] keys. With ``causal`` the query row r
    of the chunk has absolute index ``row0 + r`` and key j is valid iff j <= row0 + r;
    invalid entries are -inf (B = -inf in Eq. 2). ``row0`` may also be an array of
    absolute row indices (one per row of Qc).
    """
    dots = np.asarray(Qc, dtype=np.float64) @ np.asarray(K, dtype=np.float64).T
    if causal:
        rows = np.asarray(row0 if np.ndim(row0) else row0 + np.arange(dots.shape[0]))
        cols = np.arange(dots.shape[1])
        dots[cols[None, :] > rows[:, None]] = -np.inf
    return dots


# --------------------------------------------------------------------------- step 3
def row_wise_topk(dots: np.ndarray, k: int):
    """Each row's k largest entries in the order (score desc, index asc) (Eq. 4).

    ``dots`` is [R, Lk] fp64 with -inf at masked entries. A row with fewer than k
    valid entries keeps all of them (k_eff = min(k, #valid)).

    Returns ``top_idx`` [R, k] int64 (-1 pads), ``top_dots`` [R, k] fp64 (-inf pads),
    ``k_eff`` [R], and the tie-band values ``sigma_k`` (the k_eff-th selected score)
    and ``sigma_k1`` (the next valid score, NaN when every valid key is selected).
    """
    R, Lk = dots.shape
    if not 1 <= k <= Lk:
        raise ValueError("need 1 <= k <= Lk")
    valid = dots > -np.inf
    n_valid = valid.sum(axis=1)
    k_eff = np.minimum(k, n_valid)

    # t = the k-th largest entry of each row (masked entries count as -inf).
    neg = -dots
    if k < Lk:
        part = np.partition(neg, (k - 1, k), axis=1)
        t = -part[:, k - 1]
        t_next = -part[:, k]
    else:
        t = dots.min(axis=1)
        t_next = np.full(R, -np.inf)

    # Everything strictly above t is in; entries equal to t fill the rest, lowest index first.
    above = dots > t[:, None]
    equal = (dots == t[:, None]) & valid
    need = k_eff - above.sum(axis=1)
    take_equal = equal & (np.cumsum(equal, axis=1) <= need[:, None])
    chosen = above | take_equal
    assert np.array_equal(chosen.sum(axis=1), k_eff)

    rows, cols = np.nonzero(chosen)                       # row-major: cols ascending per row
    slot = np.arange(rows.size) - np.repeat(np.cumsum(k_eff) - k_eff, k_eff)
    top_idx = np.full((R, k), -1, dtype=np.int64)
    top_dots = np.full((R, k), -np.inf)
    top_idx[rows, slot] = cols
    top_dots[rows, slot] = dots[rows, cols]

    # Order each row by (score desc, index asc); pads (-inf, -1) go last.
    idx_key = np.where(top_idx < 0, np.iinfo(np.int64).max, top_idx)
    order = np.lexsort((idx_key, -top_dots), axis=1)
    top_idx = np.take_along_axis(top_idx, order, axis=1)
    top_dots = np.take_along_axis(top_dots, order, axis=1)

    sigma_k = top_dots[np.arange(R), k_eff - 1]
    sigma_k1 = np.where(n_valid > k, t_next, np.nan)
    return top_idx, top_dots, k_eff, sigma_k, sigma_k1


# --------------------------------------------------------------------------- step 4
def softmax_over_survivors(top_dots: np.ndarray, scale: float) -> np.ndarray:
    """Row softmax of ``scale * top_dots`` over the selected entries only (Eq. 1, Eq. 4).

    Pads (-inf) get weight 0. ``scale`` is the temperature 1/lambda of Eq. 1.
    """
    s = np.float64(np.float32(scale)) * top_dots
    m = np.max(s, axis=1, keepdims=True)
    e = np.where(np.isfinite(top_dots), np.exp(s - m), 0.0)
    return e / e.sum(axis=1, keepdims=True)


def relu_over_survivors(top_dots: np.ndarray) -> np.ndarray:
    """ReLU of the selected entries (Eq. 3 recast through Eq. 4); pads get weight 0."""
    return np.where(np.isfinite(top_dots), np.maximum(top_dots, 0.0), 0.0)


# --------------------------------------------------------------------------- step 5-6
def scatter_dense(top_actv: np.ndarray, top_idx: np.ndarray, Lk: int) -> np.ndarray:
    """``actv = matrix(top_actv, top_indices)``: a dense [R, Lk] matrix of zeros holding
    each row's activations at its selected columns."""
    R = top_idx.shape[0]
    actv = np.zeros((R, Lk))
    r, c = np.nonzero(top_idx >= 0)
    actv[r, top_idx[r, c]] = top_actv[r, c]
    return actv


def chunk_forward(Qc, K, V, k, activation, scale=1.0, row0=0, causal=False):
    """Top-k attention for one query chunk (Section 2.2 forward pseudo-code).

    Returns a dict: ``out`` [C, dv] fp64, ``idx`` [C, k], ``top`` [C, k] raw scores,
    ``k_eff``, ``sigma_k``, ``sigma_k1``.
    """
    dots = chunk_scores(Qc, K, row0, causal)
    top_idx, top_dots, k_eff, sk, sk1 = row_wise_topk(dots, k)
    del dots
    if activation == "softmax":
        top_actv = softmax_over_survivors(top_dots, scale)
    elif activation == "relu":
        top_actv = relu_over_survivors(top_dots)
    else:
        raise ValueError(activation)
    actv = scatter_dense(top_actv, top_idx, K.shape[0])
    out = actv @ np.asarray(V, dtype=np.float64)
    return {"out": out, "idx": top_idx, "top": top_dots, "k_eff": k_eff, "sigma_k": sk, "sigma_k1": sk1}


# --------------------------------------------------------------------------- whole calls
def _stack(parts, shape_prefix):
    return {key: np.concatenate([p[key] for p in parts], axis=0).reshape(shape_prefix + parts[0][key].shape[1:])
            for key in parts[0]}


def oracle_attn(Q, K, V, k, chunk, causal, scale):
    """top-k attention over [B, H, L, d] inputs, chunk by chunk (Eq. 4 + query chunking).

    Outputs have shape [B, H, Lq, ...].
    """
    B, H, Lq, _ = Q.shape
    chunk = Lq if chunk in (0, None) else int(chunk)
    res = []
    for b in range(B):
        for h in range(H):
            for c0 in range(0, Lq, chunk):
                res.append(chunk_forward(Q[b, h, c0:c0 + chunk], K[b, h], V[b, h], k, "softmax",
                                         scale, c0, causal))
    return _stack(res, (B, H, Lq))


def oracle_ffn(X, W1, W2, k, chunk):
    """top-k feed-forward layer: keys are the rows of W1, values the rows of W2, ReLU
    activation (Eq. 3 through Eq. 4), token chunk by token chunk. Outputs [N, ...]."""
    N = X.shape[0]
    chunk = N if chunk in (0, None) else int(chunk)
    res = [chunk_forward(X[c0:c0 + chunk], W1, W2, k, "relu") for c0 in range(0, N, chunk)]
    return _stack(res, (N,))


def oracle_attn_rows(Q, K, V, k, causal, scale, rows):
    """The oracle on a subset of query rows; ``rows`` is an int array [R, 3] of (b, h, i).

    Each (b, h) group of rows is one query chunk (chunking does not change the result).
    Results are returned in the order of ``rows``.
    """
    rows = np.asarray(rows, dtype=np.int64)
    out = {}
    for (b, h) in sorted({(int(r[0]), int(r[1])) for r in rows}):
        pos = np.nonzero((rows[:, 0] == b) & (rows[:, 1] == h))[0]
        i = rows[pos, 2]
        r = chunk_forward(Q[b, h][i], K[b, h], V[b, h], k, "softmax", scale, i, causal)
        for key, val in r.items():
            if key not in out:
                out[key] = np.empty((rows.shape[0],) + val.shape[1:], dtype=val.dtype)
            out[key][pos] = val
    return out


def oracle_ffn_rows(X, W1, W2, k, rows):
    """The feed-forward oracle on a subset of token rows (int array [R])."""
    rows = np.asarray(rows, dtype=np.int64)
    return chunk_forward(X[rows], W1, W2, k, "relu")


# --------------------------------------------------------------------------- given index sets
def from_indices(Qr, K, V, idx, activation, scale=1.0):
    """Steps 4-6 on a GIVEN index set per row (e.g. the one the GPU selected).

    Qr: [R, d] query rows, idx: [R, k] (-1 pads). Scores of the given keys are
    recomputed in fp64; returns ``out`` [R, dv] and the weights ``w`` [R, k].
    """
    Qr = np.asarray(Qr, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    valid = idx >= 0
    safe = np.where(valid, idx, 0)
    top = np.einsum("rd,rkd->rk", Qr, K[safe])
    top = np.where(valid, top, -np.inf)
    if activation == "softmax":
        w = softmax_over_survivors(top, scale)
    else:
        w = relu_over_survivors(top)
    actv = scatter_dense(w, idx, K.shape[0])
    return actv @ np.asarray(V, dtype=np.float64), w


def key_scores(Qr, K, idx):
    """fp64 scores q_r . K[idx[r, t]] for arbitrary (row, key) pairs (-1 -> NaN)."""
    Qr = np.asarray(Qr, dtype=np.float64)
    valid = idx >= 0
    s = np.einsum("rd,rkd->rk", Qr, np.asarray(K, dtype=np.float64)[np.where(valid, idx, 0)])
    return np.where(valid, s, np.nan)


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
