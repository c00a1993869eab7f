"""Brute-force top-k attention for tiny inputs, in pure Python loops.

TEST INFRASTRUCTURE: used by the oracle's own tests to pin it. Nothing here is
vectorised and nothing is shared with ``topk_oracle``: scores are explicit loops,
the selected set is found by enumerating every k-subset, and the weighted sum is
a loop. It follows the definition of Eq. 4 (top-k of each row of QK^T, then an
activation, then the product with V), with the Eq. 2 causal mask and the readings
stated in ``topk_oracle``'s header (ties: lower key index first).
"""
from __future__ import annotations

import itertools
import math


def dot(a, b):
    s = 0.0
    for x, y in zip(a, b):
        s += float(x) * float(y)
    return s


def scores(Q, K, causal=False, rows=None):
    """Plain loops: s[i][j] = sum_t Q[i][t] K[j][t], None where masked (j > i when causal)."""
    rows = list(range(len(Q))) if rows is None else list(rows)
    out = []
    for r, q in enumerate(Q):
        i = rows[r]
        out.append([None if (causal and j > i) else dot(q, K[j]) for j in range(len(K))])
    return out


def precedes(s, a, b):
    """Total order of Eq. 4's row-wise top-k under our tie reading: higher score first,
    then lower key index."""
    return s[a] > s[b] or (s[a] == s[b] and a < b)


def topk_subset(s_row, k):
    """The unique k_eff-subset of the valid keys in which every member precedes every
    non-member, found by trying every subset."""
    valid = [j for j, v in enumerate(s_row) if v is not None]
    k_eff = min(k, len(valid))
    found = []
    for sub in itertools.combinations(valid, k_eff):
        inside = set(sub)
        outside = [j for j in valid if j not in inside]
        if all(precedes(s_row, a, b) for a in sub for b in outside):
            found.append(sub)
    assert len(found) == 1, "the total order must give exactly one top-k subset"
    return sorted(found[0])


def attention_row(s_row, V, k, scale, activation="softmax"):
    """One output row: activation over the survivors, then the weighted sum of value rows."""
    sub = topk_subset(s_row, k)
    if activation == "softmax":
        m = max(s_row[j] for j in sub)
        e = {j: math.exp(scale * (s_row[j] - m)) for j in sub}
        z = sum(e.values())
        w = {j: e[j] / z for j in sub}
    else:
        w = {j: max(s_row[j], 0.0) for j in sub}
    out = [0.0] * len(V[0])
    for j in sub:
        for t in range(len(out)):
            out[t] += w[j] * float(V[j][t])
    return out, sub


def attention(Q, K, V, k, scale=1.0, causal=False, activation="softmax"):
    """All rows of one head; returns (out rows, selected index lists)."""
    S = scores(Q, K, causal)
    outs, subs = [], []
    for s_row in S:
        o, sub = attention_row(s_row, V, k, scale, activation)
        outs.append(o)
        subs.append(sub)
    return outs, subs
