"""CPU tests: the fp64 oracle against brute force, closed forms and invariants, plus
checks that a planted mistake in the oracle is caught by at least one pin."""
import json
import math
import os

import numpy as np
import pytest

from oracle import topk_oracle as o
from tests import oracle_pins as pins

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(o)


# ----------------------------------------------------------------------------- planted mistakes
def _caught(monkeypatch, name, fake):
    """Replace oracle function `name` by `fake` and return the pins that fail."""
    monkeypatch.setattr(o, name, fake)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(o)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    return failed


def _mut_softmax_no_scale(orig):
    return lambda top, scale: orig(top, 1.0)


def _mut_softmax_inverse_scale(orig):
    return lambda top, scale: orig(top, 1.0 / scale)


def _mut_select_smallest(orig):
    def f(S, k):
        fin = np.where(np.isfinite(S), -S, -np.inf)
        idx, top, ke, sk, sk1 = orig(fin, k)
        return idx, -top, ke, -sk, -sk1
    return f


def _mut_select_ties_high_index(orig):
    def f(S, k):
        idx, top, ke, sk, sk1 = orig(S[:, ::-1].copy(), k)
        Lk = S.shape[1]
        return np.where(idx >= 0, Lk - 1 - idx, -1), top, ke, sk, sk1
    return f


def _mut_select_k_minus_1(orig):
    def f(S, k):
        idx, top, ke, sk, sk1 = orig(S, max(k - 1, 1))
        pad = k - idx.shape[1]
        idx = np.pad(idx, ((0, 0), (0, pad)), constant_values=-1)
        top = np.pad(top, ((0, 0), (0, pad)), constant_values=-np.inf)
        return idx, top, ke, sk, sk1
    return f


def _mut_scores_drop_last_feature(orig):
    return lambda Qr, K, n_valid: orig(np.asarray(Qr)[:, :-1], np.asarray(K)[:, :-1], n_valid)


def _mut_valid_strict(orig):
    # causal mask j < i instead of j <= i (row 0 keeps key 0 so that it is not empty)
    def f(i, Lk, causal):
        n = orig(i, Lk, causal)
        return np.maximum(n - 1, 1) if causal else n
    return f


def _mut_scores_transposed(orig):
    # Q K^T replaced on a square block by its transpose: swaps the roles of rows and keys
    def f(Qr, K, n_valid):
        s = orig(Qr, K, np.full(len(n_valid), np.asarray(K).shape[0]))
        m = min(s.shape)
        s[:m, :m] = s[:m, :m].T.copy()
        s[np.arange(s.shape[1])[None, :] >= np.asarray(n_valid)[:, None]] = -np.inf
        return s
    return f


def _mut_relu_abs(orig):
    return lambda top: orig(np.where(np.isfinite(top), np.abs(top), top))


def _mut_weighted_sum_shift(orig):
    def f(w, idx, V):
        Lk = np.asarray(V).shape[0]
        return orig(w, np.where(idx >= 0, (idx + 1) % Lk, -1), V)
    return f


def _mut_rows_ignore_position(orig):
    # each (b, h) group of rows masked as if its rows were 0, 1, 2, ... (row index ignored)
    def f(Q, K, V, k, causal, scale, rows):
        rows = np.asarray(rows, dtype=np.int64).copy()
        out = orig(Q, K, V, k, False, scale, rows)
        if causal:
            for (b, h) in {(int(r[0]), int(r[1])) for r in rows}:
                pos = np.nonzero((rows[:, 0] == b) & (rows[:, 1] == h))[0]
                r = o.topk_rows(Q[b, h][rows[pos, 2]], K[b, h], V[b, h], k,
                                o.valid_lengths(np.arange(pos.size), K.shape[2], True), "softmax", scale)
                for key, val in r.items():
                    out[key][pos] = val
        return out
    return f


def _mut_rows_sorted_order(orig):
    # results returned in (b, h, i) order instead of the order of `rows`
    def f(Q, K, V, k, causal, scale, rows):
        rows = np.asarray(rows, dtype=np.int64)
        order = np.lexsort((rows[:, 2], rows[:, 1], rows[:, 0]))
        return orig(Q, K, V, k, causal, scale, rows[order])
    return f


def _mut_ffn_rows_next_token(orig):
    return lambda X, W1, W2, k, rows: orig(X, W1, W2, k, (np.asarray(rows) + 1) % X.shape[0])


def _mut_output_floor_1e6(orig):
    return lambda g, r, w, vmax: orig(g, r, w, vmax * 1e6)


def _mut_output_error_over_rows(orig):
    # the error of each column (over rows) instead of each row
    def f(g, r, w, vmax):
        g = np.asarray(g, dtype=np.float64)
        err = np.max(np.abs(g - r), axis=0)
        ref = np.max(np.abs(r), axis=0)
        return np.resize(err / np.maximum(ref, 1e-300), g.shape[0])
    return f


MUTATIONS = {
    "softmax_no_scale": ("softmax_weights", _mut_softmax_no_scale),
    "softmax_inverse_scale": ("softmax_weights", _mut_softmax_inverse_scale),
    "select_smallest": ("select", _mut_select_smallest),
    "select_ties_high_index": ("select", _mut_select_ties_high_index),
    "select_k_minus_1": ("select", _mut_select_k_minus_1),
    "scores_drop_last_feature": ("scores", _mut_scores_drop_last_feature),
    "causal_mask_strict": ("valid_lengths", _mut_valid_strict),
    "scores_transposed": ("scores", _mut_scores_transposed),
    "relu_abs": ("relu_weights", _mut_relu_abs),
    "weighted_sum_shift": ("weighted_sum", _mut_weighted_sum_shift),
    "rows_ignore_position": ("oracle_attn_rows", _mut_rows_ignore_position),
    "rows_sorted_order": ("oracle_attn_rows", _mut_rows_sorted_order),
    "ffn_rows_next_token": ("oracle_ffn_rows", _mut_ffn_rows_next_token),
    "output_floor_1e6": ("output_rel_errors", _mut_output_floor_1e6),
    "output_error_over_rows": ("output_rel_errors", _mut_output_error_over_rows),
}


@pytest.mark.parametrize("mutation", sorted(MUTATIONS))
def test_planted_mistake_is_caught(monkeypatch, mutation):
    name, make = MUTATIONS[mutation]
    failed = _caught(monkeypatch, name, make(getattr(o, name)))
    assert failed, f"no pin catches the planted mistake {mutation}"


# ----------------------------------------------------------------------------- worked examples
def _expr(s):
    """Evaluate a closed-form expression from a fixture (numbers, + - * / ( ), exp)."""
    allowed = set("0123456789.+-*/() expe")
    assert set(s) <= allowed, s
    return float(eval(s, {"__builtins__": {}}, {"exp": math.exp}))  # noqa: S307 - restricted charset


def _load_examples():
    with open(os.path.join(HERE, "golden", "worked_examples.json")) as f:
        return json.load(f)["examples"]


@pytest.mark.parametrize("ex", _load_examples(), ids=lambda e: e["name"])
def test_worked_example(ex):
    """Hand-derived examples of Eq. 2 / 3 / 4 (see the fixture for each derivation)."""
    Q = np.array(ex["Q"], dtype=np.float64)
    K = np.array(ex["K"], dtype=np.float64)
    V = np.array(ex["V"], dtype=np.float64)
    act = ex["activation"]
    n_valid = o.valid_lengths(np.arange(Q.shape[0]), K.shape[0], ex.get("causal", False))
    r = o.topk_rows(Q, K, V, ex["k"], n_valid, act, ex.get("scale", 1.0))
    for i, want in enumerate(ex["selected"]):
        got = r["idx"][i][r["idx"][i] >= 0].tolist()
        assert got == want, f"row {i}: selected {got}, expected {want}"
    for i, row in enumerate(ex["out"]):
        want = np.array([_expr(v) for v in row])
        np.testing.assert_allclose(r["out"][i], want, rtol=0, atol=1e-15)


# ----------------------------------------------------------------------------- acceptance rules
def test_index_set_rule_accepts_only_near_ties():
    rng = np.random.Generator(np.random.PCG64(5))
    Q = rng.standard_normal((4, 6))
    K = rng.standard_normal((50, 6))
    k = 5
    dots = o.scores(Q, K, np.full(4, 50))
    idx, top, ke, sk, sk1 = o.select(dots, k)
    scores_of = lambda r, js: dots[r, js]          # noqa: E731
    valid_of = lambda r, js: (js >= 0) & (js < 50)  # noqa: E731
    assert o.check_index_sets(idx, idx, sk, sk1, ke, scores_of, valid_of)[0] == 0
    bad = idx.copy()
    # swap the k-th for the (k+1)-th: accepted only if they are within 1e-5 relative
    order = np.argsort(-dots, axis=1, kind="stable")
    bad[:, k - 1] = order[:, k]
    n_bad, n_tie, _ = o.check_index_sets(bad, idx, sk, sk1, ke, scores_of, valid_of)
    gap = np.abs(sk - sk1) / np.maximum(np.abs(sk), np.abs(sk1))
    assert n_bad == int(np.sum(gap >= 1e-5)) and n_tie == 4
    # a near-tie is accepted
    dots2 = dots.copy()
    dots2[0, order[0, k]] = dots2[0, order[0, k - 1]] * (1 - 1e-7)
    idx2, _, ke2, sk2, sk12 = o.select(dots2, k)
    swapped = idx2.copy()
    swapped[0, k - 1] = order[0, k]
    assert o.check_index_sets(swapped, idx2, sk2, sk12, ke2, lambda r, js: dots2[r, js], valid_of)[0] == 0
    # duplicates and wrong sizes are rejected
    dup = idx.copy()
    dup[1, 1] = dup[1, 0]
    assert o.check_index_sets(dup, idx, sk, sk1, ke, scores_of, valid_of)[0] == 1
