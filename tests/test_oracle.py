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


def _mut_topk_smallest(orig):
    def f(dots, k):
        fin = np.where(np.isfinite(dots), -dots, -np.inf)
        idx, top, ke, sk, sk1 = orig(fin, k)
        return idx, -top, ke, -sk, -sk1
    return f


def _mut_topk_ties_high_index(orig):
    def f(dots, k):
        rev = dots[:, ::-1].copy()
        idx, top, ke, sk, sk1 = orig(rev, k)
        Lk = dots.shape[1]
        idx = np.where(idx >= 0, Lk - 1 - idx, -1)
        return idx, top, ke, sk, sk1
    return f


def _mut_topk_k_minus_1(orig):
    def f(dots, k):
        idx, top, ke, sk, sk1 = orig(dots, max(k - 1, 1))
        pad = k - idx.shape[1]
        idx = np.pad(idx, ((0, 0), (0, pad)), constant_values=-1)
        top = np.pad(top, ((0, 0), (0, pad)), constant_values=-np.inf)
        return idx, top, ke, sk, sk1
    return f


def _mut_scores_drop_last_feature(orig):
    return lambda Qc, K, row0=None, causal=False: orig(np.asarray(Qc)[:, :-1], np.asarray(K)[:, :-1], row0, causal)


def _mut_scores_causal_strict(orig):
    def f(Qc, K, row0=None, causal=False):
        d = orig(Qc, K, row0, False)
        if causal:
            rows = np.asarray(row0 if np.ndim(row0) else row0 + np.arange(d.shape[0]))
            d[np.arange(d.shape[1])[None, :] >= rows[:, None]] = -np.inf
            d[np.all(d == -np.inf, axis=1), 0] = 0.0
        return d
    return f


def _mut_scores_transposed(orig):
    # Q.K^T replaced by the transpose of K.Q^T restricted to a square block: swaps roles of rows
    def f(Qc, K, row0=None, causal=False):
        d = orig(Qc, K, row0, causal)
        m = min(d.shape)
        d[:m, :m] = d[:m, :m].T.copy()
        return d
    return f


def _mut_relu_before_select(orig):
    return lambda top: orig(np.where(np.isfinite(top), np.abs(top), top))


def _mut_scatter_shift(orig):
    def f(top_actv, top_idx, Lk):
        shifted = np.where(top_idx >= 0, (top_idx + 1) % Lk, -1)
        return orig(top_actv, shifted, Lk)
    return f


MUTATIONS = {
    "softmax_no_scale": ("softmax_over_survivors", _mut_softmax_no_scale),
    "softmax_inverse_scale": ("softmax_over_survivors", _mut_softmax_inverse_scale),
    "topk_smallest": ("row_wise_topk", _mut_topk_smallest),
    "topk_ties_high_index": ("row_wise_topk", _mut_topk_ties_high_index),
    "topk_k_minus_1": ("row_wise_topk", _mut_topk_k_minus_1),
    "scores_drop_last_feature": ("chunk_scores", _mut_scores_drop_last_feature),
    "scores_causal_strict": ("chunk_scores", _mut_scores_causal_strict),
    "scores_transposed": ("chunk_scores", _mut_scores_transposed),
    "relu_abs": ("relu_over_survivors", _mut_relu_before_select),
    "scatter_shift": ("scatter_dense", _mut_scatter_shift),
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
    r = o.chunk_forward(Q, K, V, ex["k"], act, ex.get("scale", 1.0), 0, ex.get("causal", False))
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
    dots = o.chunk_scores(Q, K)
    idx, top, ke, sk, sk1 = o.row_wise_topk(dots, k)
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
    idx2, _, ke2, sk2, sk12 = o.row_wise_topk(dots2, k)
    swapped = idx2.copy()
    swapped[0, k - 1] = order[0, k]
    assert o.check_index_sets(swapped, idx2, sk2, sk12, ke2, lambda r, js: dots2[r, js], valid_of)[0] == 0
    # duplicates and wrong sizes are rejected
    dup = idx.copy()
    dup[1, 1] = dup[1, 0]
    assert o.check_index_sets(dup, idx, sk, sk1, ke, scores_of, valid_of)[0] == 1
