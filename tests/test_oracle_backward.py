"""CPU tests: the fp64 backward oracle against finite differences, dense closed forms
and invariants, plus checks that a planted mistake in it is caught by some pin."""
import numpy as np
import pytest

from oracle import topk_backward as bo
from tests import backward_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(bo)


def _caught(monkeypatch, name, fake):
    monkeypatch.setattr(bo, name, fake)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(bo)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    return failed


def _mut_act_no_scale(orig):
    return lambda s, a, valid, act, scale: orig(s, a, valid, act, 1.0)


def _mut_act_no_centering(orig):
    def f(s, a, valid, act, scale):
        w, d = orig(s, a, valid, act, scale)
        if act == "softmax":
            d = np.float64(np.float32(scale)) * w * np.where(valid, a, 0.0)
        return w, d
    return f


def _mut_act_relu_ungated(orig):
    def f(s, a, valid, act, scale):
        w, d = orig(s, a, valid, act, scale)
        if act == "relu":
            d = np.where(valid, a, 0.0)
        return w, d
    return f


def _mut_scores_off_by_one_key(orig):
    def f(Qr, K, idx):
        shifted = np.where(idx >= 0, (idx + 1) % K.shape[0], idx)
        return orig(Qr, K, shifted)
    return f


def _mut_dk_dv_swapped(orig):
    def f(*a, **kw):
        r = orig(*a, **kw)
        (dq, dk, dv), m = r if len(r) == 2 else (r, None)
        return ((dq, dv, dk), m) if m is not None else (dq, dv, dk)
    return f


def _mut_dq_sign(orig):
    def f(*a, **kw):
        r = orig(*a, **kw)
        (dq, dk, dv), m = r if len(r) == 2 else (r, None)
        return ((-dq, dk, dv), m) if m is not None else (-dq, dk, dv)
    return f


def _mut_dv_unweighted(orig):
    # d_V as the plain sum of the selecting rows' output gradients (weights dropped)
    def f(Qh, Kh, Vh, idx, G, activation, scale=1.0, chunk=None, magnitudes=False):
        dq, dk, dv = orig(Qh, Kh, Vh, idx, G, activation, scale, chunk)
        dv = np.zeros_like(dv)
        rr, mm = np.nonzero(idx >= 0)
        np.add.at(dv, idx[rr, mm], np.asarray(G, dtype=np.float64)[rr])
        return dq, dk, dv
    return f


MUTATIONS = {
    "softmax VJP without the temperature": ("score_grads", _mut_act_no_scale),
    "softmax VJP without centring": ("score_grads", _mut_act_no_centering),
    "ReLU VJP not gated by s > 0": ("score_grads", _mut_act_relu_ungated),
    "recomputed scores of the neighbouring key": ("selected_scores", _mut_scores_off_by_one_key),
    "d_K and d_V swapped": ("head_backward", _mut_dk_dv_swapped),
    "d_Q sign flipped": ("head_backward", _mut_dq_sign),
    "d_V without the weights": ("head_backward", _mut_dv_unweighted),
}


@pytest.mark.parametrize("mutation", sorted(MUTATIONS))
def test_planted_mistake_is_caught(monkeypatch, mutation):
    name, make = MUTATIONS[mutation]
    failed = _caught(monkeypatch, name, make(getattr(bo, name)))
    assert failed, f"no pin caught: {mutation}"
