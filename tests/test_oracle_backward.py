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
    return lambda s, g, valid, act, scale: orig(s, g, valid, act, 1.0)


def _mut_act_no_centering(orig):
    def f(s, g, valid, act, scale):
        w, d = orig(s, g, valid, act, scale)
        if act == "softmax":
            d = np.float64(np.float32(scale)) * w * np.where(valid, g, 0.0)
        return w, d
    return f


def _mut_act_relu_ungated(orig):
    def f(s, g, valid, act, scale):
        w, d = orig(s, g, valid, act, scale)
        if act == "relu":
            d = np.where(valid, g, 0.0)
        return w, d
    return f


def _mut_dots_off_by_one_key(orig):
    def f(Qc, K, idx):
        shifted = np.where(idx >= 0, (idx + 1) % K.shape[0], idx)
        return orig(Qc, K, shifted)
    return f


def _mut_chunk_dk_uses_k(orig):
    def f(Qc, K, V, top_idx, d_out, activation, scale=1.0, top_dots=None):
        dq, dk, dv = orig(Qc, K, V, top_idx, d_out, activation, scale, top_dots)
        return dq, dv, dk  # d_K and d_V swapped
    return f


def _mut_chunk_dq_sign(orig):
    def f(*a, **kw):
        dq, dk, dv = orig(*a, **kw)
        return -dq, dk, dv
    return f


MUTATIONS = {
    "softmax VJP without the temperature": ("activation_backward", _mut_act_no_scale),
    "softmax VJP without centring": ("activation_backward", _mut_act_no_centering),
    "ReLU VJP not gated by s > 0": ("activation_backward", _mut_act_relu_ungated),
    "recomputed scores of the neighbouring key": ("selected_dots", _mut_dots_off_by_one_key),
    "d_K and d_V swapped": ("chunk_backward", _mut_chunk_dk_uses_k),
    "d_Q sign flipped": ("chunk_backward", _mut_chunk_dq_sign),
}


@pytest.mark.parametrize("mutation", sorted(MUTATIONS))
def test_planted_mistake_is_caught(monkeypatch, mutation):
    name, make = MUTATIONS[mutation]
    failed = _caught(monkeypatch, name, make(getattr(bo, name)))
    assert failed, f"no pin caught: {mutation}"
