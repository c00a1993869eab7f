"""CPU tests: the multi-head layer oracle against its pins, and planted mistakes."""
import numpy as np
import pytest

from oracle import topk_mha as mo
from tests import mha_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(mo)


def _planted(monkeypatch, name, fake):
    monkeypatch.setattr(mo, name, fake)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(mo)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    return failed


def test_head_split_transposed_is_caught(monkeypatch):
    """Heads taken as interleaved columns instead of contiguous blocks."""
    def split(Y, H):
        B, L, D = Y.shape
        return Y.reshape(B, L, D // H, H).transpose(0, 3, 1, 2)
    assert _planted(monkeypatch, "split_heads", split)


def test_output_projection_untransposed_is_caught(monkeypatch):
    orig = mo.mha_forward

    def f(X, Wqkv, bqkv, Wo, bo, *a, **kw):
        return orig(X, Wqkv, bqkv, np.ascontiguousarray(np.asarray(Wo).T), bo, *a, **kw)
    assert _planted(monkeypatch, "mha_forward", f)
