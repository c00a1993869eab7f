"""Calls on different streams (the library enqueues every kernel on the caller's
stream; the binding's workspace is a PyTorch tensor allocated on that stream):
forward and backward calls issued on two side streams at once give results identical,
bit for bit, to the same calls made one after another on the default stream."""
import pytest
import torch

import paper_2106_06899_amd as tk
from paper_2106_06899_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    tk.lib()
    yield


def _attn_inputs(base, **kw):
    w = wl.WORKLOADS[base].scaled(**kw)
    x = wl.make_inputs(w)
    return w, tuple(parity.to_dev(x[n]) for n in ("Q", "K", "V"))


def _forward_backward(w, q, k, v, g):
    out, idx, dots = tk.attn(q, k, v, w.k, w.chunk, w.causal, w.scale, cache=True)
    grads = tk.attn_backward(q, k, v, idx, dots, g, w.scale)
    return (out, idx, dots) + tuple(grads)


def test_two_streams_match_serial_results():
    wa, (qa, ka, va) = _attn_inputs("c3", H=2, Lq=512, Lk=4096, chunk=256)        # fused path
    wb, (qb, kb, vb) = _attn_inputs("c4", B=1, H=2, Lq=600, Lk=3000, chunk=128)    # filtered, causal
    _say("streams", wa, wb)
    ga = parity.to_dev(parity.grad_out((wa.B, wa.H, wa.Lq, wa.d), wa.dtype, 90))
    gb = parity.to_dev(parity.grad_out((wb.B, wb.H, wb.Lq, wb.d), wb.dtype, 91))
    ref_a = _forward_backward(wa, qa, ka, va, ga)
    ref_b = _forward_backward(wb, qb, kb, vb, gb)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for rep in range(3):
        with torch.cuda.stream(s1):
            got_a = _forward_backward(wa, qa, ka, va, ga)
        with torch.cuda.stream(s2):
            got_b = _forward_backward(wb, qb, kb, vb, gb)
        torch.cuda.synchronize()
        for name, got, ref in (("a", got_a, ref_a), ("b", got_b, ref_b)):
            for i, (x, y) in enumerate(zip(got, ref)):
                assert torch.equal(x, y), f"stream result {name}[{i}] differs in repetition {rep}"
    _say("streams ok")


def test_two_host_threads_match_serial_results():
    """Two host threads, each on a stream of its own (the workspace registration and the
    last-error message are per thread)."""
    import threading
    wa, (qa, ka, va) = _attn_inputs("c3", H=2, Lq=512, Lk=4096, chunk=256)
    wb, (qb, kb, vb) = _attn_inputs("c2", B=2, H=3, Lq=384, Lk=512, chunk=128)
    ga = parity.to_dev(parity.grad_out((wa.B, wa.H, wa.Lq, wa.d), wa.dtype, 92))
    gb = parity.to_dev(parity.grad_out((wb.B, wb.H, wb.Lq, wb.d), wb.dtype, 93))
    refs = {"a": _forward_backward(wa, qa, ka, va, ga), "b": _forward_backward(wb, qb, kb, vb, gb)}
    torch.cuda.synchronize()
    results, errors = {}, []

    def work(name, w, q, k, v, g):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                outs = [_forward_backward(w, q, k, v, g) for _ in range(3)]
            s.synchronize()
            results[name] = outs
        except Exception as e:  # reported by the main thread
            errors.append(f"{name}: {e!r}")

    threads = [threading.Thread(target=work, args=("a", wa, qa, ka, va, ga)),
               threading.Thread(target=work, args=("b", wb, qb, kb, vb, gb))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    assert not errors, errors
    for name, outs in results.items():
        for rep, got in enumerate(outs):
            for i, (x, y) in enumerate(zip(got, refs[name])):
                assert torch.equal(x, y), f"thread {name} result {i} differs in repetition {rep}"
    assert set(results) == {"a", "b"}
    _say("threads ok")
