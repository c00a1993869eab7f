"""Seeded synthetic workloads for top-k attention and the top-k feed-forward layer.

This module only draws input tensors. It holds none of the method's arithmetic
(no scores, no selection, no activation, no gather): the oracle and the HIP path
both consume what it returns, and neither is imported here.

The paper benchmarks on random inputs (Section 3, "Experimental details", and the
appendix on benchmarking details); the shapes below stand in for its benchmark
shapes:

* ``c1`` a small fp32 single-head case (query chunk 256, Eq. 1 temperature sqrt(d));
* ``c2`` the BERT-base encoder attention shape (12 heads of 64, Section 3);
* ``c3`` a long sequence, 32768 tokens, whose queries have a planted top set;
* ``c4`` a causal decoder with top-128 and chunk 1024, the setting of the
  multi-head attention benchmark in Section 3 (Eq. 2 mask);
* ``c5`` the feed-forward recast (Eq. 3) at the top-512, d_ff = 65536 point of the
  feed-forward benchmark in Section 3, on one 16384-token slice.

Every value is drawn in float32 from ``numpy.random.Generator(PCG64(seed))`` and,
for bf16 workloads, rounded to nearest-even to bfloat16. bf16 tensors are returned
as raw ``uint16`` bit patterns plus their exact float32 values.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class Workload:
    """One benchmark / parity configuration.

    Attention (``kind == "attn"``): Q is [B, H, Lq, d], K and V are [B, H, Lk, d].
    Feed-forward (``kind == "ffn"``): X is [N, d_model], W1 (keys) and W2 (values)
    are [d_ff, d_model]; row j of W1 is key j and row j of W2 is value j.
    ``std`` is the standard deviation of the Gaussian draws (for the FFN it applies
    to W1 and W2; X is always unit variance).
    """
    name: str
    kind: str                      # "attn" or "ffn"
    dtype: str                     # "f32" or "bf16"
    k: int
    chunk: int
    seed: int
    B: int = 1
    H: int = 1
    Lq: int = 0
    Lk: int = 0
    d: int = 0
    causal: bool = False
    scale: float = 1.0             # softmax temperature 1/lambda (Eq. 1); unused by the FFN
    planted: int = 0               # >0: each query = sum of `planted` key rows + noise
    noise_std: float = 0.0
    N: int = 0
    d_model: int = 0
    d_ff: int = 0
    std: float = 1.0
    note: str = ""

    @property
    def queries(self) -> int:
        return self.B * self.H * self.Lq if self.kind == "attn" else self.N

    def scaled(self, **kw) -> "Workload":
        """Same recipe at other sizes (used for small parity cases)."""
        return replace(self, **kw)


def _f32_scale(x: float) -> float:
    return float(np.float32(x))


WORKLOADS = {
    "c1": Workload("c1", "attn", F32, k=32, chunk=256, seed=1001, B=1, H=1, Lq=1024, Lk=1024, d=64,
                   scale=_f32_scale(1 / math.sqrt(64)),
                   note="1x1x1024, d=64, fp32, k=32, chunk 256, no mask"),
    "c2": Workload("c2", "attn", BF16, k=64, chunk=512, seed=1002, B=8, H=12, Lq=512, Lk=512, d=64,
                   scale=_f32_scale(1 / math.sqrt(64)),
                   note="encoder layer 8x12x512, d=64, bf16, k=64, chunk 512, no mask"),
    "c3": Workload("c3", "attn", BF16, k=64, chunk=1024, seed=1003, B=1, H=16, Lq=32768, Lk=32768, d=64,
                   scale=_f32_scale(1 / math.sqrt(64)), planted=4, noise_std=0.5,
                   note="long sequence 1x16x32768, d=64, bf16, k=64, chunk 1024, planted top set"),
    "c4": Workload("c4", "attn", BF16, k=128, chunk=1024, seed=1004, B=4, H=16, Lq=8192, Lk=8192, d=128,
                   causal=True, scale=_f32_scale(1 / math.sqrt(128)),
                   note="causal decoder 4x16x8192, d=128, bf16, k=128, chunk 1024"),
    "c5": Workload("c5", "ffn", BF16, k=512, chunk=1024, seed=1005, N=16384, d_model=1024, d_ff=65536,
                   std=0.02,
                   note="feed-forward N=16384, d_model=1024, d_ff=65536, bf16, k=512, chunk 1024"),
}


# ----------------------------------------------------------------------------- bf16 storage
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16, nearest-even, returning uint16 bit patterns (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact float32 value of bfloat16 bit patterns."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Tensor:
    """A synthetic input: its float32 value and, for bf16, its storage bits."""
    values: np.ndarray                 # float32, exact value of the stored element
    bits: np.ndarray | None = None     # uint16 bf16 bit patterns when dtype is bf16
    dtype: str = F32

    def storage(self) -> np.ndarray:
        return self.bits if self.dtype == BF16 else self.values


def _store(x32: np.ndarray, dtype: str) -> Tensor:
    if dtype == BF16:
        bits = f32_to_bf16_bits(x32)
        return Tensor(bf16_bits_to_f32(bits), bits, BF16)
    return Tensor(np.ascontiguousarray(x32, dtype=np.float32), None, F32)


def _distinct_indices(rng: np.random.Generator, rows: int, n: int, count: int) -> np.ndarray:
    """`count` distinct integers in [0, n) per row, uniform without replacement."""
    idx = rng.integers(0, n, size=(rows, count), dtype=np.int64)
    while True:
        s = np.sort(idx, axis=1)
        dup = np.any(s[:, 1:] == s[:, :-1], axis=1)
        if not dup.any():
            return idx
        idx[dup] = rng.integers(0, n, size=(int(dup.sum()), count), dtype=np.int64)


def make_inputs(w: Workload, seed: int | None = None) -> dict:
    """Draw the inputs of workload `w` (seed defaults to the workload's own).

    Returns a dict with Tensors ``Q, K, V`` (attention) or ``X, W1, W2`` (FFN) and,
    for planted workloads, ``planted_idx`` [B, H, Lq, planted] (the key rows summed
    into each query; a generator check, not part of the method).
    """
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    if w.kind == "ffn":
        X = rng.standard_normal((w.N, w.d_model), dtype=np.float32)
        W1 = rng.standard_normal((w.d_ff, w.d_model), dtype=np.float32) * np.float32(w.std)
        W2 = rng.standard_normal((w.d_ff, w.d_model), dtype=np.float32) * np.float32(w.std)
        return {"X": _store(X, w.dtype), "W1": _store(W1, w.dtype), "W2": _store(W2, w.dtype)}

    shape_k = (w.B, w.H, w.Lk, w.d)
    K = _store(rng.standard_normal(shape_k, dtype=np.float32), w.dtype)
    V = _store(rng.standard_normal(shape_k, dtype=np.float32), w.dtype)
    out = {"K": K, "V": V}
    if w.planted > 0:
        Q32 = np.empty((w.B, w.H, w.Lq, w.d), dtype=np.float32)
        pidx = np.empty((w.B, w.H, w.Lq, w.planted), dtype=np.int64)
        for b in range(w.B):
            for h in range(w.H):
                sel = _distinct_indices(rng, w.Lq, w.Lk, w.planted)
                pidx[b, h] = sel
                acc = np.zeros((w.Lq, w.d), dtype=np.float32)
                for t in range(w.planted):              # sum of the chosen bf16 key rows, in fp32
                    acc += K.values[b, h][sel[:, t]]
                acc += rng.standard_normal((w.Lq, w.d), dtype=np.float32) * np.float32(w.noise_std)
                Q32[b, h] = acc
        out["Q"] = _store(Q32, w.dtype)
        out["planted_idx"] = pidx
    else:
        out["Q"] = _store(rng.standard_normal((w.B, w.H, w.Lq, w.d), dtype=np.float32), w.dtype)
    return out


def small_case(name: str, **kw) -> Workload:
    """A reduced-size copy of a named workload's recipe (same dtype, k/L ratio chosen by caller)."""
    return replace(WORKLOADS[name], **kw)
