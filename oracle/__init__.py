"""CPU oracle for top-k attention (arXiv 2106.06899, Eq. 4) -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import, call or execute anything in this package. It shares no code with the HIP
library under ``paper_2106_06899_amd/``; the two meet only on the seeded inputs of
``paper_2106_06899_amd.workloads``.

* ``topk_oracle``   -- the forward definition (Eq. 1-4) in fp64 NumPy, row by row;
  the row-subset variants and the acceptance rules the GPU tests use.
* ``topk_backward`` -- the gradients of that definition for fixed survivor sets.
* ``topk_mha``      -- a multi-head layer around it.
* ``brute``         -- pure-Python loops and k-subset enumeration for tiny inputs,
  used to pin ``topk_oracle``.

Parity status: every function of ``topk_oracle`` and ``topk_backward`` is pinned by
tests that do not re-type its formulas (brute force, closed forms, finite
differences, invariants, the whole-call results for the row-subset variants, planted
wrong outputs for the acceptance metric). The GPU's own fp32 accumulation order and
its exp rounding are "parity unpinned": they are covered only by the tolerances of
the acceptance rules.
"""
from . import topk_oracle, brute  # noqa: F401
