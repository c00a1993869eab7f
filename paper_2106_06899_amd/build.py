"""Build the gfx950 HIP library in place (hipcc, no CUDA, no JIT).

Three builds of the same sources:

* ``libtopk.so``       -- the library;
* ``libtopk_check.so`` -- with ``TOPK_CHECK_INDICES``: forward calls wait for their
  stream and report asynchronous kernel errors, and the finalize counts selected
  indices outside the value matrix (``topk_debug_bad_indices``);
* ``libtopk_san.so``   -- the host code built with AddressSanitizer and
  UndefinedBehaviorSanitizer (device code unchanged), for the CPU tests of the
  C ABI's argument checks and planning; it needs the sanitizer runtime preloaded.

Run as ``python -m paper_2106_06899_amd.build`` or call ``build()``.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SOURCES = ["csrc/topk_kernels.hip", "csrc/topk_dense.hip", "csrc/topk_api.hip"]
LIB = os.path.join(PKG, "libtopk.so")
LIB_CHECK = os.path.join(PKG, "libtopk_check.so")
LIB_SAN = os.path.join(PKG, "libtopk_san.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",      # MFMA accumulators in VGPRs: no accvgpr copies
    "-Wall", "-Wno-unused-function",
]
VARIANTS = {
    "main": (LIB, []),
    "check": (LIB_CHECK, ["-DTOPK_CHECK_INDICES"]),
    # host code only: each -fsanitize= applies to the host compilation
    "san": (LIB_SAN, ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                      "-Xarch_host", "-fno-omit-frame-pointer", "-shared-libsan", "-O1"]),
}


def sanitizer_runtime() -> str | None:
    """The ASan runtime a process must preload to load libtopk_san.so."""
    pats = ["/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so",
            "/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"]
    for p in pats:
        hits = sorted(glob.glob(p))
        if hits:
            return hits[-1]
    return None


def _command(out: str, extra: list[str]) -> list[str]:
    return [HIPCC, *FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"),
            *[os.path.join(PKG, s) for s in SOURCES], "-o", out + ".tmp"]


def build(verbose: bool = False, variants=("main", "check", "san")) -> str:
    """Compile every HIP source for gfx950 into each requested library (always
    recompiles; the builds run in parallel). Returns the path of libtopk.so."""
    procs = []
    for name in variants:
        out, extra = VARIANTS[name]
        cmd = _command(out, extra)
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((out, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    failed = []
    for out, p in procs:
        log, _ = p.communicate()
        if p.returncode != 0:
            sys.stderr.write(log)
            failed.append(os.path.basename(out))
        else:
            os.replace(out + ".tmp", out)
    if failed:
        raise RuntimeError("hipcc failed building " + ", ".join(failed))
    return LIB


if __name__ == "__main__":
    which = tuple(sys.argv[1:]) or ("main", "check", "san")
    print(build(verbose=True, variants=which))
