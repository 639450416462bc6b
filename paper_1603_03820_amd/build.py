"""Build libals.so (the HIP kernels and the C ABI of include/als.h) for gfx950, in tree."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "als.hip")
HEADER = os.path.join(ROOT, "include", "als.h")
LIB = os.path.join(PKG, "libals.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # code object v5: loadable by the HIP runtime that ships with the PyTorch-ROCm wheel
    "-mcode-object-version=5",
    # no packed-FP32 VALU instructions anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # keep MFMA accumulators in the unified VGPR file: the solve works on them with VALU ops,
    # and one register pool (not VGPR + AGPR copies) doubles the resident waves
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.isabs(cand) and os.path.exists(cand) or not os.path.isabs(cand)):
            return cand
    return "hipcc"


PEAKS_SRC = os.path.join(PKG, "csrc", "peaks.hip")
PEAKS_LIB = os.path.join(PKG, "libpeaks.so")


def build(verbose: bool = False) -> str:
    """Compile libals.so and the bench's peak microbenchmarks (libpeaks.so) unconditionally (the
    build check compiles every time); return the libals.so path."""
    _compile(PEAKS_SRC, PEAKS_LIB, verbose)
    return _compile(SRC, LIB, verbose)


def _compile(src: str, lib: str, verbose: bool) -> str:
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), src, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the device-only target feature; that note is harmless
    err = "\n".join(l for l in r.stderr.splitlines() if "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
