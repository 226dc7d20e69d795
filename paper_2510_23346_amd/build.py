"""Build the gfx950 HIP library ``libbdlora.so`` in place.

    python -m paper_2510_23346_amd.build

The library holds the kernels and the C ABI declared in ``include/bdlora.h``.
It is compiled for gfx950 only.  Packed-fp32 instruction forms are switched
off for the device code (``-packed-fp32-ops``): the kernels do their fp32
arithmetic with ordinary scalar instructions.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libbdlora.so")

SOURCES = ["bdl_prep.hip", "bdl_decode.hip", "bdl_kernels.hip", "bdl_gemm.hip", "bdl_static.hip", "bdl_api.cpp"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libbdlora.so)")


def build(verbose: bool = False) -> str:
    """Compile every source into ``libbdlora.so`` (always recompiles)."""
    tmp = LIB + ".tmp"
    cmd = [
        hipcc(), "-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-shared",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wno-unused-command-line-argument",
        "-I", INCLUDE, "-I", CSRC,
    ] + [os.path.join(CSRC, s) for s in SOURCES] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature; that warning is harmless
    noise = ("packed-fp32-ops", "is not a recognized feature for this target")
    err = "\n".join(ln for ln in (r.stderr or "").splitlines() if not any(n in ln for n in noise))
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
