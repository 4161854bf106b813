"""Build of the HIP library ``libmadd.so`` (gfx950), in-tree.

The flags are part of the numerical contract of the kernels:
  * ``-ffp-contract=off``: only the fmaf calls written in the source fuse;
  * ``-fno-gpu-flush-denormals-to-zero``: fp32 denormals are kept;
  * no fast-math: ``/`` and ``sqrtf`` stay correctly rounded;
  * ``-Xclang -target-feature -Xclang -packed-fp32-ops``: packed-FP32 VALU
    instructions are not generated.
"""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "madd.hip")
HDR = os.path.join(ROOT, "include", "madd.h")
LIB = os.path.join(PKG, "libmadd.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def build(verbose: bool = False) -> str:
    """Compile csrc/madd.hip into libmadd.so next to this file; returns its path."""
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), "-o", tmp, SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in (SRC, HDR))


if __name__ == "__main__":
    print(build(verbose=True))
