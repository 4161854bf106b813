"""Build of the HIP libraries (gfx950), in-tree: ``libmadd.so`` (the
optimizer step, include/madd.h) and, outside the package,
``bench_probes/libmadd_probes.so`` (measurement probes, not part of the
optimizer: the streaming ceiling the benchmark reports beside the HBM peak,
and the exhaustive check of the bf16 conversion instructions;
bench_probes/madd_probes.h).

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
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "madd.hip")
HDR = os.path.join(ROOT, "include", "madd.h")
CACHE_HDR = os.path.join(PKG, "csrc", "table_cache.h")
LIB = os.path.join(PKG, "libmadd.so")
PROBE_DIR = os.path.join(ROOT, "bench_probes")
PROBE_SRC = os.path.join(PROBE_DIR, "probes.hip")
PROBE_HDR = os.path.join(PROBE_DIR, "madd_probes.h")
PROBE_LIB = os.path.join(PROBE_DIR, "libmadd_probes.so")
TARGETS = ((SRC, HDR, LIB), (PROBE_SRC, PROBE_HDR, PROBE_LIB))
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


NPARTS = 10  # csrc/madd.hip is compiled as parts 0..9 (-DMADD_PART=k), in parallel


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = False) -> str:
    """Compile every library next to this file; returns libmadd.so's path."""
    inc = ["-I", os.path.join(ROOT, "include")]
    compile_flags = [f for f in HIPCC_FLAGS if f != "-shared"]
    with tempfile.TemporaryDirectory(prefix="madd_build_") as tmpdir:
        objs = [os.path.join(tmpdir, f"madd_part{k}.o") for k in range(NPARTS)]
        cmds = [[hipcc(), *compile_flags, *inc, f"-DMADD_PART={k}", "-c", "-o", objs[k], SRC]
                for k in range(NPARTS)]
        cmds.append([hipcc(), *HIPCC_FLAGS, "-I", PROBE_DIR, "-o", PROBE_LIB + ".tmp", PROBE_SRC])
        workers = max(1, min(len(cmds), os.cpu_count() or 1))
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(lambda c: _run(c, verbose), cmds))
        _run([hipcc(), *HIPCC_FLAGS, "-o", LIB + ".tmp", *objs], verbose)
    os.replace(LIB + ".tmp", LIB)
    os.replace(PROBE_LIB + ".tmp", PROBE_LIB)
    return LIB


def is_stale() -> bool:
    for src, hdr, lib in TARGETS:
        if not os.path.exists(lib):
            return True
        t = os.path.getmtime(lib)
        deps = (src, hdr, CACHE_HDR) if lib == LIB else (src, hdr)
        if any(os.path.getmtime(p) > t for p in deps):
            return True
    return False


if __name__ == "__main__":
    print(build(verbose=True))
