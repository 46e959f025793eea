"""Build libart.so (the HIP library behind include/art.h) for gfx950.

    python -m paper_2606_00024_amd.build

The library is built in-tree (paper_2606_00024_amd/libart.so) with hipcc.
All HIP code is compiled without packed-fp32 instructions and without
floating-point contraction (fused multiply-adds are written explicitly where
they are wanted), so that every code path that merges softmax states
produces the same bits.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libart.so")
# read-only streaming kernels for the benchmark's measured read ceiling
BENCH_LIB = os.path.join(HERE, "libart_bench.so")
BENCH_SOURCES = ["art_read_peak.hip"]
# the race-stress test build: the same library with seeded delays at every
# hand-over between workgroups (ART_RACE_STRESS), loaded only by its test
STRESS_LIB = os.path.join(HERE, "libart_stress.so")
SOURCES = ["art_kernels.hip", "art_lists.hip", "art_static.hip", "art_api.cpp"]
ARCH = os.environ.get("ART_OFFLOAD_ARCH", "gfx950")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def flags(extra=()) -> list[str]:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
            "-ffp-contract=off",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
            f"-I{INCLUDE}", f"-I{CSRC}", *extra]


def build(verbose: bool = False, extra=()) -> str:
    """Compile every source and link libart.so, libart_bench.so and the
    race-stress build libart_stress.so (always rebuilds)."""
    _link(LIB, SOURCES, verbose, extra)
    _link(BENCH_LIB, BENCH_SOURCES, verbose, extra)
    _link(STRESS_LIB, SOURCES, verbose, (*extra, "-DART_RACE_STRESS"))
    return LIB


def _link(lib: str, sources, verbose: bool, extra) -> None:
    cc = hipcc()
    tmp = lib + ".tmp"
    cmd = [cc, *flags(extra), "-shared", "-o", tmp] + [os.path.join(CSRC, s) for s in sources]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines()
                    if "packed-fp32-ops" not in l)  # host pass does not know the feature
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{out}")
    if verbose and out.strip():
        print(out)
    os.replace(tmp, lib)


def resource_usage() -> str:
    """Per-kernel register/LDS/scratch report of the device code."""
    cc = hipcc()
    cmd = [cc, *flags(), "--cuda-device-only", "-c", "-o", os.devnull,
           "-Rpass-analysis=kernel-resource-usage", os.path.join(CSRC, "art_kernels.hip")]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    return res.stdout


if __name__ == "__main__":
    if "--usage" in sys.argv:
        print(resource_usage())
    else:
        print(build(verbose=True))
