"""Build libart.so (the HIP library behind include/art.h) for gfx950.

    python -m paper_2606_00024_amd.build

The library is built in-tree (paper_2606_00024_amd/libart.so) with hipcc.
All HIP code is compiled without packed-fp32 instructions and without
floating-point contraction (fused multiply-adds are written explicitly where
they are wanted), so that every code path that merges softmax states
produces the same bits.

Besides the product library, the build links three test and measurement
builds of the same sources:
  libart_bench.so   read-only streaming kernels (the benchmark's measured
                    read ceiling; not part of the decode path)
  libart_stress.so  the library with ART_RACE_STRESS: seeded delays at every
                    hand-over between workgroups (the race-stress test)
  libart_asan.so    the library with its host code (art_api.cpp) compiled by
                    g++ with AddressSanitizer; the device code is the same
                    (the host-ASan test runs the CPU suite against it)
Objects go to _build/ and the sources compile in parallel.
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
OBJ = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libart.so")
BENCH_LIB = os.path.join(HERE, "libart_bench.so")
STRESS_LIB = os.path.join(HERE, "libart_stress.so")
ASAN_LIB = os.path.join(HERE, "libart_asan.so")
ARCH = os.environ.get("ART_OFFLOAD_ARCH", "gfx950")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

DEVICE_SOURCES = ["art_kernels.hip", "art_lists.hip", "art_static.hip"]
HOST_SOURCE = "art_api.cpp"
SOURCES = DEVICE_SOURCES + [HOST_SOURCE]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), os.path.join(ROCM, "bin", "hipcc"), shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def flags(extra=()) -> list[str]:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
            "-ffp-contract=off",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
            f"-I{INCLUDE}", f"-I{CSRC}", *extra]


def _asan_host_flags() -> list[str]:
    """g++ flags for the host code with AddressSanitizer (the HIP runtime's
    host API headers need the platform macro when not compiled by hipcc)."""
    return ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-fno-omit-frame-pointer",
            "-fsanitize=address", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
            f"-I{INCLUDE}", f"-I{CSRC}", "-Wall", "-Wno-unused-function"]


def _quiet(text: str) -> str:
    # the host pass does not know the packed-fp32 feature flag
    return "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)


def _run_all(jobs, verbose):
    """Run (name, cmd) jobs in parallel; raise with the output of a failure."""
    procs = []
    for name, cmd in jobs:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((name, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                             text=True)))
    errors = []
    for name, p in procs:
        out, _ = p.communicate()
        out = _quiet(out)
        if p.returncode != 0:
            errors.append(f"{name} failed ({p.returncode}):\n{out}")
        elif verbose and out.strip():
            print(out)
    if errors:
        raise RuntimeError("\n".join(errors))


def _obj(name: str) -> str:
    return os.path.join(OBJ, name + ".o")


def build(verbose: bool = False, extra=()) -> str:
    """Compile every source and link libart.so and the three test and
    measurement builds (always rebuilds)."""
    os.makedirs(OBJ, exist_ok=True)
    cc = hipcc()
    src = lambda s: os.path.join(CSRC, s)
    jobs = [(s, [cc, *flags(extra), "-c", "-o", _obj(s), src(s)]) for s in SOURCES]
    jobs.append(("art_kernels.hip (stress)", [cc, *flags(extra), "-DART_RACE_STRESS", "-c",
                                              "-o", _obj("art_kernels_stress"), src("art_kernels.hip")]))
    jobs.append(("art_read_peak.hip", [cc, *flags(extra), "-c", "-o", _obj("art_read_peak.hip"),
                                       src("art_read_peak.hip")]))
    jobs.append(("art_api.cpp (asan)", [*_asan_host_flags(), "-c", "-o", _obj("art_api_asan"),
                                        src(HOST_SOURCE)]))
    _run_all(jobs, verbose)
    dev = [_obj(s) for s in DEVICE_SOURCES]
    links = {
        LIB: dev + [_obj(HOST_SOURCE)],
        STRESS_LIB: [_obj("art_kernels_stress")] + dev[1:] + [_obj(HOST_SOURCE)],
        BENCH_LIB: [_obj("art_read_peak.hip")],
        # the AddressSanitizer runtime is not linked in: the process that
        # loads this library preloads gcc's libasan (tests/test_host_asan.py)
        ASAN_LIB: dev + [_obj("art_api_asan")],
    }
    _run_all([(os.path.basename(lib), [cc, f"--offload-arch={ARCH}", "-shared", "-o", lib + ".tmp", *objs])
              for lib, objs in links.items()], verbose)
    for lib in links:
        os.replace(lib + ".tmp", lib)
    return LIB


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
