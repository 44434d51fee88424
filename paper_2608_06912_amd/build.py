"""Build liblapsum.so in-tree with hipcc for gfx950.

    python -m paper_2608_06912_amd.build          # or __graft_entry__.build()

Every HIP source is compiled for gfx950 only, with packed-FP32 instructions
disabled (-target-feature -packed-fp32-ops); the host orchestration is
compiled without floating-point contraction so that the bracket ranks are
evaluated exactly as written.  Objects go to _build/ next to this file and
the library to liblapsum.so beside it.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "liblapsum.so")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")

HIP_SOURCES = ["row_kernels.hip", "stream_kernels.hip", "sort_kernels.hip",
               "solve_kernels.hip", "bracket_kernels.hip", "band_kernels.hip", "bucket_solve.hip",
               "comparator_kernels.hip", "noalloc.hip"]
HOST_SOURCES = ["lapsum_api.cpp"]

ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}"]
HIP_FLAGS = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_FLAGS = ["-x", "c++", "-ffp-contract=off", "-D__HIP_PLATFORM_AMD__"]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the LapSum library)")


def _compile(args):
    cmd, src = args
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        err = "\n".join(l for l in proc.stderr.splitlines() if "packed-fp32-ops" not in l)
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{err}")
    return src


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every source and link liblapsum.so; returns the library path."""
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    work = []
    objs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        objs.append(obj)
        work.append(([hipcc, *COMMON, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj], src))
    rocm_inc = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(hipcc))), "include")
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        objs.append(obj)
        work.append(([hipcc, *COMMON, *HOST_FLAGS, f"-I{rocm_inc}", "-c", os.path.join(CSRC, src),
                      "-o", obj], src))
    jobs = jobs or min(len(work), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for src in ex.map(_compile, work):
            if verbose:
                print(f"compiled {src}", flush=True)
    tmp = LIB + ".tmp"
    link = [hipcc, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    proc = subprocess.run(link, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError(f"linking failed:\n{' '.join(link)}\n{proc.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}", flush=True)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
