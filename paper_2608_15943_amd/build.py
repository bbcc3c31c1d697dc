"""Build the HIP library libkvpipe.so in-tree for gfx950.

    python -m paper_2608_15943_amd.build

HIP sources go through hipcc (--offload-arch=gfx950); the planner is plain
host C++ built by g++ with -ffp-contract=off and no fast-math, so its double
arithmetic rounds exactly as written.  Objects land in ``_build/`` and the
library in ``paper_2608_15943_amd/lib/``.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libkvpipe.so")
# Device filler of the seeded input generator (its own library: not the method).
INPUTS_SRC = os.path.join(ROOT, "kvp_inputs", "fill.hip")
INPUTS_LIB = os.path.join(ROOT, "kvp_inputs", "libkvp_inputs.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall",
             "-Wno-unused-result"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-fast-math", "-I", INCLUDE,
              "-I", CSRC, "-Wall"]

HIP_SOURCES = ["gemm_bf16.hip", "flash_prefill.hip", "decode_attn.hip", "decode_gemm.hip",
               "small_kernels.hip", "calib.hip", "attn_bwd.hip", "bwd_f32.hip", "noalloc.hip"]
HIP_HOST_SOURCES = ["runtime.cpp"]   # host code that calls the HIP runtime
HOST_SOURCES = ["planner.cpp", "pager.cpp"]   # pure host C++, no HIP


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    jobs = []
    for s in HIP_SOURCES:
        jobs.append([HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, s), "-o",
                     os.path.join(BUILD, s + ".o")])
    for s in HIP_HOST_SOURCES:
        jobs.append([HIPCC, "-O2", "-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC, "-Wall", "-c",
                     os.path.join(CSRC, s), "-o", os.path.join(BUILD, s + ".o")])
    for s in HOST_SOURCES:
        jobs.append(["g++", *HOST_FLAGS, "-c", os.path.join(CSRC, s), "-o",
                     os.path.join(BUILD, s + ".o")])
    workers = max(1, min(len(jobs), int(os.environ.get("MAX_JOBS", "8"))))
    with cf.ThreadPoolExecutor(workers) as ex:
        for r in ex.map(_run, jobs):
            if verbose and (r.stdout or r.stderr):
                print(r.stdout, r.stderr, file=sys.stderr)
    objs = [os.path.join(BUILD, s + ".o") for s in HIP_SOURCES + HIP_HOST_SOURCES + HOST_SOURCES]
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    tmp = INPUTS_LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-shared", "-o", tmp, INPUTS_SRC])
    os.replace(tmp, INPUTS_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
