"""Build the UnionSparse shared library in-tree for gfx950.

    python -m paper_2608_09291_amd.build

compiles ``csrc/*.hip`` with hipcc (gfx950 only, packed FP32 instructions
disabled, kernel arguments preloaded into scalar registers, iterative ILP
scheduling) and
``csrc/*.cpp`` with g++, and links ``libunionsparse.so`` next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libunionsparse.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Kernel-argument preloading: the leading argument dwords of every kernel
# arrive in scalar registers at wavefront start (the SpMM kernel orders its
# arguments for it).
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-fno-strict-aliasing",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-mllvm", "-amdgpu-kernarg-preload-count=16",
             "-I", INCLUDE]
# The iterative ILP scheduling strategy measured 0-3 % faster than the
# default on the SpMM workloads with rows in stored order, 4- and 2-bit. The
# kernels above 16 columns with 8-LT chunks (us_spmm_wide8.hip) keep the
# default, with which they fit the registers of four wavefronts per SIMD,
# and so do the row-reordered ones up to 16 columns (us_spmm_perm.hip),
# which measured 1 % slower with it.
DEFAULT_SCHED_UNITS = ("us_spmm_wide8.hip", "us_spmm_perm.hip")


def hip_flags(source: str) -> list:
    """hipcc flags for one csrc/*.hip file (without -c/-o)."""
    sched = [] if source in DEFAULT_SCHED_UNITS else ["-mllvm", "-amdgpu-sched-strategy=iterative-ilp"]
    return HIP_FLAGS + sched
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-fno-strict-aliasing", "-Wall", "-I", INCLUDE]


def _sources():
    hip = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    cpp = sorted(f for f in os.listdir(CSRC) if f.endswith(".cpp"))
    return hip, cpp


def _compile(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("compile failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r.stderr


def build(verbose: bool = False) -> str:
    """Compile every source and link the library; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    hip, cpp = _sources()
    jobs = []
    for f in hip:
        obj = os.path.join(BUILD, f + ".o")
        jobs.append((obj, [HIPCC, *hip_flags(f), "-c", os.path.join(CSRC, f), "-o", obj]))
    for f in cpp:
        obj = os.path.join(BUILD, f + ".o")
        jobs.append((obj, ["g++", *CXX_FLAGS, "-c", os.path.join(CSRC, f), "-o", obj]))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        logs = list(ex.map(lambda j: _compile(j[1]), jobs))
    if verbose:
        for (obj, cmd), log in zip(jobs, logs):
            print(" ".join(cmd))
    tmp = LIB + ".tmp"
    _compile([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *[o for o, _ in jobs],
              "-o", tmp, "-lpthread"])
    os.replace(tmp, LIB)
    return LIB


def clean():
    shutil.rmtree(BUILD, ignore_errors=True)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
