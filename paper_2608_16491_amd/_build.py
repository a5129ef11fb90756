"""Compile the HIP library ``libfrog.so`` for gfx950, in-tree.

Host C++ (index construction) is compiled with g++ (no FMA contraction, so
the construction's distances keep their documented rounding); the C-ABI and
the kernels with hipcc for ``--offload-arch=gfx950``.  Device code is built
with packed-FP32 instructions disabled.
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
OBJ = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libfrog.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

HOST_SOURCES = ["build_index.cpp"]
HIP_SOURCES = ["capi.cpp", "search.hip", "search_shared.hip", "search_scan.hip", "search_pool.hip", "search_trav.hip",
               "exact.hip", "bruteforce.hip", "build_gpu.hip"]

DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def _compile_one(src, obj, verbose):
    path = os.path.join(CSRC, src)
    if src in HOST_SOURCES:
        cmd = ["g++", "-O3", "-std=c++17", "-fPIC", "-mavx2", "-ffp-contract=off", "-fno-fast-math",
               "-pthread", "-Wall", f"-I{INCLUDE}", f"-I{CSRC}", "-c", path, "-o", obj]
    else:
        cmd = [HIPCC, "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", *DEVICE_FLAGS,
               "-ffp-contract=off", "-Wall", "-Wno-unused-result",
               f"-I{INCLUDE}", f"-I{CSRC}", "-c", path, "-o", obj]
        if src.endswith(".cpp"):
            cmd[1:1] = ["-x", "hip"]
    _run(cmd, verbose)


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source (always) and link libfrog.so; returns its path."""
    os.makedirs(OBJ, exist_ok=True)
    objs = []
    procs = []
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        for src in HOST_SOURCES + HIP_SOURCES:
            obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
            objs.append(obj)
            procs.append(ex.submit(_compile_one, src, obj, verbose))
        for p in procs:
            p.result()
    tmp = LIB + f".tmp{os.getpid()}"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs, "-pthread"], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
