"""Build libeahr.so in-tree: gfx950 HIP kernels plus the host runtime.

Usage: ``python -m paper_2608_07152_amd.build`` (or ``build()`` from Python).
Every HIP source is compiled without fp contraction (the interval arithmetic
is specified one rounding per operation) and without packed-fp32 ops.
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
OUT = os.path.join(HERE, "libeahr.so")
BUILD_DIR = os.path.join(ROOT, "_build")

HIP_SOURCES = ["pvs_kernels.hip", "pvs_scan.hip", "pvs_rank.hip", "pvs_noalloc.hip", "pbm_gpu.hip"]
HOST_SOURCES = ["pvs_api.cpp", "pvs_merge.cpp", "pbm.cpp", "eahr.cpp", "errors.cpp"]

ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")
ARCH = os.environ.get("EAHR_OFFLOAD_ARCH", "gfx950")


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd):
    print("+", " ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = True) -> str:
    """Compile every source and link ``libeahr.so``; returns its path."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    common = ["-O3", "-fPIC", "-std=c++17", "-I", INCLUDE, "-I", CSRC, "-ffp-contract=off",
              "-Wall", "-Wno-unused-function", "-pthread"]
    objs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        _run([hipcc, "-c", "-x", "hip", f"--offload-arch={ARCH}", *common,
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              "-fno-gpu-rdc",
              os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        _run([hipcc, "-c", "-x", "c++", "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE, *common,
              os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    tmp = OUT + ".tmp"
    _run([hipcc, "-shared", f"--offload-arch={ARCH}", "-pthread", "-o", tmp, *objs])
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    build()
    sys.exit(0)
