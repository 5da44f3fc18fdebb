"""Build libnsgcqt.so in-tree for gfx950.

The host plan builder is plain C++ (g++); the kernels and the C ABI are HIP
(hipcc). Every HIP translation unit is compiled with packed-FP32 instructions
disabled. Usage: ``python -m paper_2609_29119_amd.build`` or ``build()``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libnsgcqt.so")
ARCH = os.environ.get("NSGCQT_ARCH", "gfx950")

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument", "-Wno-gnu-zero-variadic-macro-arguments",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd[:3])} ...")
    return r


def build(verbose: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    os.makedirs(BUILD, exist_ok=True)
    _run([sys.executable, os.path.join(CSRC, "gen_radix_consts.py"), os.path.join(CSRC, "radix_consts.hpp")],
         verbose)
    plan_o = os.path.join(BUILD, "plan.o")
    hip_o = os.path.join(BUILD, "nsgcqt.o")
    _run(["g++", "-O2", "-std=c++17", "-fPIC", "-Wall", "-c",
          os.path.join(CSRC, "plan.cpp"), "-o", plan_o], verbose)
    _run([hipcc, *HIP_FLAGS, "-c", os.path.join(CSRC, "nsgcqt.hip"), "-o", hip_o], verbose)
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, plan_o, hip_o], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
