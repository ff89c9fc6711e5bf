"""Build libsaki.so in-tree for gfx950.

The host calibration (C++17, float64) is compiled with g++ and the HIP
kernels with hipcc; hipcc links both into paper_2608_03228_amd/libsaki.so.
Run ``python -m paper_2608_03228_amd.build`` (or call ``build()``).
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
LIB = os.path.join(PKG, "libsaki.so")
BUILD_DIR = os.path.join(PKG, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed FP32 instructions are disabled for all device code.
NO_PACKED_FP32 = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# MFMA results are written to the architectural VGPRs rather than the
# accumulation registers, which saves a copy of every result the kernels
# inspect (the selection passes read each score).
MFMA_VGPR = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]


def _run(cmd, verbose):
    if verbose:
        print("+", " ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = True) -> str:
    """Compile every source and link libsaki.so; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    host_o = os.path.join(BUILD_DIR, "saki_host.o")
    dev_o = os.path.join(BUILD_DIR, "saki_kernels.o")
    _run(["g++", "-O3", "-std=c++17", "-fPIC", "-march=x86-64-v3", "-pthread",
          "-Wall", "-Wextra", "-I", INCLUDE, "-I", CSRC, "-c",
          os.path.join(CSRC, "saki_host.cpp"), "-o", host_o], verbose)
    _run([HIPCC, "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", *NO_PACKED_FP32, *MFMA_VGPR,
          "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "saki_kernels.hip"),
          "-o", dev_o], verbose)
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-pthread", host_o, dev_o,
          "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


def clean():
    shutil.rmtree(BUILD_DIR, ignore_errors=True)
    if os.path.exists(LIB):
        os.remove(LIB)


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
