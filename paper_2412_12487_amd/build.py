"""Build libecho.so (HIP kernels for gfx950 + host loader) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libecho.so")
ARCH = "gfx950"

# -packed-fp32-ops: keep the compiler from emitting packed FP32 VALU forms.
# atomic optimizer off: the kernels' same-address atomics already come from one lane
# (arrival counts), and the optimizer's lane-count prologue only lengthens the barrier path.
DEVICE_FLAGS = ["--offload-arch=" + ARCH, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I", INCLUDE, "-I", CSRC]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = False) -> str:
    """Compile every source and link libecho.so; always rebuilds."""
    os.makedirs(BUILD, exist_ok=True)
    kobj = os.path.join(BUILD, "echo_kernels.o")
    hobj = os.path.join(BUILD, "echo_host.o")
    _run(["hipcc", "-c", *DEVICE_FLAGS, *COMMON, os.path.join(CSRC, "echo_kernels.hip"), "-o", kobj], verbose)
    _run(["hipcc", "-c", *COMMON, os.path.join(CSRC, "echo_host.cpp"), "-o", hobj], verbose)
    tmp = LIB + ".tmp"
    _run(["hipcc", "-shared", "-fPIC", "--offload-arch=" + ARCH, kobj, hobj, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
