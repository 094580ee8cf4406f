"""Compile the HIP sources of the package into ``libkrpe.so`` (gfx950).

    python -m paper_2106_12566_amd.build          # or: python paper_2106_12566_amd/build.py

The library is built in-tree, next to this file, so that it travels with the
source tree.  Packed-FP32 instruction selection is disabled for all device
code (``-packed-fp32-ops``).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libkrpe.so")
SOURCES = [os.path.join(HERE, "csrc", "kernels.hip"), os.path.join(HERE, "csrc", "grad_bias.hip"),
           os.path.join(HERE, "csrc", "long_seq.hip"), os.path.join(HERE, "csrc", "api.hip")]
# The convolution kernel at N = 16384, compiled on its own with LLVM's
# maximum-ILP machine scheduler (measured faster for that length only).
TOP = os.path.join(HERE, "csrc", "conv_top.hip")
TOP_FLAGS = ["-mllvm", "-amdgpu-sched-strategy=max-ilp"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the ROCm toolchain is required to build libkrpe.so")


def _flags() -> list[str]:
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-Wno-unused-function",
        "-I", os.path.join(ROOT, "include"),
    ]


def command(out: str = LIB, top: str = TOP) -> list[str]:
    """One hipcc run linking every source (`top`: conv_top.hip, or its object built by
    top_command) into `out`."""
    # (the object goes first: hipcc marks every input after a .hip file as HIP source)
    return [hipcc(), *_flags(), "-shared", "-o", out, top, *SOURCES]


def top_command(obj: str) -> list[str]:
    return [hipcc(), *_flags(), *TOP_FLAGS, "-c", "-o", obj, TOP]


def _run(cmd: list[str], verbose: bool) -> None:
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stdout}\n{res.stderr}")


def build(verbose: bool = False) -> str:
    """Compile libkrpe.so (always recompiles); return its path."""
    tmp, obj = LIB + ".tmp", LIB + ".top.o"
    _run(top_command(obj), verbose)
    _run(command(tmp, obj), verbose)
    os.remove(obj)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-q" not in sys.argv))
