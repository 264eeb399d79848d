"""Build libvp.so (host planner + gfx950 kernels) in-tree with hipcc.

    python -m paper_2604_16893_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libvp.so")
SOURCES = [os.path.join(CSRC, "vp_api.cpp"), os.path.join(CSRC, "vp_kernels.hip")]
ARCH = "gfx950"

# Packed FP32 instructions are disabled for all device code: plain float
# code is compiled to scalar v_fma_f32 / v_add_f32 only.
# Common-code sinking is off: it would merge the streaming kernel's
# per-slot close paths (each naming its own accumulator registers) into one
# path over copied registers.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-simplifycfg-sink-common=false"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def command(out: str = LIB) -> list:
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++20", "-fPIC", "-shared",
            "-Wall", "-I", os.path.join(ROOT, "include"), "-I", CSRC, *DEVICE_FLAGS,
            "-o", out, *SOURCES]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
