"""Build libvp.so (host planner + gfx950 kernels) in-tree with hipcc.

    python -m paper_2604_16893_amd.build

The kernel source is compiled as KERNEL_PARTS translation units in parallel
(each one a share of the streaming kernels' template shapes, selected with
-DVP_PART), next to the host planner, and the objects are linked into one
shared library.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libvp.so")
API_SRC = os.path.join(CSRC, "vp_api.cpp")
KERNEL_SRC = os.path.join(CSRC, "vp_kernels.hip")
SOURCES = [API_SRC, KERNEL_SRC]
ARCH = "gfx950"
KERNEL_PARTS = 8

# Packed FP32 instructions are disabled for all device code: plain float
# code is compiled to scalar v_fma_f32 / v_add_f32 only.
# Common-code sinking is off: it would merge the streaming kernel's
# per-slot close paths (each naming its own accumulator registers) into one
# path over copied registers.
# Regions whose branches are uniform (scalar) are left unstructured: the
# hardware branches on them directly, and structurizing them inserts flow
# blocks whose merges the register allocator resolves by copying every
# accumulator slot out and back at each closed row (about 7% of the
# 720p -> 256x448 workload's time, 12% of the mixed batch's).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-simplifycfg-sink-common=false",
                "-mllvm", "-structurizecfg-skip-uniform-regions=true"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def _common() -> list:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++20", "-fPIC", "-Wall",
            "-I", os.path.join(ROOT, "include"), "-I", CSRC, *DEVICE_FLAGS]


def compile_commands(objdir: str) -> list:
    """(command, object) pairs: the host planner and every kernel part."""
    cmds = [([hipcc(), *_common(), "-c", "-o", os.path.join(objdir, "vp_api.o"), API_SRC],
             os.path.join(objdir, "vp_api.o"))]
    for k in range(KERNEL_PARTS):
        obj = os.path.join(objdir, f"vp_kernels_{k}.o")
        cmds.append(([hipcc(), *_common(), f"-DVP_PART={k}", f"-DVP_PARTS={KERNEL_PARTS}",
                      "-c", "-o", obj, KERNEL_SRC], obj))
    return cmds


def link_command(objs: list, out: str) -> list:
    return [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out, *objs]


def command(out: str = LIB) -> list:
    """The equivalent single-command build (one translation unit, serial)."""
    return [hipcc(), *_common(), "-shared", "-o", out, *SOURCES]


def build(verbose: bool = False, jobs: int | None = None) -> str:
    objdir = tempfile.mkdtemp(prefix="vp_build_")
    try:
        cmds = compile_commands(objdir)
        jobs = jobs or min(len(cmds), max(1, min(16, os.cpu_count() or 1)))
        with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
            futs = []
            for cmd, _ in cmds:
                if verbose:
                    print(" ".join(cmd), flush=True)
                futs.append(ex.submit(subprocess.run, cmd, capture_output=True, text=True))
            for f, (cmd, _) in zip(futs, cmds):
                r = f.result()
                if r.stdout or r.stderr:
                    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                                    if "packed-fp32-ops" not in l and l.strip())
                    if msg:
                        print(msg, file=sys.stderr, flush=True)
                if r.returncode != 0:
                    raise subprocess.CalledProcessError(r.returncode, cmd)
        tmp = LIB + ".tmp"
        link = link_command([o for _, o in cmds], tmp)
        if verbose:
            print(" ".join(link), flush=True)
        subprocess.check_call(link)
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(objdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    sys.exit(0)
