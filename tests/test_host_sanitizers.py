"""The library's host code and the oracle under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU.

tests/sanitize/host_checks.cpp drives every host path of the C ABI (the
planner of each entry point, the filter tables, smart_resize, sampling, the
plan cache, the argument checks) and every oracle function over seeded random
and degenerate inputs.  The planner (vp_api.cpp) and the oracle (oracle.c)
are compiled with g++/gcc and both sanitizers, recovery off, so the first
report aborts the run; the kernel file contributes only its host side (the
launchers and shape tables, built as the library builds it; no launcher is
called here).
"""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_16893_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return shutil.which("hipcc")


@pytest.mark.timeout(600)
def test_host_code_and_oracle_under_sanitizers(tmp_path):
    hipcc = _hipcc()
    if hipcc is None or shutil.which("g++") is None or shutil.which("gcc") is None:
        pytest.skip("needs hipcc, g++ and gcc")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    # the kernel file as the library builds it (its launchers are never called here)
    from paper_2604_16893_amd import build as B
    cmds = [[hipcc, *B._common(), f"-DVP_PART={k}", f"-DVP_PARTS={B.KERNEL_PARTS}", "-c", "-o",
             str(tmp_path / f"k{k}.o"), B.KERNEL_SRC] for k in range(B.KERNEL_PARTS)]
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        for r in ex.map(lambda c: subprocess.run(c, capture_output=True, text=True), cmds):
            assert r.returncode == 0, r.stderr[-2000:]
    objs = [c[c.index("-o") + 1] for c in cmds]
    api = str(tmp_path / "vp_api.o")
    subprocess.run(["g++", "-std=c++20", "-O1", "-g", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    *inc, "-c", "-o", api, os.path.join(CSRC, "vp_api.cpp")], check=True)
    orc = str(tmp_path / "oracle.o")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", *SAN, "-ffp-contract=off", "-c", "-o", orc,
                    os.path.join(ROOT, "oracle", "oracle.c")], check=True)
    drv = str(tmp_path / "driver.o")
    subprocess.run(["g++", "-std=c++20", "-O1", "-g", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    *inc, "-c", "-o", drv, os.path.join(ROOT, "tests", "sanitize", "host_checks.cpp")],
                   check=True)
    exe = str(tmp_path / "host_checks")
    subprocess.run(["g++", *SAN, "-o", exe, drv, api, orc, *objs, "-L/opt/rocm/lib", "-lamdhip64", "-lm",
                    "-Wl,-rpath,/opt/rocm/lib"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=500, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert "host checks:" in r.stdout
