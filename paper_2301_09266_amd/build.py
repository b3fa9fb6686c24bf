"""Build the HIP library in-tree for gfx950: paper_2301_09266_amd/csrc/libfinc.so.

finc.hip compiles as several translation units in parallel (FINC_PART: one
per group of inverse kernel instances, and one with everything else), flow.hip
as one more; all are linked into the one shared library.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "finc.hip")
FLOW_SRC = os.path.join(PKG, "csrc", "flow.hip")
BACKWARD_SRC = os.path.join(PKG, "csrc", "backward.hip")
LIB = os.path.join(PKG, "csrc", "libfinc.so")
CALIB_SRC = os.path.join(PKG, "csrc", "calib.hip")
CALIB_LIB = os.path.join(PKG, "csrc", "libfinc_calib.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

ARCH = "--offload-arch=gfx950"
FLAGS = [
    ARCH, "-O3", "-std=c++17", "-fPIC",
    # packed fp32 VALU ops stay off: plain fp32 FMAs only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-const-variable",
]
INVERSE_GROUPS = 18   # kInverseGroups in finc.hip


def _jobs() -> int:
    for var in ("MAX_JOBS", "CMAKE_BUILD_PARALLEL_LEVEL"):
        if os.environ.get(var, "").isdigit() and int(os.environ[var]) > 0:
            return min(int(os.environ[var]), 16)
    return max(1, min(os.cpu_count() or 1, 16))


def build(out: str = LIB, extra: list[str] | None = None) -> str:
    """Compile every part of finc.hip and link them into `out`."""
    tmpdir = tempfile.mkdtemp(prefix="finc_build_")
    try:
        # finc.hip in parts (FINC_PART), then flow.hip and backward.hip
        parts = [-2] + list(range(INVERSE_GROUPS)) + [FLOW_SRC, BACKWARD_SRC]
        objs = [os.path.join(tmpdir, f"part{i}.o") for i in range(len(parts))]

        def compile_part(i: int) -> None:
            src, defs = ((parts[i], []) if isinstance(parts[i], str)
                         else (SRC, [f"-DFINC_PART={parts[i]}"]))
            cmd = [HIPCC, *FLAGS, *(extra or []), *defs,
                   "-I", os.path.join(ROOT, "include"), "-c", "-o", objs[i], src]
            subprocess.run(cmd, check=True)

        with concurrent.futures.ThreadPoolExecutor(_jobs()) as pool:
            for f in [pool.submit(compile_part, i) for i in range(len(parts))]:
                f.result()
        tmp = out + ".tmp"
        subprocess.run([HIPCC, ARCH, "-shared", "-fPIC", "-o", tmp, *objs], check=True)
        os.replace(tmp, out)
        # the benchmark's measurement kernels, a library of their own
        if out == LIB:
            tmp = CALIB_LIB + ".tmp"
            subprocess.run([HIPCC, *FLAGS, "-shared", "-o", tmp, CALIB_SRC], check=True)
            os.replace(tmp, CALIB_LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return out


if __name__ == "__main__":
    print(build())
