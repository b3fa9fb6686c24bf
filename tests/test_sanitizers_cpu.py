"""The C on the CPU under AddressSanitizer and UndefinedBehaviorSanitizer:
the oracle (gcc) and the library's host side -- argument checks, plan
queries, workspace sizes -- (hipcc, sanitizers on the host pass only).

The host-side build compiles the HIP sources with --offload-host-only: no
device code is built, the kernels' registration records point at no code
object, and the driver makes no call that reaches a launch (each call it
makes is host arithmetic or is rejected before any HIP call), so nothing
ever needs one.  The drivers are tests/sanitize/*.c*: every buffer they pass
has exactly the size the documented layout gives."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(exe, env):
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, f"{exe} failed ({r.returncode}):\n{r.stderr[-4000:]}"
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    return r.stdout


def test_oracle_under_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_drive")
    subprocess.run(["gcc", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "tests", "sanitize", "oracle_drive.c"),
                    os.path.join(ROOT, "oracle", "finc_oracle.c"), "-lm", "-o", exe],
                   check=True)
    out = _run(exe, dict(SAN_ENV, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1"))
    assert "all calls returned 0" in out


def test_host_side_under_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not found")
    san = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined".split()
    flags = ["--offload-arch=gfx950", "--offload-host-only", "-O1", "-g", "-std=c++17",
             "-fPIC", *san, *"-Xarch_host -fno-sanitize-recover=all".split(),
             "-I", os.path.join(ROOT, "include")]
    csrc = os.path.join(ROOT, "paper_2301_09266_amd", "csrc")
    srcs = [os.path.join(csrc, f) for f in ("finc.hip", "flow.hip", "backward.hip")]
    srcs.append(os.path.join(ROOT, "tests", "sanitize", "host_drive.cpp"))
    procs, objs = [], []
    for src in srcs:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", src, "-o", obj],
                                      stderr=subprocess.PIPE, text=True))
    for p in procs:
        err = p.communicate()[1]
        assert p.returncode == 0, err[-4000:]
    exe = str(tmp_path / "host_drive")
    # the registration records name code objects that a host-only build
    # does not make: left unresolved, never used
    subprocess.run([HIPCC, "--offload-arch=gfx950", *san, *objs,
                    "-Wl,--unresolved-symbols=ignore-all", "-o", exe], check=True)
    # the HIP runtime keeps allocations until exit: leaks are not checked here
    out = _run(exe, dict(SAN_ENV, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1"))
    assert "all checks held" in out
