"""Host code under the address and undefined-behaviour sanitizers (CPU only).

Two drivers are built with gcc / g++ and run in a subprocess:
  * tests/sanitize/host_plan_check.cpp with paper_2609_12399_amd/csrc/host_plan.cpp:
    the library's configuration, workspace-layout, selection-plan and per-step
    protocol checks (the host validation every entry point runs before it
    enqueues anything), over grids of valid and invalid arguments and a long
    random walk of protocol calls;
  * tests/sanitize/oracle_check.c with oracle/gdn_oracle.c: the fp64 oracle's
    prefill, ancestry and decode on small random problems with exactly sized
    buffers, including the rejected-argument paths.
Any out-of-bounds access, use after free, leak or undefined behaviour aborts
the driver (-fno-sanitize-recover=all), which fails the test.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]


def _build_and_run(tmp_path, compiler, std, sources, extra=()):
    if shutil.which(compiler) is None:
        pytest.skip(f"{compiler} not available")
    exe = str(tmp_path / "driver")
    cmd = [compiler, f"-std={std}", *SAN, *[os.path.join(ROOT, s) for s in sources],
           *extra, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"build failed:\n{r.stderr}"
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, f"driver failed ({r.returncode}):\n{r.stdout}\n{r.stderr[-4000:]}"
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr
    return r.stdout


def test_host_plan_checks_under_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, "g++", "c++17",
                         ["tests/sanitize/host_plan_check.cpp",
                          "paper_2609_12399_amd/csrc/host_plan.cpp"])
    assert "host plan checks: ok" in out


def test_oracle_under_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, "gcc", "c11",
                         ["tests/sanitize/oracle_check.c", "oracle/gdn_oracle.c"], ["-lm"])
    assert "oracle checks: ok" in out
