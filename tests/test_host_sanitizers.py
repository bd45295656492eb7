"""The host-side schedule generator and cost model under AddressSanitizer and
UndefinedBehaviorSanitizer, CPU only: tests/c/plan_sweep.cpp, built with g++ against plan.cpp
and cost.cpp (plain C++, no GPU), builds plans for about 900 ring and torus requests in every
variant and placement, calls every host entry point on every pass, collective and block, and the
documented error paths. Any sanitizer report aborts the run and fails the test."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_17254_amd", "csrc")


def test_plan_sweep_under_sanitizers(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not found")
    exe = str(tmp_path / "plan_sweep")
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer", "-I", CSRC, "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "plan_sweep.cpp"),
                    os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "cost.cpp"), "-o", exe],
                   check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-4000:]
    assert "0 failures" in res.stdout
