"""The host-side planner (paper_1611_06565_amd/csrc/plan.cpp) under the host
sanitizers: tests/host/plan_checks.cpp and the planner are built with g++ and
-fsanitize=address,undefined (every finding aborts) and run on the CPU.  The
checks cover every workload's plan and sizes past every integer range (C or K
of 2^31 - 1, extents, pads and max-pool leads whose products overflow)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1611_06565_amd", "csrc")


def test_planner_under_sanitizers(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("no host C++ compiler")
    exe = tmp_path / "plan_checks"
    cmd = ["g++", "-std=c++20", "-g", "-O1", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-Wall", "-Wextra", "-Werror",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "plan.cpp"), os.path.join(ROOT, "tests", "host", "plan_checks.cpp"),
           "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120, env=env)
    assert res.returncode == 0, res.stdout[-4000:] + res.stderr[-4000:]
    assert "all planner checks ok" in res.stdout
