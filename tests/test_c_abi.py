"""The C ABI from C: tests/c_abi/host_calls.c compiles against include/wino.h
as strict C99, links libwino.so and runs its host-side checks (no GPU)."""
import os
import shutil
import subprocess

import pytest

import paper_1611_06565_amd.wino as wino

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_c99_client(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    lib = wino.library_path()
    assert os.path.exists(lib), "libwino.so is not built"
    exe = tmp_path / "host_calls"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c_abi", "host_calls.c"),
           "-o", str(exe), lib, "-Wl,-rpath," + os.path.dirname(lib), "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "all host calls ok" in res.stdout
