"""Compile libwino.so for gfx950 in-tree with hipcc.

The library is C++/HIP only (no torch headers); it is loaded through ctypes
by ``paper_1611_06565_amd.wino``.  Its translation units (the host-side
planner, the entry points and one unit per size family of kernels) compile
in parallel, then link into one shared object.
"""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libwino.so")
SOURCES = ["plan.cpp", "wino.hip", "sizes_m2.hip", "sizes_f42.hip", "sizes_f43.hip", "fused_f43.hip", "sizes_f54.hip",
           "sizes_f45.hip", "sizes_f36.hip", "sizes_f32.hip", "sizes_ax.hip", "sizes_a8.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX", "g++")

FLAGS = [
    "-std=c++20", "--offload-arch=gfx950", "-O3", "-fPIC",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-pass-failed",
    # the LDS copies set M0 in inline assembly; nothing else in the library uses it
    "-Wno-inline-asm",
]


def _check_kernel_stubs(path):
    """Fail if a kernel's host launch stub is missing.

    clang drops a kernel template's host stub without a diagnostic when its
    body does not type-check for the host target (a gfx950-only builtin
    operand, say); the library then fails to load with an undefined symbol.
    """
    res = subprocess.run(["nm", "-u", path], capture_output=True, text=True)
    if res.returncode != 0:
        return  # nm unavailable: the load-time check still catches it
    missing = [ln.split()[-1] for ln in res.stdout.splitlines() if "__device_stub__" in ln]
    if missing:
        raise RuntimeError("kernel launch stubs missing from the host pass: " + ", ".join(missing))


def _compile(src, obj, verbose):
    if src.endswith(".hip"):
        cmd = [HIPCC] + FLAGS + ["-I" + INCLUDE, "-I" + CSRC, "-c", src, "-o", obj]
    else:
        # the host-side planner is plain C++ (no device code)
        cmd = [CXX, "-std=c++20", "-O2", "-fPIC", "-Wall", "-Wextra", "-I" + INCLUDE, "-I" + CSRC,
               "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {os.path.basename(src)}:\n" + res.stdout + res.stderr)


def build(verbose=False, jobs=None):
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    tmpdir = tempfile.mkdtemp(prefix=".libwino.", dir=HERE)
    objs = [os.path.join(tmpdir, os.path.basename(s) + ".o") for s in srcs]
    tmp = os.path.join(tmpdir, "libwino.so")
    try:
        jobs = jobs or min(len(srcs), max(1, os.cpu_count() or 1))
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            for f in [ex.submit(_compile, s, o, verbose) for s, o in zip(srcs, objs)]:
                f.result()
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("link failed:\n" + res.stdout + res.stderr)
        _check_kernel_stubs(tmp)
        os.replace(tmp, LIB)
    finally:
        for f in objs + [tmp]:
            if os.path.exists(f):
                os.unlink(f)
        os.rmdir(tmpdir)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
