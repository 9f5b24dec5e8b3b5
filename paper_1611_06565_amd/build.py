"""Compile libwino.so for gfx950 in-tree with hipcc.

The library is C++/HIP only (no torch headers); it is loaded through ctypes
by ``paper_1611_06565_amd.wino``.
"""
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libwino.so")
SOURCES = ["wino.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "-std=c++20", "--offload-arch=gfx950", "-O3", "-fPIC", "-shared",
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


def build(verbose=False):
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    fd, tmp = tempfile.mkstemp(prefix=".libwino.", suffix=".so", dir=HERE)
    os.close(fd)
    cmd = [HIPCC] + FLAGS + ["-I" + INCLUDE, "-I" + CSRC] + srcs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    try:
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
        _check_kernel_stubs(tmp)
        os.replace(tmp, LIB)
    finally:
        if os.path.exists(tmp):
            os.unlink(tmp)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
