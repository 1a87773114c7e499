"""Build of the gfx950 shared library ``libflashrestore.so`` (in-tree), and of
``libfrceil.so``, the plain streaming kernels the benchmark measures the
chip's copy and read ceilings with (not part of the library).

One hipcc invocation per library compiles the host sources and the kernels
for gfx950 only.  Packed fp32 instructions are disabled for all device code.
"""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libflashrestore.so")
SOURCES = ["plan.cpp", "api.cpp", "steptag.cpp", "layout.cpp", "kernels.hip"]
CEIL_LIB = os.path.join(PKG, "libfrceil.so")
CEIL_SOURCES = ["ceilings.hip"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def hipcc_command(out: str = LIB, extra=(), sources=SOURCES):
    return [
        os.path.join(ROCM, "bin", "hipcc"),
        "--offload-arch=gfx950",
        "-O3",
        "-std=c++17",
        "-fPIC",
        "-shared",
        "-Wall",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", os.path.join(ROOT, "include"),
        *[os.path.join(CSRC, s) for s in sources],
        "-o", out,
        f"-Wl,-rpath,{ROCM}/lib",
        *extra,
    ]


# The library's host code exports only what include/flashrestore.h declares
# (its declarations sit in a default-visibility region); device code is
# compiled as before.
LIB_EXTRA = ("-Xarch_host", "-fvisibility=hidden")


def build(verbose: bool = False) -> str:
    for lib, sources, extra in ((LIB, SOURCES, LIB_EXTRA), (CEIL_LIB, CEIL_SOURCES, ())):
        tmp = lib + ".tmp"
        cmd = hipcc_command(tmp, extra=extra, sources=sources)
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(tmp, lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
