"""Build of the gfx950 shared library ``libflashrestore.so`` (in-tree).

One hipcc invocation compiles the host sources and the kernels for gfx950
only.  Packed fp32 instructions are disabled for all device code.
"""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libflashrestore.so")
SOURCES = ["plan.cpp", "api.cpp", "steptag.cpp", "layout.cpp", "kernels.hip"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def hipcc_command(out: str = LIB, extra=()):
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
        *[os.path.join(CSRC, s) for s in SOURCES],
        "-o", out,
        f"-Wl,-rpath,{ROCM}/lib",
        *extra,
    ]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = hipcc_command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
