"""CPU oracle for data-parallel replica state restore.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The product library
(``paper_2509_03047_amd``) never imports it, and it imports nothing of the
product except the seeded workload generators, which hold none of the
method's arithmetic.

* ``oracle.cpu``  -- ctypes wrapper of the plain-C oracle ``fr_oracle.c``.
* ``oracle.mini`` -- a second, pure-Python oracle for tiny inputs.

Both follow the same definitions (chunking, FRSUM-128, payload layout,
round-to-nearest-even, unpack and verify); the tests pin them to values
fixed independently of either (worked values, closed forms, exhaustive
comparison with torch's bf16 cast, invariants, brute force).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libfroracle.so")


def build(verbose: bool = False) -> str:
    """Compile the C oracle with gcc (plain -O2, OpenMP)."""
    cmd = [
        "gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra",
        os.path.join(HERE, "fr_oracle.c"), "-o", LIB + ".tmp", "-lm",
    ]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB
