"""The C ABI from plain C: tests/host/abi_demo (built with the library)
allocates device memory and a stream with the HIP runtime, restores a small
state across differing layouts, compares two replicas and checksums through
libflashrestore, and checks every output byte against the C oracle."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DEMO = os.path.join(ROOT, "tests", "host", "abi_demo")


def test_c_program_restores_through_the_c_abi():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(DEMO), "tests/host/abi_demo is missing: run __graft_entry__.build()"
    r = subprocess.run([DEMO], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stderr
    assert "c abi ok" in r.stdout
