"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): tests/host/host_fuzz.cpp is built with g++ together with the
host sources (plan, ABI, step-tag tracker, planner) and the C oracle, then
run.  It exercises the tracker and planner with random call sequences, table
validation with adversarial tables, and the delta payload layout against the
oracle's.  No device code is built or run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2509_03047_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.mark.slow
def test_host_code_under_sanitizers(tmp_path):
    if shutil.which("g++") is None or not os.path.isdir(os.path.join(ROCM, "include", "hip")):
        pytest.skip("needs g++ and the HIP headers")
    exe = str(tmp_path / "host_fuzz")
    srcs = [os.path.join(ROOT, "tests", "host", "host_fuzz.cpp")] + [
        os.path.join(CSRC, f) for f in ("plan.cpp", "api.cpp", "steptag.cpp", "layout.cpp")]
    cmd = (["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
            "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
            "-I", os.path.join(ROOT, "oracle"), "-I", os.path.join(ROCM, "include")] + srcs
           + ["-x", "c", os.path.join(ROOT, "oracle", "fr_oracle.c"), "-x", "none", "-fopenmp",
              "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"),
              "-o", exe])
    b = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert b.returncode == 0, b.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
    assert "0 delta layout mismatches" in r.stdout
