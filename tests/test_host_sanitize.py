"""The C ABI's host-side validation and planning (simsd_plan.cpp) built
without HIP by g++ under AddressSanitizer and UndefinedBehaviorSanitizer and
run on the CPU: the error cases of the ABI tests, the workloads' workspace
sizes and a seeded fuzz of extreme descriptors (tests/host/validation_check.cpp).
Any sanitizer report aborts the program and fails the test."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_02544_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_validation_under_sanitizers(tmp_path):
    exe = str(tmp_path / "validation_check")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(CSRC, "simsd_plan.cpp"),
           os.path.join(ROOT, "tests", "host", "validation_check.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out
    assert "runtime error" not in out and "AddressSanitizer" not in out, out
    assert ", 0 failed" in r.stdout, out
