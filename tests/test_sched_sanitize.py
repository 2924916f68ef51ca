"""The scheduler's host code (csrc/sched.cpp, the C ABI of include/sd_sched.h)
built with AddressSanitizer and UndefinedBehaviorSanitizer and driven over
random task sets and invalid arguments (tests/native/sched_sanitize.cpp):
no out-of-bounds access, leak or undefined operation, and every valid plan
is consistent across the entry points."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_scheduler_under_address_and_ub_sanitizers(tmp_path):
    exe = tmp_path / "sched_sanitize"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2510_11331_amd", "csrc"),
           os.path.join(ROOT, "paper_2510_11331_amd", "csrc", "sched.cpp"),
           os.path.join(ROOT, "tests", "native", "sched_sanitize.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, timeout=300)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "plans checked" in r.stdout
