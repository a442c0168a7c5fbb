"""The planner's bounds invariants, checked natively under AddressSanitizer and UBSan (host only).

Builds tests/native/planner_check.cpp together with the library's plan.cpp using g++ (no HIP, no
GPU) and runs it over random and full-size layouts."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_planner_invariants_under_sanitizers(tmp_path):
    exe = tmp_path / "planner_check"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2607_22614_amd", "csrc"),
           os.path.join(ROOT, "tests", "native", "planner_check.cpp"),
           os.path.join(ROOT, "paper_2607_22614_amd", "csrc", "plan.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe), "400"], capture_output=True, text=True, timeout=600,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
    assert r.returncode == 0, r.stdout + r.stderr
    assert " 0 errors" in r.stdout
