"""The launch planning of the layer sweep (split-K factors, tile choice, per-chunk workspace
layout) compiled on the CPU with AddressSanitizer and UndefinedBehaviorSanitizer, and replayed
against buffers of exactly the planned sizes (tests/host/plan_test.cpp)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_00049_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_plan_under_address_sanitizer(tmp_path):
    exe = tmp_path / "plan_test"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-static-libasan", "-static-libubsan",
           "-fno-sanitize-recover=undefined", f"-I{CSRC}", os.path.join(ROOT, "tests", "host", "plan_test.cpp"),
           os.path.join(CSRC, "plan.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    res = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "all checks passed" in res.stdout
