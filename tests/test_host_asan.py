"""The library's host-only C++ under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Builds the host part of the ABI (shape rules, stage plan), the cue machine, the
host FFN of the offloaded experts and the copy-or-host plan from source with
g++ into a small driver
(tests/host_asan/driver.cpp) with the sanitizers on, and runs it: the driver
checks the cue machine against a brute-force matcher over random streams and
exercises the host FFN and the plan with several thread counts and their error
paths.  Any memory error or undefined behaviour aborts the run.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_21614_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_code_under_sanitizers(tmp_path):
    exe = tmp_path / "driver"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-pthread",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "host_asan", "driver.cpp"),
           os.path.join(CSRC, "host_abi.cpp"), os.path.join(CSRC, "cue_fsm.cpp"), os.path.join(CSRC, "host_ffn.cpp"),
           "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host code ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
