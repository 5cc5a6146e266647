"""The host half of the library (plan compiler and transition-DAG planner) built with g++ under
AddressSanitizer, UndefinedBehaviorSanitizer and LeakSanitizer, driven through the C ABI by
tests/sanitize_host_driver.cpp: every micro layout pair sampled in both element types, fused,
converting, alias and receiver (from-buckets) plans, the 8B plans, bucket geometry and per-bucket records, the workspace image
(the host's copy of the tile and chunk maps the upload builds on the device), table checks, the DAG
planner on random and malformed scenarios, and the error paths. Any report, or any unexpected status,
fails the run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_34645_amd", "csrc")


def test_plan_compiler_and_dag_planner_under_sanitizers(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ is not available")
    exe = str(tmp_path / "driver")
    cmd = ["g++", "-std=c++17", "-Wall", "-Wextra", "-Werror", "-g", "-O1",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "emu_plan.cpp"), os.path.join(CSRC, "emu_transition.cpp"),
           os.path.join(ROOT, "tests", "sanitize_host_driver.cpp"), "-o", exe]
    subprocess.run(cmd, check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    assert "ERROR: AddressSanitizer" not in res.stderr and "runtime error" not in res.stderr
    assert res.stdout.strip().splitlines()[-1].startswith("ok ")
