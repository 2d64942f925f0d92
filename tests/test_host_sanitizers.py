"""The planner's host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

tests/c_abi/plan_check.cpp drives csrc/plan.cpp -- plain host C++, no device
code -- over a seeded sweep of prefill, decode and GEMM shapes and checks every
plan's legality (the tile domains, LDS capacity, the launch grid, key splits
with no empty split) and the formatters' truncation; it is compiled here with
g++ and both sanitizers, any report aborting the run.  A planted corruption
checks that the checks can fail.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_29219_amd", "csrc")


@pytest.fixture(scope="module")
def plan_check(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    out = str(tmp_path_factory.mktemp("sanitize") / "plan_check")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           os.path.join(CSRC, "plan.cpp"), os.path.join(ROOT, "tests", "c_abi", "plan_check.cpp"),
           "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    return out


def _run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    return subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=env)


def test_planner_sweep_is_clean_under_sanitizers(plan_check):
    r = _run(plan_check)
    assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
    assert "plan_check ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr


def test_planted_violation_is_caught(plan_check):
    r = _run(plan_check, "--planted")
    assert r.returncode == 0 and "caught" in r.stdout, (r.stdout + r.stderr)[-2000:]
