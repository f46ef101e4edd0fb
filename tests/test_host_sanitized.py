"""The library's host code under AddressSanitizer and UBSan (CPU, no GPU).

tests/helpers/plan_check.cpp links the launch planner and validation (csrc/zo_plan.cpp) and
the coefficient function (csrc/zo_host.cpp), built with g++ -fsanitize=address,undefined,
and checks on the CPU that the index arithmetic of the sweeps covers every element of a
tensor exactly once: head and tail tiles and full row groups for offsets up to the top of
the 64-bit index range and n up to ZO_N_MAX - 1, the kernels' 32-bit chunk walk with one to
four waves per stream, segment batches below 2^31 chunks, dispatch sizes below 2^32
work-items, and the validation codes. Any sanitizer report fails the run."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_38095_amd", "csrc")


@pytest.fixture(scope="module")
def plan_check(tmp_path_factory):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no g++")
    exe = str(tmp_path_factory.mktemp("asan") / "plan_check")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-ffp-contract=off", "-Wall", "-Wextra", "-Werror",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "helpers", "plan_check.cpp"), os.path.join(CSRC, "zo_plan.cpp"),
           os.path.join(CSRC, "zo_host.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_planner_and_validation_under_asan_ubsan(plan_check):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([plan_check], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "plan_check ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
