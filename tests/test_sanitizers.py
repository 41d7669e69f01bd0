"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Two drivers in tests/sanitize/ are built with gcc/g++ and
-fsanitize=address,undefined (any report aborts the run):

  * host_plan_check.cpp: the library's host-side planning and validation
    (paper_2606_26344_amd/csrc/plan.hpp, plain C++ with no HIP dependency)
    over a grid of shapes up to the validated limits, every path, the
    workspace layouts and the error paths;
  * oracle_check.c: both CPU fp64 oracles on small inputs, every variant,
    row lists, thread counts and error returns.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer", "-Wall", "-Wextra", "-Werror"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _build_and_run(cmd, exe):
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stdout + build.stderr
    run = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=600)
    print(run.stdout)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "runtime error" not in run.stderr and "AddressSanitizer" not in run.stderr, run.stderr
    return run.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_planning_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_plan_check")
    out = _build_and_run(["g++", "-std=c++20", *SAN, "-Wno-unused-function",
                          "-I", os.path.join(ROOT, "include"),
                          "-I", os.path.join(ROOT, "paper_2606_26344_amd", "csrc"),
                          "-o", exe, os.path.join(HERE, "sanitize", "host_plan_check.cpp")], exe)
    assert "0 failures" in out


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_check")
    out = _build_and_run(["gcc", "-std=c11", *SAN, "-fopenmp", "-ffp-contract=off", "-o", exe,
                          os.path.join(HERE, "sanitize", "oracle_check.c"),
                          os.path.join(ROOT, "oracle", "gmlp_oracle.c"),
                          os.path.join(ROOT, "oracle", "softmax_matmul_oracle.c"), "-lm"], exe)
    assert "0 failures" in out
