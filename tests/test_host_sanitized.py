"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

* ``tests/host/plan_check.cpp`` with the planner (``skew_plan.cpp``) and the C ABI's host
  code (``skew_api.cpp``): the HIP runtime calls act on host memory and the kernel launchers
  check the items they receive. It checks that every element of the unit, ragged, >2^31 and
  stacked tables lies in exactly one update tile and one row band or pass-1 tile, that the
  row-band geometry fits the kernel, that state and workspace regions are 256-byte aligned,
  in bounds and disjoint, and that a step launches exactly the planned items.
* ``tests/host/oracle_check.c`` with the CPU oracle: every tier and option, checking the
  clip bound on the way.
Both are compiled here with g++/gcc (host code only) and run as child processes.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST = os.path.join(ROOT, "tests", "host")
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _build_and_run(cmd, exe, tmp_path, expect):
    res = subprocess.run(cmd, cwd=HOST, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    run = subprocess.run([exe], cwd=HOST, capture_output=True, text=True, env=ENV, timeout=600)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "ERROR: AddressSanitizer" not in out, out[-4000:]
    assert expect in out, out[-2000:]
    return out


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the HIP headers")
def test_planner_and_host_abi_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_check")
    cmd = ["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-o", exe, "plan_check.cpp",
           os.path.join(ROOT, "paper_2607_19058_amd", "csrc", "skew_plan.cpp"),
           os.path.join(ROOT, "paper_2607_19058_amd", "csrc", "skew_api.cpp")]
    out = _build_and_run(cmd, exe, tmp_path, "planner and host checks passed")
    print(out.strip().splitlines()[-1])


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_check")
    cmd = ["gcc", "-std=c11", *SAN, "-fopenmp", "-ffp-contract=off", "-o", exe, "oracle_check.c",
           os.path.join(ROOT, "oracle", "skew_oracle.c"), "-lm"]
    _build_and_run(cmd, exe, tmp_path, "all steps clean")
