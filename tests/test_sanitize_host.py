"""The host planner under AddressSanitizer and UBSan (CPU only).

tests/native/sanitize_plan.cpp sweeps build_layout, the plans' host tables
and the allocation-free step's scratch layout over the benchmark workloads,
every tile policy, K split, apply mode and dtype, ragged and degenerate
shapes and the refusals.  It is built here with g++ and the sanitizers (no
GPU code, no HIP call) and must end with "ok" and no sanitizer report."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2510_16981_amd", "csrc")
ROCM_INCLUDE = "/opt/rocm/include"


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir(ROCM_INCLUDE),
                    reason="needs g++ and the HIP headers")
def test_planner_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "sanitize_plan"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", CSRC, "-I", os.path.join(ROOT, "include"),
           "-I", ROCM_INCLUDE,
           os.path.join(ROOT, "tests", "native", "sanitize_plan.cpp"),
           os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "step_core.cpp"),
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), (r.stdout[-2000:], r.stderr[-4000:])
