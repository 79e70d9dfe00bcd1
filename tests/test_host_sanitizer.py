"""The host planner (plan.cpp) and bit allocation (alloc.cpp) built with g++
under AddressSanitizer and UndefinedBehaviorSanitizer, driven by
tests/host/plan_check.cpp: random valid block lists up to the largest k, the
statuses of invalid ones, the decode work split's coverage and alignment
properties, and the allocation's outputs on random layers.  Host code only: no
HIP compiler and no GPU are involved."""
import os
import shutil
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
CSRC = ROOT / "paper_2607_14618_amd" / "csrc"
ROCM_INCLUDE = Path(os.environ.get("ROCM_PATH", "/opt/rocm")) / "include"


@pytest.fixture(scope="module")
def plan_check(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None or not (ROCM_INCLUDE / "hip" / "hip_runtime.h").exists():
        pytest.skip("g++ or the HIP headers are not available")
    exe = tmp_path_factory.mktemp("asan") / "plan_check"
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", f"-I{ROCM_INCLUDE}", f"-I{ROOT / 'include'}", f"-I{CSRC}",
           str(CSRC / "plan.cpp"), str(CSRC / "alloc.cpp"), str(ROOT / "tests" / "host" / "plan_check.cpp"),
           "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


@pytest.mark.parametrize("seed,iters", [(1, 400), (2024, 1500)])
def test_planner_under_sanitizers(plan_check, seed, iters):
    env = dict(os.environ, ASAN_OPTIONS="abort_on_error=0:detect_leaks=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(plan_check), str(seed), str(iters)], capture_output=True, text=True,
                       env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "plan_check ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
