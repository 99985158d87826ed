"""CPU correctness tier: the library's host code and the kernels' index
arithmetic built with g++ under the address and undefined-behaviour sanitizers.

* tests/cpu_tier/index_harness.cpp runs the kernels' index functions
  (paper_2609_20888_amd/csrc/eta_index.h: proportional split plan, union-list
  tile prefix and item lookup, split shares, compaction slots, screening's
  record offsets, the predictor's row groups) on edge geometries -- ragged T,
  T below one block, capacities that are not a multiple of 4, 2048 screening
  tiles, 1024 splits -- over heap buffers of exactly the kernels' sizes.
* tests/cpu_tier/api_harness.cpp links eta_api.cpp (argument validation,
  split planning, workspace carve-up) against stub launchers that check every
  workspace region lies inside a workspace of exactly the requested size and
  that no two overlap, then drives every entry point, including the invalid
  calls that must be refused before any launch.

Both need only g++ and the HIP headers; nothing here touches a GPU.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TIER = os.path.join(ROOT, "tests", "cpu_tier")
CSRC = os.path.join(ROOT, "paper_2609_20888_amd", "csrc")
INC = os.path.join(ROOT, "include")
ROCM_INC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")
SAN = ["-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")


def _build_and_run(tmp_path, name, sources, extra):
    exe = str(tmp_path / name)
    cmd = ["g++", *SAN, *extra, *sources, "-o", exe]
    b = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert b.returncode == 0, "build failed:\n" + b.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, f"{name} failed ({r.returncode}):\n{r.stderr[-6000:]}"
    assert "all checks passed" in r.stdout
    return r.stdout


def test_index_arithmetic_sanitized(tmp_path):
    _build_and_run(tmp_path, "index_harness",
                   [os.path.join(TIER, "index_harness.cpp")], ["-I" + CSRC])


@pytest.mark.skipif(not os.path.exists(os.path.join(ROCM_INC, "hip", "hip_runtime_api.h")),
                    reason="HIP headers not installed")
def test_host_api_sanitized(tmp_path):
    out = _build_and_run(
        tmp_path, "api_harness",
        [os.path.join(CSRC, "eta_api.cpp"), os.path.join(TIER, "api_harness.cpp")],
        ["-D__HIP_PLATFORM_AMD__", "-I" + ROCM_INC, "-I" + INC, "-I" + CSRC])
    n = int(out.split("api harness:")[1].split()[0])
    assert n > 1000
