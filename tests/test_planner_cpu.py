"""Host planner of the history calls, checked on the CPU.

tests/cpp/plan_check.cpp links the library's host code (ss_host.cpp) with
stub kernel launchers that record every launch's item and unit tables, and
walks each unit's tiles the way the chunk kernels do.  Over the five
workload shapes (per-chunk and batched calls, forced piece sizes, both chunk
layouts) and random ragged batches it checks that every history token of
every request is visited exactly once per KV head, every buffer resource
lies inside its chunk, a unit's chain belongs to one request and one state
slot, slots are dense and fresh flags match the slots already written.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "cpp", "plan_check.cpp")
HOST = os.path.join(ROOT, "paper_2609_33184_amd", "csrc", "ss_host.cpp")


def test_planner_covers_every_token_once(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None or not os.path.exists("/opt/rocm/lib/libamdhip64.so"):
        pytest.skip("needs g++ and the ROCm runtime library to link the host code")
    exe = tmp_path / "plan_check"
    subprocess.run([cxx, "-O1", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    f"-I{ROOT}/include", f"-I{ROOT}/paper_2609_33184_amd/csrc", SRC, HOST,
                    "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", str(exe)],
                   check=True, capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    print(res.stdout[-3000:])
    assert res.returncode == 0 and "all ok" in res.stdout, res.stdout[-3000:] + res.stderr[-2000:]
