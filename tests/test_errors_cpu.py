"""Error paths of the host library, checked on the CPU.

tests/cpp/error_check.cpp links the library's host code (ss_host.cpp) with
stub kernel launchers and stub HIP runtime calls that fail on demand, and a
global operator new that can throw.  It checks that a call failing after part
of its work was enqueued marks the round (and the pipeline it went through)
failed, so later calls return SS_ERR_BAD_STATE without enqueueing anything;
that a failure before anything was enqueued leaves the round usable; and that
host allocation failures return SS_ERR_OUT_OF_MEMORY.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "cpp", "error_check.cpp")
HOST = os.path.join(ROOT, "paper_2609_33184_amd", "csrc", "ss_host.cpp")


def test_failed_calls_poison_the_round(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None or not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"):
        pytest.skip("needs g++ and the HIP headers")
    exe = tmp_path / "error_check"
    subprocess.run([cxx, "-O1", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    f"-I{ROOT}/include", f"-I{ROOT}/paper_2609_33184_amd/csrc", SRC, HOST, "-o", str(exe)],
                   check=True, capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    print(res.stdout[-3000:])
    assert res.returncode == 0 and "all ok" in res.stdout, res.stdout[-3000:] + res.stderr[-2000:]
