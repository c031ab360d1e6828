"""Build libspecstream.so (gfx950) in-tree with hipcc.

Usage: python -m paper_2609_33184_amd.build_lib   (or __graft_entry__.build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libspecstream.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}", "-Wall"]
# packed FP32 instructions stay disabled in every device compile
DEVICE_ONLY = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = True) -> str:
    bdir = os.path.join(ROOT, "_build")
    os.makedirs(bdir, exist_ok=True)
    objs = []
    kobj = os.path.join(bdir, "ss_kernels.o")
    _run([HIPCC, *COMMON, *DEVICE_ONLY, "-c", os.path.join(CSRC, "ss_kernels.hip"), "-o", kobj])
    objs.append(kobj)
    for name in ("ss_host", "ss_tier", "ss_width"):
        hobj = os.path.join(bdir, name + ".o")
        _run([HIPCC, *COMMON, "-x", "c++", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-c",
              os.path.join(CSRC, name + ".cpp"), "-o", hobj])
        objs.append(hobj)
    tmp = LIB + ".tmp"
    _run([HIPCC, *DEVICE_ONLY, "-shared", "-fPIC", *objs, "-o", tmp])
    shutil.move(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
    sys.exit(0)
