"""Build liboptcc.so in-tree for gfx950 (MI355X) with hipcc.

    python -m paper_2606_01680_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "liboptcc.so")
BUILD = os.path.join(PKG, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 instructions are disabled for all device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result", f"-I{INCLUDE}", f"-I{CSRC}"]


def sources():
    return [os.path.join(CSRC, f) for f in ("optcc_plan.cpp", "optcc_exec.hip")]


def _run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    plan_o = os.path.join(BUILD, "optcc_plan.o")
    _run(["g++", *COMMON, "-c", os.path.join(CSRC, "optcc_plan.cpp"), "-o", plan_o,
          "-I/opt/rocm/include"])
    objs.append(plan_o)
    exec_o = os.path.join(BUILD, "optcc_exec.o")
    _run([HIPCC, f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS, "-c",
          os.path.join(CSRC, "optcc_exec.hip"), "-o", exec_o])
    objs.append(exec_o)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
