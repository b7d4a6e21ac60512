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


KERNEL_TUS = ("optcc_exec.hip", "optcc_kern_f32.hip", "optcc_kern_bf16.hip", "optcc_kern_i32.hip",
              "optcc_kern_f16.hip", "optcc_kern_f32_g58.hip", "optcc_kern_bf16_g58.hip",
              "optcc_kern_i32_g58.hip", "optcc_kern_f16_g58.hip", "optcc_narrow.hip")


def sources():
    return [os.path.join(CSRC, f) for f in ("optcc_plan.cpp",) + KERNEL_TUS]


def _run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = True) -> str:
    """Compile every translation unit (in parallel) and link liboptcc.so."""
    from concurrent.futures import ThreadPoolExecutor

    os.makedirs(BUILD, exist_ok=True)
    jobs = [["g++", *COMMON, "-c", os.path.join(CSRC, "optcc_plan.cpp"), "-o",
             os.path.join(BUILD, "optcc_plan.o"), "-I/opt/rocm/include"]]
    for tu in KERNEL_TUS:
        jobs.append([HIPCC, f"--offload-arch={ARCH}", *COMMON, *DEVICE_FLAGS, "-c",
                     os.path.join(CSRC, tu), "-o", os.path.join(BUILD, tu.replace(".hip", ".o"))])
    workers = max(1, min(len(jobs), os.cpu_count() or 1, 16))
    with ThreadPoolExecutor(workers) as ex:
        for f in [ex.submit(_run, j) for j in jobs]:
            f.result()
    objs = [j[j.index("-o") + 1] for j in jobs]
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


C_CHECK_SRC = os.path.join(ROOT, "tests", "c_abi_check.c")
C_CHECK = os.path.join(ROOT, "tests", "c_abi_check")


def build_c_check() -> str:
    """Compile the plain-C user of the C ABI (tests/c_abi_check.c) with gcc
    against include/optcc.h, liboptcc.so and the HIP runtime."""
    _run(["gcc", "-std=c99", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
          f"-I{INCLUDE}", C_CHECK_SRC, "-o", C_CHECK + ".tmp", f"-L{PKG}", "-loptcc",
          "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,$ORIGIN/../paper_2606_01680_amd"])
    os.replace(C_CHECK + ".tmp", C_CHECK)
    return C_CHECK


SANITIZE_SRC = os.path.join(ROOT, "tests", "host_sanitize.cpp")
SANITIZE = os.path.join(ROOT, "tests", "host_sanitize")


def build_host_sanitize() -> str:
    """Compile the host half of the library (optcc_plan.cpp, no device code)
    with its test driver under AddressSanitizer and UndefinedBehaviorSanitizer."""
    _run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", f"-I{INCLUDE}", f"-I{CSRC}",
          SANITIZE_SRC, os.path.join(CSRC, "optcc_plan.cpp"), "-o", SANITIZE + ".tmp"])
    os.replace(SANITIZE + ".tmp", SANITIZE)
    return SANITIZE


if __name__ == "__main__":
    build()
    build_c_check()
    build_host_sanitize()
    sys.exit(0)
