"""Builds the native libraries in-tree.

* ``libaqua.so``       -- the C-ABI library with the gfx950 kernels (hipcc).
* ``libaqua_core.so``  -- the host core alone, with test entry points, built
                          by the system C++ compiler so that CPU-only tests
                          can drive validation, planning and hazard tracking.
* ``tests/c_abi_client`` -- a plain C program (gcc) that uses ``libaqua.so``
                          through ``include/aqua.h`` alone; a GPU test runs it.

Run ``python -m paper_2407_21255_amd.build``.

The sanitizer build of the host core and the oracle is
``python -m paper_2407_21255_amd.sanitize`` (CPU only).
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
HIP_LIB = os.path.join(PKG, "libaqua.so")
C_CLIENT_SRC = os.path.join(ROOT, "tests", "c_abi_client.c")
C_CLIENT = os.path.join(ROOT, "tests", "c_abi_client")
CORE_LIB = os.path.join(PKG, "libaqua_core.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

HIP_SOURCES = ["aqua_core.cpp", "cfs.cpp", "swap_kernels.hip", "link_engine.hip",
               "aqua_capi.hip"]
CORE_SOURCES = ["aqua_core.cpp", "core_testapi.cpp"]

# Packed fp32 instructions are switched off for every device compile.
HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-fvisibility=hidden",
]


def _run(cmd):
    print("+", " ".join(cmd), flush=True)
    subprocess.check_call(cmd)


def build_hip(out: str = HIP_LIB, extra=()) -> str:
    """``extra``: additional compiler flags (measurement variants)."""
    srcs = []
    for s in HIP_SOURCES:
        p = os.path.join(CSRC, s)
        # hipcc compiles .cpp files as host code unless told they are HIP.
        srcs += (["-x", "hip", p] if s.endswith(".hip") else ["-x", "c++", p])
    tmp = out + ".tmp"
    _run([HIPCC, *HIP_FLAGS, *extra, "-I", INCLUDE, "-I", CSRC, *srcs, "-o", tmp,
          "-L/opt/rocm/lib", "-lhsa-runtime64", "-lrocprofiler-sdk-roctx"])
    os.replace(tmp, out)
    return out


def build_core(out: str = CORE_LIB) -> str:
    tmp = out + ".tmp"
    _run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wextra",
          "-I", INCLUDE, "-I", CSRC,
          *[os.path.join(CSRC, s) for s in CORE_SOURCES], "-o", tmp])
    os.replace(tmp, out)
    return out


def build_c_client(out: str = C_CLIENT) -> str:
    """C11, the HIP runtime's C API and libaqua.so: nothing else."""
    tmp = out + ".tmp"
    _run(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
          "-I", INCLUDE, "-I/opt/rocm/include", C_CLIENT_SRC, "-o", tmp,
          "-L", PKG, "-laqua", "-L/opt/rocm/lib", "-lamdhip64",
          "-Wl,-rpath,$ORIGIN/../paper_2407_21255_amd", "-Wl,-rpath,/opt/rocm/lib"])
    os.replace(tmp, out)
    return out


def build_all() -> None:
    build_core()
    build_hip()
    build_c_client()


if __name__ == "__main__":
    what = sys.argv[1:] or ["all"]
    if "all" in what:
        build_all()
    if "core" in what:
        build_core()
    if "hip" in what:
        build_hip()
    if "client" in what:
        build_c_client()

