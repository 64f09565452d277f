"""Host sanitizer build: the host core and the oracle with AddressSanitizer
and UndefinedBehaviorSanitizer, and a run of their CPU tests against it.

``python -m paper_2407_21255_amd.sanitize`` compiles both with g++ / gcc into
``_build/sanitize/`` (host code only: neither contains device code) and runs
the CPU tests that drive them (validation, planning, hazard tracking, the
range allocator, the engine choice, the oracle and its pins) in a child
process with the sanitizer runtime preloaded, since the Python interpreter
itself is not instrumented.  Any sanitizer report ends that process with an
error, so the exit status is the verdict.  Leak checking is off: the
interpreter's own allocations would drown the report.
"""
from __future__ import annotations

import os
import subprocess
import sys

from paper_2407_21255_amd.build import CORE_SOURCES, CSRC, INCLUDE, ROOT

OUT_DIR = os.path.join(ROOT, "_build", "sanitize")
FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-fno-omit-frame-pointer", "-g", "-O1"]
TESTS = ["tests/test_core_plan.py", "tests/test_core_hazards.py", "tests/test_core_ranges.py",
         "tests/test_core_links.py", "tests/test_oracle_pins.py",
         "tests/test_oracle_ext_pins.py"]


def _run(cmd):
    print("+", " ".join(cmd), flush=True)
    subprocess.check_call(cmd)


def build() -> tuple:
    """Returns the paths of the instrumented core and oracle."""
    os.makedirs(OUT_DIR, exist_ok=True)
    core = os.path.join(OUT_DIR, "libaqua_core.so")
    orc = os.path.join(OUT_DIR, "liboracle.so")
    _run(["g++", *FLAGS, "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wextra",
          "-I", INCLUDE, "-I", CSRC, *[os.path.join(CSRC, s) for s in CORE_SOURCES],
          "-o", core])
    _run(["gcc", *FLAGS, "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
          os.path.join(ROOT, "oracle", "aqua_oracle.c"), "-o", orc])
    return core, orc


def run(extra=()) -> int:
    core, orc = build()
    runtime = subprocess.check_output(["gcc", "-print-file-name=libasan.so"],
                                      text=True).strip()
    env = dict(os.environ)
    env.update({"AQUA_CORE_LIB": core, "AQUA_ORACLE_LIB": orc, "LD_PRELOAD": runtime,
                "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"})
    cmd = [sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
           *TESTS, *extra]
    print("+", " ".join(cmd), flush=True)
    return subprocess.call(cmd, cwd=ROOT, env=env)


if __name__ == "__main__":
    sys.exit(run(sys.argv[1:]))
