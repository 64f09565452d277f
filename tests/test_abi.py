"""The C-ABI library loads and exports every entry point include/aqua.h
declares (no compute call: this runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aqua.h")
LIB = os.path.join(ROOT, "paper_2407_21255_amd", "libaqua.so")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"AQUA_API\s+[\w\s\*]+?\b(aqua_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ["aqua_kv_pool_create", "aqua_kv_pool_destroy", "aqua_swap_out",
              "aqua_swap_in", "aqua_sync", "aqua_stream_wait", "aqua_status_str"]:
        assert n in names


def test_library_exports_every_declared_symbol():
    if not os.path.exists(LIB):
        from paper_2407_21255_amd import build
        build.build_hip()
    lib = ctypes.CDLL(LIB)
    for n in _declared():
        assert hasattr(lib, n), n
    lib.aqua_status_str.restype = ctypes.c_char_p
    lib.aqua_status_str.argtypes = [ctypes.c_int32]
    assert lib.aqua_status_str(0) == b"ok"
    assert lib.aqua_status_str(-3) == b"duplicate destination"


def test_binding_mirrors_the_header():
    from paper_2407_21255_amd import aqua
    assert sorted(aqua.EXPORTS) == _declared()
    for n in _declared():
        assert callable(getattr(aqua, n)), n


def test_binding_fails_loudly_without_the_library(tmp_path):
    from paper_2407_21255_amd import aqua
    saved = aqua._lib
    aqua._lib = None
    try:
        with pytest.raises(FileNotFoundError):
            aqua.load(str(tmp_path / "libaqua.so"))
    finally:
        aqua._lib = saved


def test_null_handles_are_rejected_without_a_gpu():
    lib = ctypes.CDLL(LIB)
    for n in ["aqua_kv_pool_destroy"]:
        f = getattr(lib, n)
        f.argtypes = [ctypes.c_void_p]
        f.restype = ctypes.c_int32
        assert f(None) == -1
    lib.aqua_sync.argtypes = [ctypes.c_void_p, ctypes.c_uint64]
    lib.aqua_sync.restype = ctypes.c_int32
    assert lib.aqua_sync(None, 0) == -1
    lib.aqua_kv_pool_create.restype = ctypes.c_int32
    assert lib.aqua_kv_pool_create(None, None, ctypes.c_uint64(0), None) == -1


def test_c_client_links_the_library_and_the_hip_runtime_only():
    """The C program that a GPU test runs uses the boundary with no Python
    or torch: its dynamic dependencies name neither."""
    import subprocess
    client = os.path.join(ROOT, "tests", "c_abi_client")
    if not os.path.exists(client):
        from paper_2407_21255_amd import build
        if not os.path.exists(LIB):
            build.build_hip()
        build.build_c_client()
    out = subprocess.run(["ldd", client], capture_output=True, text=True, check=True).stdout
    assert "libaqua.so" in out and "libamdhip64" in out
    assert "python" not in out and "torch" not in out
