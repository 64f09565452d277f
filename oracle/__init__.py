"""CPU oracle for the KV page-swap path -- TEST INFRASTRUCTURE ONLY.

This package wraps ``aqua_oracle.c``, a plain single-threaded C loop that
defines what swap-out (gather) and swap-in (scatter) compute (Aqua, section 7,
"Efficient context switching").  Only the tests, the smoke check and the
bench's CPU-baseline leg may import it; the GPU library never does, and the
two share no code.

All buffers are host numpy arrays (C-contiguous).  Status codes are the
library's: 0 ok, -1 invalid, -2 range, -3 duplicate, -4 capacity.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "aqua_oracle.c")
# AQUA_ORACLE_LIB names another build of the oracle (the sanitizer build).
_LIB = os.environ.get("AQUA_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

OK, ERR_INVALID, ERR_RANGE, ERR_DUPLICATE, ERR_CAPACITY = 0, -1, -2, -3, -4
F16, BF16, FP8_E4M3 = 1, 2, 3


class KVDesc(ctypes.Structure):
    _fields_ = [
        ("num_layers", ctypes.c_uint32),
        ("num_blocks", ctypes.c_uint32),
        ("num_kv_heads", ctypes.c_uint32),
        ("block_tokens", ctypes.c_uint32),
        ("head_dim", ctypes.c_uint32),
        ("dtype", ctypes.c_int32),
    ]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/liboracle.so``."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
             "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        u32, u64, i32 = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32
        D = ctypes.POINTER(KVDesc)
        L.oracle_chunk_bytes.argtypes = [D]
        L.oracle_chunk_bytes.restype = u64
        L.oracle_bytes_per_token.argtypes = [D]
        L.oracle_bytes_per_token.restype = u64
        L.oracle_pool_check.argtypes = [D, P, u64]
        L.oracle_pool_check.restype = i32
        L.oracle_swap_out.argtypes = [D, P, u64, u32, P, P, P, u64, P]
        L.oracle_swap_out.restype = i32
        L.oracle_swap_in.argtypes = [D, P, u64, u32, P, P, P, u64, P]
        L.oracle_swap_in.restype = i32
        L.oracle_swap_out_ex.argtypes = [D, P, u64, u32, P, P, P, u64, P, P, u32, u32]
        L.oracle_swap_out_ex.restype = i32
        L.oracle_swap_in_ex.argtypes = [D, P, u64, u32, P, P, P, u64, P, P, u32, u32]
        L.oracle_swap_in_ex.restype = i32
        L.oracle_migrate.argtypes = [P, u64, P, u64, u32, P, P, P]
        L.oracle_migrate.restype = i32
        _lib = L
    return _lib


def desc(num_layers, num_blocks, num_kv_heads, block_tokens, head_dim, dtype):
    return KVDesc(num_layers, num_blocks, num_kv_heads, block_tokens, head_dim,
                  dtype)


def _ptr(a):
    if a is None:
        return None
    if isinstance(a, int):
        return a
    assert a.flags["C_CONTIGUOUS"], "oracle buffers must be C-contiguous"
    return a.ctypes.data


def _tables(tables):
    """CSR form of a list of block tables: (int32 ids, uint64 offsets)."""
    ids = np.ascontiguousarray(
        np.concatenate([np.asarray(t, dtype=np.int64) for t in tables])
        if tables else np.zeros(0, np.int64)).astype(np.int32)
    offs = np.zeros(len(tables) + 1, dtype=np.uint64)
    if tables:
        offs[1:] = np.cumsum([len(t) for t in tables])
    return ids, offs


def chunk_bytes(d: KVDesc) -> int:
    return int(lib().oracle_chunk_bytes(ctypes.byref(d)))


def bytes_per_token(d: KVDesc) -> int:
    return int(lib().oracle_bytes_per_token(ctypes.byref(d)))


def pool_check(d: KVDesc, pool, pool_bytes=None) -> int:
    nb = pool.nbytes if pool_bytes is None else pool_bytes
    return int(lib().oracle_pool_check(ctypes.byref(d), _ptr(pool), nb))


def swap_out(d: KVDesc, pool: np.ndarray, tables, dst: np.ndarray,
             img_offsets=None, *, ids=None, offs=None, dst_bytes=None) -> int:
    """Gather the chunks named by ``tables`` from ``pool`` into ``dst``."""
    if ids is None:
        ids, offs = _tables(tables)
    io = None if img_offsets is None else np.ascontiguousarray(
        img_offsets, dtype=np.uint64)
    return int(lib().oracle_swap_out(
        ctypes.byref(d), _ptr(pool), pool.nbytes, len(offs) - 1, _ptr(ids),
        _ptr(offs), _ptr(dst), dst.nbytes if dst_bytes is None else dst_bytes,
        _ptr(io)))


def swap_in(d: KVDesc, pool: np.ndarray, tables, src: np.ndarray,
            img_offsets=None, *, ids=None, offs=None, src_bytes=None) -> int:
    """Scatter the image(s) in ``src`` into the pool chunks named by ``tables``."""
    if ids is None:
        ids, offs = _tables(tables)
    io = None if img_offsets is None else np.ascontiguousarray(
        img_offsets, dtype=np.uint64)
    return int(lib().oracle_swap_in(
        ctypes.byref(d), _ptr(pool), pool.nbytes, len(offs) - 1, _ptr(ids),
        _ptr(offs), _ptr(src), src.nbytes if src_bytes is None else src_bytes,
        _ptr(io)))


def _u64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.uint64)


def swap_out_ex(d: KVDesc, pool: np.ndarray, tables, dst: np.ndarray,
                img_offsets=None, img_blocks=None, first_layer=0, num_layers=0,
                *, ids=None, offs=None, dst_bytes=None) -> int:
    """Swap-out of layers [first_layer, first_layer + num_layers) (all when
    num_layers is 0) into images of img_blocks[s] blocks per layer."""
    if ids is None:
        ids, offs = _tables(tables)
    io, ib = _u64(img_offsets), _u64(img_blocks)
    return int(lib().oracle_swap_out_ex(
        ctypes.byref(d), _ptr(pool), pool.nbytes, len(offs) - 1, _ptr(ids),
        _ptr(offs), _ptr(dst), dst.nbytes if dst_bytes is None else dst_bytes,
        _ptr(io), _ptr(ib), first_layer, num_layers))


def swap_in_ex(d: KVDesc, pool: np.ndarray, tables, src: np.ndarray,
               img_offsets=None, img_blocks=None, first_layer=0, num_layers=0,
               *, ids=None, offs=None, src_bytes=None) -> int:
    if ids is None:
        ids, offs = _tables(tables)
    io, ib = _u64(img_offsets), _u64(img_blocks)
    return int(lib().oracle_swap_in_ex(
        ctypes.byref(d), _ptr(pool), pool.nbytes, len(offs) - 1, _ptr(ids),
        _ptr(offs), _ptr(src), src.nbytes if src_bytes is None else src_bytes,
        _ptr(io), _ptr(ib), first_layer, num_layers))


def migrate(src: np.ndarray, dst: np.ndarray, src_offsets, dst_offsets, lengths,
            src_bytes=None, dst_bytes=None) -> int:
    """Copy byte ranges from one offload buffer to another."""
    so, do, ln = _u64(src_offsets), _u64(dst_offsets), _u64(lengths)
    return int(lib().oracle_migrate(
        _ptr(src), src.nbytes if src_bytes is None else src_bytes, _ptr(dst),
        dst.nbytes if dst_bytes is None else dst_bytes, len(ln), _ptr(so), _ptr(do),
        _ptr(ln)))
