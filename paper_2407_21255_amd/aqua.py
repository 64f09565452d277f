"""Python binding of the C ABI in ``include/aqua.h`` (ctypes).

Argument marshalling only: every byte of a swap is moved by the library's
HIP kernels.  The low-level functions carry the C names and return the
C status (plus the ticket where the C call writes one); ``KVPool`` wraps
them for torch tensors and raises ``AquaError`` on a failed call.

torch is imported before the library is loaded so that the library binds
to the HIP runtime torch already holds (both carry the same soname), and
pointers and streams from torch are valid in it.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libaqua.so")

AQUA_OK = 0
AQUA_ERR_INVALID = -1
AQUA_ERR_RANGE = -2
AQUA_ERR_DUPLICATE = -3
AQUA_ERR_CAPACITY = -4
AQUA_ERR_HIP = -5
AQUA_ERR_STATE = -6

AQUA_F16, AQUA_BF16, AQUA_FP8_E4M3 = 1, 2, 3
AQUA_TARGET_DEVICE, AQUA_TARGET_HOST = 0, 1
AQUA_HOST_ZERO_COPY, AQUA_HOST_STAGED = 0, 1
AQUA_LINK_RUNTIME, AQUA_LINK_AUTO = -1, -2
AQUA_YARDSTICK_COPY, AQUA_YARDSTICK_READ, AQUA_YARDSTICK_WRITE = 0, 1, 2

EXPORTS = (
    "aqua_kv_pool_create", "aqua_kv_pool_destroy", "aqua_swap_out",
    "aqua_swap_in", "aqua_swap_out_ex", "aqua_swap_in_ex", "aqua_migrate",
    "aqua_sync", "aqua_stream_wait", "aqua_query",
    "aqua_kv_pool_set_max_workgroups", "aqua_kv_pool_set_host_path",
    "aqua_kv_pool_set_link_engine", "aqua_kv_pool_get_link_engine",
    "aqua_pool_stats_get", "aqua_status_str", "aqua_cfs_partition",
    "aqua_swap_space_create", "aqua_swap_space_destroy", "aqua_swap_alloc", "aqua_swap_free",
    "aqua_swap_locate", "aqua_swap_reclaim", "aqua_swap_restore", "aqua_swap_usage",
    "aqua_hbm_yardstick", "aqua_swap_noalloc",
)


class aqua_kv_desc(ctypes.Structure):
    _fields_ = [
        ("num_layers", ctypes.c_uint32),
        ("num_blocks", ctypes.c_uint32),
        ("num_kv_heads", ctypes.c_uint32),
        ("block_tokens", ctypes.c_uint32),
        ("head_dim", ctypes.c_uint32),
        ("dtype", ctypes.c_int32),
    ]


class aqua_swap_range(ctypes.Structure):
    _fields_ = [
        ("img_blocks", ctypes.c_void_p),
        ("first_layer", ctypes.c_uint32),
        ("num_layers", ctypes.c_uint32),
    ]


class aqua_pool_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "calls_out", "calls_in", "bytes_out", "bytes_in", "bytes_host",
        "descriptors", "waits_inserted", "waits_elided", "calls_migrate",
        "bytes_migrated", "host_ns", "wait_ns")] + [
        ("hip_error", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("launches", ctypes.c_uint64)]


class aqua_cfs_request(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint32) for n in (
        "prompt_tokens", "prefill_done", "generated", "held_blocks")]


class aqua_cfs_params(ctypes.Structure):
    _fields_ = [("batch_tokens", ctypes.c_uint32), ("decode_slots", ctypes.c_uint32),
                ("block_tokens", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("capacity_blocks", ctypes.c_uint64)]


class AquaError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {aqua_status_str(status)} ({status})")
        self.status = status


_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads the library; fails loudly when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(
            f"{path} is missing: build it with "
            "`python -m paper_2407_21255_amd.build` (hipcc, gfx950)")
    L = ctypes.CDLL(path)
    P, u32, u64, i32 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32
    L.aqua_kv_pool_create.argtypes = [ctypes.POINTER(aqua_kv_desc), P, u64,
                                      ctypes.POINTER(P)]
    L.aqua_kv_pool_destroy.argtypes = [P]
    L.aqua_swap_out.argtypes = [P, u32, P, P, P, u64, P, i32, P, ctypes.POINTER(u64)]
    L.aqua_swap_in.argtypes = [P, u32, P, P, P, u64, P, i32, P, ctypes.POINTER(u64)]
    R = ctypes.POINTER(aqua_swap_range)
    L.aqua_swap_out_ex.argtypes = [P, u32, P, P, P, u64, P, R, i32, P, ctypes.POINTER(u64)]
    L.aqua_swap_in_ex.argtypes = [P, u32, P, P, P, u64, P, R, i32, P, ctypes.POINTER(u64)]
    L.aqua_migrate.argtypes = [P, P, u64, i32, P, u64, i32, u32, P, P, P, P,
                               ctypes.POINTER(u64)]
    L.aqua_sync.argtypes = [P, u64]
    L.aqua_stream_wait.argtypes = [P, u64, P]
    L.aqua_query.argtypes = [P, u64]
    L.aqua_kv_pool_set_max_workgroups.argtypes = [P, i32, u32]
    L.aqua_kv_pool_set_host_path.argtypes = [P, i32]
    L.aqua_kv_pool_set_link_engine.argtypes = [P, i32, i32]
    L.aqua_kv_pool_get_link_engine.argtypes = [P, i32, ctypes.POINTER(i32)]
    L.aqua_pool_stats_get.argtypes = [P, ctypes.POINTER(aqua_pool_stats)]
    L.aqua_cfs_partition.argtypes = [P, u32, ctypes.POINTER(aqua_cfs_params), P, P,
                                     ctypes.POINTER(u32), ctypes.POINTER(u64)]
    L.aqua_swap_space_create.argtypes = [P, u64, u64, ctypes.POINTER(P)]
    L.aqua_swap_space_destroy.argtypes = [P]
    L.aqua_swap_alloc.argtypes = [P, u64, ctypes.POINTER(u64)]
    L.aqua_swap_free.argtypes = [P, u64]
    L.aqua_swap_locate.argtypes = [P, u64, ctypes.POINTER(P), ctypes.POINTER(u64),
                                   ctypes.POINTER(i32)]
    L.aqua_swap_reclaim.argtypes = [P, u64, P, ctypes.POINTER(u64)]
    L.aqua_swap_restore.argtypes = [P, P, ctypes.POINTER(u64)]
    L.aqua_swap_usage.argtypes = [P] + [ctypes.POINTER(u64)] * 4
    L.aqua_hbm_yardstick.argtypes = [i32, P, P, u64, P]
    L.aqua_swap_noalloc.argtypes = [P, i32, u32, P, P, P, u64, P, i32, P, ctypes.POINTER(u64)]
    L.aqua_status_str.argtypes = [i32]
    L.aqua_status_str.restype = ctypes.c_char_p
    for n in EXPORTS:
        if n != "aqua_status_str":
            getattr(L, n).restype = i32
    _lib = L
    return L


# -- the C entry points, one to one ------------------------------------------

def aqua_kv_pool_create(desc: aqua_kv_desc, pool_base: int, pool_bytes: int):
    h = ctypes.c_void_p()
    st = load().aqua_kv_pool_create(ctypes.byref(desc), pool_base, pool_bytes,
                                    ctypes.byref(h))
    return st, h


def aqua_kv_pool_destroy(pool) -> int:
    return load().aqua_kv_pool_destroy(pool)


def aqua_swap_out(pool, num_seqs, block_ids, seq_offsets, dst, dst_bytes,
                  img_offsets, target, stream):
    t = ctypes.c_uint64(0)
    st = load().aqua_swap_out(pool, num_seqs, block_ids, seq_offsets, dst, dst_bytes,
                              img_offsets, target, stream, ctypes.byref(t))
    return st, t.value


def aqua_swap_in(pool, num_seqs, block_ids, seq_offsets, src, src_bytes,
                 img_offsets, target, stream):
    t = ctypes.c_uint64(0)
    st = load().aqua_swap_in(pool, num_seqs, block_ids, seq_offsets, src, src_bytes,
                             img_offsets, target, stream, ctypes.byref(t))
    return st, t.value


def aqua_swap_out_ex(pool, num_seqs, block_ids, seq_offsets, dst, dst_bytes,
                     img_offsets, rng, target, stream):
    t = ctypes.c_uint64(0)
    st = load().aqua_swap_out_ex(pool, num_seqs, block_ids, seq_offsets, dst, dst_bytes,
                                 img_offsets, rng, target, stream, ctypes.byref(t))
    return st, t.value


def aqua_swap_in_ex(pool, num_seqs, block_ids, seq_offsets, src, src_bytes,
                    img_offsets, rng, target, stream):
    t = ctypes.c_uint64(0)
    st = load().aqua_swap_in_ex(pool, num_seqs, block_ids, seq_offsets, src, src_bytes,
                                img_offsets, rng, target, stream, ctypes.byref(t))
    return st, t.value


def aqua_swap_noalloc(pool, direction, num_seqs, block_ids, seq_offsets, buf, buf_bytes,
                      img_offsets, target, stream):
    t = ctypes.c_uint64(0)
    st = load().aqua_swap_noalloc(pool, direction, num_seqs, block_ids, seq_offsets, buf,
                                  buf_bytes, img_offsets, target, stream, ctypes.byref(t))
    return st, t.value


def aqua_migrate(pool, src, src_bytes, src_target, dst, dst_bytes, dst_target, n,
                 src_offsets, dst_offsets, lengths, stream):
    t = ctypes.c_uint64(0)
    st = load().aqua_migrate(pool, src, src_bytes, src_target, dst, dst_bytes, dst_target, n,
                             src_offsets, dst_offsets, lengths, stream, ctypes.byref(t))
    return st, t.value


def aqua_sync(pool, ticket: int = 0) -> int:
    return load().aqua_sync(pool, ticket)


def aqua_stream_wait(pool, ticket: int, stream) -> int:
    return load().aqua_stream_wait(pool, ticket, stream)


def aqua_query(pool, ticket: int) -> int:
    return load().aqua_query(pool, ticket)


def aqua_kv_pool_set_max_workgroups(pool, target: int, n: int) -> int:
    return load().aqua_kv_pool_set_max_workgroups(pool, target, n)


def aqua_kv_pool_set_host_path(pool, path: int) -> int:
    return load().aqua_kv_pool_set_host_path(pool, path)


def aqua_kv_pool_set_link_engine(pool, direction: int, engine: int) -> int:
    return load().aqua_kv_pool_set_link_engine(pool, direction, engine)


def aqua_kv_pool_get_link_engine(pool, direction: int):
    e = ctypes.c_int32(0)
    st = load().aqua_kv_pool_get_link_engine(pool, direction, ctypes.byref(e))
    return st, e.value


def aqua_pool_stats_get(pool):
    s = aqua_pool_stats()
    st = load().aqua_pool_stats_get(pool, ctypes.byref(s))
    return st, s


def aqua_hbm_yardstick(kind: int, dst, src, nbytes: int, stream) -> int:
    return load().aqua_hbm_yardstick(kind, dst, src, nbytes, stream)


def hbm_yardstick(kind: int, dst: torch.Tensor, src: Optional[torch.Tensor] = None,
                  stream: Optional[torch.cuda.Stream] = None) -> None:
    """Enqueues one HBM yardstick pass (AQUA_YARDSTICK_COPY / _READ / _WRITE)
    over src's bytes (dst's for a write) on ``stream``; raises AquaError on
    a failed call."""
    nbytes = (src if kind != AQUA_YARDSTICK_WRITE else dst).numel() * \
        (src if kind != AQUA_YARDSTICK_WRITE else dst).element_size()
    st = aqua_hbm_yardstick(kind, dst.data_ptr(), src.data_ptr() if src is not None else None,
                            nbytes, stream.cuda_stream if stream is not None else None)
    if st != AQUA_OK:
        raise AquaError(st, "aqua_hbm_yardstick")


def aqua_status_str(status: int) -> str:
    try:
        return load().aqua_status_str(status).decode()
    except FileNotFoundError:
        return f"status {status}"


def aqua_cfs_partition(requests: np.ndarray, params: aqua_cfs_params,
                       batch_index: np.ndarray, batch_tokens: np.ndarray):
    """requests: uint32 array [n, 4] (the fields of aqua_cfs_request);
    batch_index / batch_tokens: uint32 arrays of n entries.  Returns
    (status, batch size, blocks taken)."""
    n = len(requests)
    size, taken = ctypes.c_uint32(0), ctypes.c_uint64(0)
    st = load().aqua_cfs_partition(
        requests.ctypes.data if n else None, n, ctypes.byref(params),
        batch_index.ctypes.data if n else None, batch_tokens.ctypes.data if n else None,
        ctypes.byref(size), ctypes.byref(taken))
    return st, size.value, taken.value


def cfs_partition(requests, batch_tokens: int, decode_slots: int, capacity_blocks: int,
                  block_tokens: int):
    """One iteration's fair batch (section 7): ``requests`` rows are
    (prompt_tokens, prefill_done, generated, held_blocks).  Returns
    (index array, token array, blocks taken), admission order."""
    req = np.ascontiguousarray(np.asarray(requests, dtype=np.uint32).reshape(-1, 4))
    n = len(req)
    idx = np.zeros(n, dtype=np.uint32)
    tok = np.zeros(n, dtype=np.uint32)
    prm = aqua_cfs_params(batch_tokens, decode_slots, block_tokens, 0, capacity_blocks)
    st, size, taken = aqua_cfs_partition(req, prm, idx, tok)
    if st != AQUA_OK:
        raise AquaError(st, "aqua_cfs_partition")
    return idx[:size], tok[:size], taken


def aqua_swap_space_create(pool, device_bytes: int, host_bytes: int):
    h = ctypes.c_void_p()
    st = load().aqua_swap_space_create(pool, device_bytes, host_bytes, ctypes.byref(h))
    return st, h.value


def aqua_swap_space_destroy(space) -> int:
    return load().aqua_swap_space_destroy(space)


def aqua_swap_alloc(space, nbytes: int):
    h = ctypes.c_uint64(0)
    st = load().aqua_swap_alloc(space, nbytes, ctypes.byref(h))
    return st, h.value


def aqua_swap_free(space, handle: int) -> int:
    return load().aqua_swap_free(space, handle)


def aqua_swap_locate(space, handle: int):
    """(status, pointer, bytes, target)."""
    ptr, nb, tg = ctypes.c_void_p(), ctypes.c_uint64(0), ctypes.c_int32(0)
    st = load().aqua_swap_locate(space, handle, ctypes.byref(ptr), ctypes.byref(nb),
                                 ctypes.byref(tg))
    return st, ptr.value, nb.value, tg.value


def aqua_swap_reclaim(space, nbytes: int, stream):
    t = ctypes.c_uint64(0)
    st = load().aqua_swap_reclaim(space, nbytes, stream, ctypes.byref(t))
    return st, t.value


def aqua_swap_restore(space, stream):
    t = ctypes.c_uint64(0)
    st = load().aqua_swap_restore(space, stream, ctypes.byref(t))
    return st, t.value


def aqua_swap_usage(space):
    """(status, device free bytes, host free bytes, device tensors, host tensors)."""
    v = [ctypes.c_uint64(0) for _ in range(4)]
    st = load().aqua_swap_usage(space, *[ctypes.byref(x) for x in v])
    return (st, *[x.value for x in v])


# -- torch-facing wrapper ------------------------------------------------------

class RawBuffer:
    """A byte buffer the library placed (a swap-space tensor), usable where
    the swap calls take a tensor."""

    def __init__(self, ptr: int, nbytes: int, target: int):
        self.ptr, self.nbytes, self.aqua_target = ptr, nbytes, target

    def data_ptr(self) -> int:
        return self.ptr

    def numel(self) -> int:
        return self.nbytes

    def element_size(self) -> int:
        return 1


def _csr(tables):
    """(int32 ids, uint64 offsets) from a list of tables or an (ids, offs) pair."""
    if isinstance(tables, tuple) and len(tables) == 2 and isinstance(tables[0], np.ndarray):
        ids, offs = tables
    else:
        ids = np.asarray([b for t in tables for b in t], dtype=np.int32)
        offs = np.zeros(len(tables) + 1, dtype=np.uint64)
        if len(tables):
            offs[1:] = np.cumsum([len(t) for t in tables])
    return (np.ascontiguousarray(ids, dtype=np.int32),
            np.ascontiguousarray(offs, dtype=np.uint64))


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream or None


def _target_of(t) -> int:
    if isinstance(t, RawBuffer):
        return t.aqua_target
    if t.is_cuda:
        return AQUA_TARGET_DEVICE
    if t.is_pinned():
        return AQUA_TARGET_HOST
    raise AquaError(AQUA_ERR_INVALID, "offload buffer must be a device or pinned host tensor")


class KVPool:
    """A paged KV pool bound to a caller-owned uint8 device tensor."""

    def __init__(self, shape: Sequence[int], pool: torch.Tensor):
        L, N, H, T, D, dtype = shape
        self.desc = aqua_kv_desc(L, N, H, T, D, dtype)
        self.pool = pool
        st, h = aqua_kv_pool_create(self.desc, pool.data_ptr(),
                                    pool.numel() * pool.element_size())
        if st != AQUA_OK:
            raise AquaError(st, "aqua_kv_pool_create")
        self.handle = h
        self._spaces = []      # swap spaces on this pool, closed before it
        self._held = {}        # ticket -> the tensors its call names, until it completes
        self._prune_at = 64    # prune completed entries when this many are held

    def _hold(self, ticket: int, *tensors) -> None:
        """Keeps the tensors that a call reads or writes alive until the call
        completes: the library only borrows their memory, and a tensor freed
        early could be handed out again while a kernel or a copy engine still
        uses it."""
        if len(self._held) >= self._prune_at:
            done = [t for t in self._held if aqua_query(self.handle, t) == 1]
            for t in done:
                del self._held[t]
            # Amortised: the next pass waits until the held set has doubled.
            self._prune_at = max(64, 2 * len(self._held))
        self._held[ticket] = tensors

    def _swap(self, is_in, tables, buf, img_offsets, stream, target, img_blocks, layers):
        ids, offs = _csr(tables)
        io = None
        if img_offsets is not None:
            io = np.ascontiguousarray(img_offsets, dtype=np.uint64)
        tgt = _target_of(buf) if target is None else target
        args = (self.handle, len(offs) - 1, ids.ctypes.data, offs.ctypes.data,
                buf.data_ptr(), buf.numel() * buf.element_size(),
                None if io is None else io.ctypes.data)
        if img_blocks is None and layers is None:
            fn, name = (aqua_swap_in, "aqua_swap_in") if is_in else (aqua_swap_out, "aqua_swap_out")
            st, ticket = fn(*args, tgt, _stream_handle(stream))
        else:
            ib = None if img_blocks is None else np.ascontiguousarray(img_blocks, dtype=np.uint64)
            l0, nl = (0, 0) if layers is None else layers
            rng = aqua_swap_range(None if ib is None else ib.ctypes.data, l0, nl)
            fn, name = ((aqua_swap_in_ex, "aqua_swap_in_ex") if is_in
                        else (aqua_swap_out_ex, "aqua_swap_out_ex"))
            st, ticket = fn(*args, ctypes.byref(rng), tgt, _stream_handle(stream))
        if st != AQUA_OK:
            raise AquaError(st, name)
        self._hold(ticket, buf)
        return ticket

    def swap_out(self, tables, dst: torch.Tensor, img_offsets=None, stream=None,
                 target=None, img_blocks=None, layers=None) -> int:
        """Gather; ``img_blocks`` (blocks per layer of each image) and
        ``layers`` = (first, count) select the extended form."""
        return self._swap(False, tables, dst, img_offsets, stream, target, img_blocks, layers)

    def swap_in(self, tables, src: torch.Tensor, img_offsets=None, stream=None,
                target=None, img_blocks=None, layers=None) -> int:
        return self._swap(True, tables, src, img_offsets, stream, target, img_blocks, layers)

    def swap_noalloc(self, direction: int, tables, buf: torch.Tensor, img_offsets=None,
                     stream=None, target=None) -> int:
        """aqua_swap_noalloc: swap-out (direction 0) or swap-in (1) that
        allocates nothing."""
        ids, offs = _csr(tables)
        io = None
        if img_offsets is not None:
            io = np.ascontiguousarray(img_offsets, dtype=np.uint64)
        tgt = _target_of(buf) if target is None else target
        st, ticket = aqua_swap_noalloc(
            self.handle, direction, len(offs) - 1, ids.ctypes.data, offs.ctypes.data,
            buf.data_ptr(), buf.numel() * buf.element_size(),
            None if io is None else io.ctypes.data, tgt, _stream_handle(stream))
        if st != AQUA_OK:
            raise AquaError(st, "aqua_swap_noalloc")
        self._hold(ticket, buf)
        return ticket

    def migrate(self, src: torch.Tensor, dst: torch.Tensor, src_offsets, dst_offsets,
                lengths, stream=None) -> int:
        """Copy byte ranges between offload buffers (device or pinned host)."""
        so, do, ln = (np.ascontiguousarray(x, dtype=np.uint64)
                      for x in (src_offsets, dst_offsets, lengths))
        st, ticket = aqua_migrate(self.handle, src.data_ptr(), src.numel() * src.element_size(),
                                  _target_of(src), dst.data_ptr(),
                                  dst.numel() * dst.element_size(), _target_of(dst), len(ln),
                                  so.ctypes.data, do.ctypes.data, ln.ctypes.data,
                                  _stream_handle(stream))
        if st != AQUA_OK:
            raise AquaError(st, "aqua_migrate")
        self._hold(ticket, src, dst)
        return ticket

    def sync(self, ticket: int = 0) -> None:
        st = aqua_sync(self.handle, ticket)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_sync")
        if ticket == 0:
            self._held.clear()
        else:
            self._held.pop(ticket, None)

    def stream_wait(self, ticket: int, stream=None) -> None:
        st = aqua_stream_wait(self.handle, ticket, _stream_handle(stream))
        if st != AQUA_OK:
            raise AquaError(st, "aqua_stream_wait")

    def query(self, ticket: int) -> bool:
        st = aqua_query(self.handle, ticket)
        if st < 0:
            raise AquaError(st, "aqua_query")
        return st == 1

    def set_max_workgroups(self, target: int, n: int) -> None:
        st = aqua_kv_pool_set_max_workgroups(self.handle, target, n)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_kv_pool_set_max_workgroups")

    def set_host_path(self, path: int) -> None:
        st = aqua_kv_pool_set_host_path(self.handle, path)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_kv_pool_set_host_path")

    def set_link_engine(self, direction: int, engine: int) -> None:
        """Carrier of the staged path's link copies for one direction (0:
        swap-out, 1: swap-in): an SDMA engine index, AQUA_LINK_RUNTIME or
        AQUA_LINK_AUTO."""
        st = aqua_kv_pool_set_link_engine(self.handle, direction, engine)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_kv_pool_set_link_engine")

    def link_engine(self, direction: int) -> int:
        st, e = aqua_kv_pool_get_link_engine(self.handle, direction)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_kv_pool_get_link_engine")
        return e

    def stats(self) -> dict:
        st, s = aqua_pool_stats_get(self.handle)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_pool_stats_get")
        return {n: getattr(s, n) for n, _ in s._fields_ if n != "reserved"}

    def close(self) -> None:
        for sp in list(getattr(self, "_spaces", [])):
            sp.close()
        if getattr(self, "handle", None):
            st = aqua_kv_pool_destroy(self.handle)
            self.handle = None
            self._held.clear()   # destroy waited for every call
            if st != AQUA_OK:
                raise AquaError(st, "aqua_kv_pool_destroy")

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


class SwapSpace:
    """Offload tensors with a device region and a pinned-host fallback, on a
    pool (see aqua_swap_space_create)."""

    def __init__(self, pool: "KVPool", device_bytes: int, host_bytes: int):
        st, h = aqua_swap_space_create(pool.handle, device_bytes, host_bytes)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_swap_space_create")
        self.handle = h
        self.pool = pool
        pool._spaces.append(self)

    def alloc(self, nbytes: int) -> int:
        st, h = aqua_swap_alloc(self.handle, nbytes)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_swap_alloc")
        return h

    def free(self, tensor: int) -> None:
        st = aqua_swap_free(self.handle, tensor)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_swap_free")

    def locate(self, tensor: int):
        """(pointer, bytes, target) of a tensor now."""
        st, ptr, nb, tg = aqua_swap_locate(self.handle, tensor)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_swap_locate")
        return ptr, nb, tg

    def buffer(self, tensor: int) -> RawBuffer:
        """The tensor's current bytes, for KVPool.swap_out / swap_in."""
        return RawBuffer(*self.locate(tensor))

    def reclaim(self, nbytes: Optional[int] = None, stream=None) -> int:
        st, t = aqua_swap_reclaim(self.handle, (1 << 64) - 1 if nbytes is None else nbytes,
                                  _stream_handle(stream))
        if st != AQUA_OK:
            raise AquaError(st, "aqua_swap_reclaim")
        return t

    def restore(self, stream=None) -> int:
        st, t = aqua_swap_restore(self.handle, _stream_handle(stream))
        if st != AQUA_OK:
            raise AquaError(st, "aqua_swap_restore")
        return t

    def usage(self) -> dict:
        st, df, hf, dn, hn = aqua_swap_usage(self.handle)
        if st != AQUA_OK:
            raise AquaError(st, "aqua_swap_usage")
        return {"device_free": df, "host_free": hf, "device_tensors": dn, "host_tensors": hn}

    def close(self) -> None:
        if getattr(self, "handle", None):
            st = aqua_swap_space_destroy(self.handle)
            self.handle = None
            self.pool._spaces.remove(self)
            if st != AQUA_OK:
                raise AquaError(st, "aqua_swap_space_destroy")

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
