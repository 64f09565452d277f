"""ctypes access to libaqua_core.so: the library's host core (validation,
run planning, hazard tracking, the swap space's range allocator) built
without HIP for CPU tests."""
from __future__ import annotations

import ctypes
import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# AQUA_CORE_LIB names another build of the core (the sanitizer build).
CORE = os.environ.get("AQUA_CORE_LIB") or os.path.join(ROOT, "paper_2407_21255_amd",
                                                       "libaqua_core.so")

RUN_DESC = np.dtype([("img_off", "<u8"), ("img_lstride", "<u8"), ("block", "<u4"),
                     ("nchunks", "<u4"), ("r0", "<u4"), ("r1", "<u4")])
assert RUN_DESC.itemsize == 32


class Desc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_uint32), ("num_blocks", ctypes.c_uint32),
                ("num_kv_heads", ctypes.c_uint32), ("block_tokens", ctypes.c_uint32),
                ("head_dim", ctypes.c_uint32), ("dtype", ctypes.c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(CORE):
            from paper_2407_21255_amd import build
            build.build_core()
        L = ctypes.CDLL(CORE)
        P, u32, u64, i32, i64 = (ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64,
                                 ctypes.c_int32, ctypes.c_int64)
        L.aqua_core_validate.argtypes = [ctypes.POINTER(Desc), u32, P, P, u64, u64, P, i32]
        L.aqua_core_validate.restype = i32
        L.aqua_core_plan.argtypes = [ctypes.POINTER(Desc), u32, P, P, P, u64, P, u64]
        L.aqua_core_plan.restype = i64
        L.aqua_core_plan_ex.argtypes = [ctypes.POINTER(Desc), u32, P, P, P, P, u64, P, u64]
        L.aqua_core_plan_ex.restype = i64
        L.aqua_core_validate_ex.argtypes = [ctypes.POINTER(Desc), u32, P, P, u64, u64, P, P,
                                            u32, u32, i32]
        L.aqua_core_validate_ex.restype = i32
        L.aqua_core_validate_migrate.argtypes = [u64, u64, u64, u64, u32, P, P, P]
        L.aqua_core_validate_migrate.restype = i32
        L.aqua_core_tracker_new.argtypes = [u32]
        L.aqua_core_tracker_new.restype = P
        L.aqua_core_tracker_free.argtypes = [P]
        L.aqua_core_tracker_issue.argtypes = [P, u64, u32, i32, P, u64, P, u64, P, P, u64]
        L.aqua_core_tracker_issue.restype = i64
        L.aqua_core_tracker_issue_rw.argtypes = [P, u64, u32, P, u64, P, u64, P, u64, P, u64,
                                                 P, P, u64]
        L.aqua_core_tracker_issue_rw.restype = i64
        L.aqua_core_tracker_complete.argtypes = [P, u32, u64]
        L.aqua_core_tracker_live_ranges.argtypes = [P]
        for n in ("aqua_core_tracker_tickets_kept", "aqua_core_tracker_lanes"):
            getattr(L, n).argtypes = [P]
            getattr(L, n).restype = u64
        L.aqua_core_tracker_done.argtypes = [P, u64]
        L.aqua_core_tracker_done.restype = i32
        L.aqua_core_lanes_new.restype = P
        L.aqua_core_lanes_free.argtypes = [P]
        L.aqua_core_lanes_lane_for.argtypes = [P, u64, P]
        L.aqua_core_lanes_lane_for.restype = u32
        L.aqua_core_lanes_size.argtypes = [P]
        L.aqua_core_lanes_size.restype = u64
        L.aqua_core_tracker_soak.argtypes = [u64, u32, u32, u64, u32, ctypes.POINTER(u64),
                                             ctypes.POINTER(u64)]
        L.aqua_core_swap_threads.argtypes = [u64, u32]
        L.aqua_core_swap_threads.restype = u32
        L.aqua_core_sort_by_block.argtypes = [P, u64, u32]
        L.aqua_core_interleave_runs.argtypes = [P, u64, u32]
        L.aqua_core_xcd_ways.restype = u32
        L.aqua_core_xcd_unit.argtypes = [u32, u32]
        L.aqua_core_xcd_unit.restype = u32
        L.aqua_core_xcd_unit_order.argtypes = [u64, i32]
        L.aqua_core_xcd_unit_order.restype = i32
        L.aqua_core_run_order.argtypes = [i32, u64, u64, u32, u32]
        L.aqua_core_run_order.restype = i32
        L.aqua_core_layers_per_launch.argtypes = [u32]
        L.aqua_core_layers_per_launch.restype = u32
        L.aqua_core_launch_grid.argtypes = [u64, u32]
        L.aqua_core_launch_grid.restype = u32
        L.aqua_core_tracker_live_ranges.restype = u64
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def validate(desc: Desc, ids, offs, buf_addr, buf_bytes, img_offsets=None, is_in=False,
             num_seqs=None):
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    offs = np.ascontiguousarray(offs, dtype=np.uint64)
    io = None if img_offsets is None else np.ascontiguousarray(img_offsets, dtype=np.uint64)
    ns = len(offs) - 1 if num_seqs is None else num_seqs
    return lib().aqua_core_validate(ctypes.byref(desc), ns, _p(ids), _p(offs), buf_addr,
                                    buf_bytes, _p(io), int(is_in))


def validate_ex(desc: Desc, ids, offs, buf_addr, buf_bytes, img_offsets=None,
                img_blocks=None, first_layer=0, num_layers=0, is_in=False):
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    offs = np.ascontiguousarray(offs, dtype=np.uint64)
    io = None if img_offsets is None else np.ascontiguousarray(img_offsets, dtype=np.uint64)
    ib = None if img_blocks is None else np.ascontiguousarray(img_blocks, dtype=np.uint64)
    return lib().aqua_core_validate_ex(ctypes.byref(desc), len(offs) - 1, _p(ids), _p(offs),
                                       buf_addr, buf_bytes, _p(io), _p(ib), first_layer,
                                       num_layers, int(is_in))


def validate_migrate(src, src_bytes, dst, dst_bytes, so, do, ln):
    so, do, ln = (np.ascontiguousarray(x, dtype=np.uint64) for x in (so, do, ln))
    return lib().aqua_core_validate_migrate(src, src_bytes, dst, dst_bytes, len(ln), _p(so),
                                            _p(do), _p(ln))


def plan_ex(desc: Desc, ids, offs, img_offsets=None, img_blocks=None, unit_bytes=64 << 10):
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    offs = np.ascontiguousarray(offs, dtype=np.uint64)
    io = None if img_offsets is None else np.ascontiguousarray(img_offsets, dtype=np.uint64)
    ib = None if img_blocks is None else np.ascontiguousarray(img_blocks, dtype=np.uint64)
    n = lib().aqua_core_plan_ex(ctypes.byref(desc), len(offs) - 1, _p(ids), _p(offs), _p(io),
                                _p(ib), unit_bytes, None, 0)
    out = np.zeros(n, dtype=RUN_DESC)
    lib().aqua_core_plan_ex(ctypes.byref(desc), len(offs) - 1, _p(ids), _p(offs), _p(io),
                            _p(ib), unit_bytes, _p(out), n)
    return out


def plan(desc: Desc, ids, offs, img_offsets=None, unit_bytes=64 << 10):
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    offs = np.ascontiguousarray(offs, dtype=np.uint64)
    io = None if img_offsets is None else np.ascontiguousarray(img_offsets, dtype=np.uint64)
    n = lib().aqua_core_plan(ctypes.byref(desc), len(offs) - 1, _p(ids), _p(offs), _p(io),
                             unit_bytes, None, 0)
    assert n >= 0, n
    out = np.zeros(n, dtype=RUN_DESC)
    lib().aqua_core_plan(ctypes.byref(desc), len(offs) - 1, _p(ids), _p(offs), _p(io),
                         unit_bytes, _p(out), n)
    return out


class Tracker:
    def __init__(self, num_blocks: int):
        self.h = lib().aqua_core_tracker_new(num_blocks)

    def issue(self, ticket, lane, is_in, blocks, ranges):
        b = np.ascontiguousarray(blocks, dtype=np.int32)
        r = np.ascontiguousarray(np.asarray(ranges, dtype=np.uint64).reshape(-1))
        lanes = np.zeros(64, dtype=np.uint32)
        tickets = np.zeros(64, dtype=np.uint64)
        n = lib().aqua_core_tracker_issue(self.h, ticket, lane, int(is_in), _p(b), b.size,
                                          _p(r), r.size // 2, _p(lanes), _p(tickets), 64)
        assert 0 <= n <= 64
        return [(int(lanes[k]), int(tickets[k])) for k in range(n)]

    def issue_rw(self, ticket, lane, blocks_r, blocks_w, ranges_r, ranges_w):
        br = np.ascontiguousarray(blocks_r, dtype=np.int32)
        bw = np.ascontiguousarray(blocks_w, dtype=np.int32)
        rr = np.ascontiguousarray(np.asarray(ranges_r, dtype=np.uint64).reshape(-1))
        rw = np.ascontiguousarray(np.asarray(ranges_w, dtype=np.uint64).reshape(-1))
        lanes = np.zeros(64, dtype=np.uint32)
        tickets = np.zeros(64, dtype=np.uint64)
        n = lib().aqua_core_tracker_issue_rw(self.h, ticket, lane, _p(br), br.size, _p(bw),
                                             bw.size, _p(rr), rr.size // 2, _p(rw),
                                             rw.size // 2, _p(lanes), _p(tickets), 64)
        assert 0 <= n <= 64
        return [(int(lanes[k]), int(tickets[k])) for k in range(n)]

    def complete(self, lane, ticket):
        lib().aqua_core_tracker_complete(self.h, lane, ticket)

    def live_ranges(self):
        return int(lib().aqua_core_tracker_live_ranges(self.h))

    def tickets_kept(self):
        return int(lib().aqua_core_tracker_tickets_kept(self.h))

    def lanes(self):
        return int(lib().aqua_core_tracker_lanes(self.h))

    def done(self, ticket):
        return bool(lib().aqua_core_tracker_done(self.h, ticket))

    def __del__(self):
        if getattr(self, "h", None):
            lib().aqua_core_tracker_free(self.h)
            self.h = None


class Ranges:
    """The core's first-fit range allocator."""

    def __init__(self, size: int, align: int):
        L = lib()
        u64, P = ctypes.c_uint64, ctypes.c_void_p
        L.aqua_core_ranges_new.argtypes = [u64, u64]
        L.aqua_core_ranges_new.restype = P
        L.aqua_core_ranges_free_all.argtypes = [P]
        L.aqua_core_ranges_alloc.argtypes = [P, u64, ctypes.POINTER(u64)]
        L.aqua_core_ranges_alloc.restype = ctypes.c_int
        L.aqua_core_ranges_release.argtypes = [P, u64]
        L.aqua_core_ranges_release.restype = ctypes.c_int
        L.aqua_core_ranges_free_bytes.argtypes = [P]
        L.aqua_core_ranges_free_bytes.restype = u64
        L.aqua_core_ranges_largest_free.argtypes = [P]
        L.aqua_core_ranges_largest_free.restype = u64
        self.L = L
        self.h = L.aqua_core_ranges_new(size, align)

    def alloc(self, nbytes: int):
        off = ctypes.c_uint64(0)
        return off.value if self.L.aqua_core_ranges_alloc(self.h, nbytes, ctypes.byref(off)) else None

    def free(self, off: int) -> bool:
        return bool(self.L.aqua_core_ranges_release(self.h, off))

    def free_bytes(self) -> int:
        return int(self.L.aqua_core_ranges_free_bytes(self.h))

    def largest_free(self) -> int:
        return int(self.L.aqua_core_ranges_largest_free(self.h))

    def close(self):
        if self.h:
            self.L.aqua_core_ranges_free_all(self.h)
            self.h = None


class LaneMap:
    """The core's stream -> lane map, over a Tracker."""

    def __init__(self):
        self.h = lib().aqua_core_lanes_new()

    def lane_for(self, stream: int, tracker: "Tracker") -> int:
        return int(lib().aqua_core_lanes_lane_for(self.h, stream, tracker.h))

    def size(self) -> int:
        return int(lib().aqua_core_lanes_size(self.h))

    def __del__(self):
        if getattr(self, "h", None):
            lib().aqua_core_lanes_free(self.h)
            self.h = None


def swap_threads(chunk_bytes: int, min_threads: int) -> int:
    return int(lib().aqua_core_swap_threads(chunk_bytes, min_threads))


def launch_grid(units: int, max_workgroups: int) -> int:
    return int(lib().aqua_core_launch_grid(units, max_workgroups))


def tracker_soak(n_calls: int, num_blocks: int, streams: int, rotate: int, depth: int):
    """(largest tickets kept, largest lane count) over a simulated serving
    loop; see aqua_core_tracker_soak."""
    kept, lanes = ctypes.c_uint64(0), ctypes.c_uint64(0)
    lib().aqua_core_tracker_soak(n_calls, num_blocks, streams, rotate, depth,
                                 ctypes.byref(kept), ctypes.byref(lanes))
    return int(kept.value), int(lanes.value)


TABLE, SORTED_DEALT, TABLE_DEALT = 0, 1, 2   # aqua::RunOrder


def run_order(is_in: bool, chunk_bytes: int, blocks: int, num_blocks: int,
              num_seqs: int = 1) -> int:
    return int(lib().aqua_core_run_order(int(is_in), chunk_bytes, blocks, num_blocks, num_seqs))


def sort_by_block(descs: np.ndarray, num_blocks: int) -> np.ndarray:
    """The core's counting sort of RUN_DESC records by block (a copy)."""
    out = np.ascontiguousarray(descs.copy())
    lib().aqua_core_sort_by_block(out.ctypes.data if len(out) else None, len(out), num_blocks)
    return out


def interleave_runs(descs: np.ndarray, ways: int) -> np.ndarray:
    """The core's XCD-aware reordering of RUN_DESC records (a copy)."""
    out = np.ascontiguousarray(descs.copy())
    lib().aqua_core_interleave_runs(out.ctypes.data if len(out) else None, len(out), ways)
    return out


def xcd_ways() -> int:
    return int(lib().aqua_core_xcd_ways())


def xcd_unit(block: int, units: int) -> int:
    return int(lib().aqua_core_xcd_unit(block, units))


def xcd_unit_order(chunk_bytes: int, dealt: bool) -> bool:
    return bool(lib().aqua_core_xcd_unit_order(chunk_bytes, int(dealt)))


def layers_per_launch(ndesc: int) -> int:
    return int(lib().aqua_core_layers_per_launch(ndesc))
