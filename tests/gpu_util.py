"""Helpers for the GPU parity tests: generated inputs on the device, host
copies for the oracle, and the oracle's replay of a preemption schedule."""
from __future__ import annotations

import ctypes
import sys
import threading

import numpy as np
import torch

import oracle
from paper_2407_21255_amd import workload as wl


def say(*a):
    """Progress line that reaches the log even if the process dies next."""
    print(*a, file=sys.stderr, flush=True)


def odesc(shape: wl.KVShape) -> oracle.KVDesc:
    return oracle.desc(*shape.as_tuple())


def device_pool(shape: wl.KVShape, seed: int, owner=None, extra: int = 0) -> torch.Tensor:
    pool = torch.empty(shape.pool_bytes + extra, dtype=torch.uint8, device="cuda")
    wl.fill_pool(pool, shape, seed, owner)
    if extra:
        pool[shape.pool_bytes:].fill_(wl.GUARD_BYTE)
    return pool


def host(t: torch.Tensor) -> np.ndarray:
    """Host copy (pageable numpy array) of a tensor."""
    torch.cuda.synchronize()
    return t.detach().to("cpu", copy=True).numpy()


def guarded_buffer(nbytes: int, guard: int = 4096, pinned: bool = False) -> torch.Tensor:
    if pinned:
        buf = torch.empty(nbytes + 2 * guard, dtype=torch.uint8, pin_memory=True)
    else:
        buf = torch.empty(nbytes + 2 * guard, dtype=torch.uint8, device="cuda")
    buf.fill_(wl.GUARD_BYTE)
    return buf


def region_for(sched: wl.Schedule, device="cuda") -> torch.Tensor:
    reg = torch.empty(sched.region_bytes, dtype=torch.uint8, device=device)
    wl.fill_region(reg, sched)
    return reg


def schedule_owner(sched: wl.Schedule) -> dict:
    return wl.schedule_owner(sched)


def apply_mutations_host(sched, s, pool_np, region_np):
    offs, words, slots = wl.mutation_writes(sched, s)
    for o, w in zip(offs, words):
        pool_np[o:o + 16] = w
    for o, n in slots:
        region_np[o:o + n] = wl.CONSUMED_BYTE


def apply_pool_mutations_device(sched, s, pool_t):
    """The residents' 16-byte stamps of slice s (no offload-slot marks)."""
    offs, words, _ = wl.mutation_writes(sched, s)
    if len(offs):
        idx = torch.from_numpy(offs).to(pool_t.device).reshape(-1, 1) + \
            torch.arange(16, device=pool_t.device).reshape(1, -1)
        pool_t[idx.reshape(-1)] = torch.from_numpy(words.reshape(-1)).to(pool_t.device)


def apply_mutations_device(sched, s, pool_t, region_t):
    offs, words, slots = wl.mutation_writes(sched, s)
    if len(offs):
        idx = torch.from_numpy(offs).to(pool_t.device).reshape(-1, 1) + \
            torch.arange(16, device=pool_t.device).reshape(1, -1)
        pool_t[idx.reshape(-1)] = torch.from_numpy(words.reshape(-1)).to(pool_t.device)
    for o, n in slots:
        region_t[o:o + n].fill_(wl.CONSUMED_BYTE)


def apply_pool_mutations_host(sched, s, pool_np):
    offs, words, _ = wl.mutation_writes(sched, s)
    for o, w in zip(offs, words):
        pool_np[o:o + 16] = w


def oracle_replay(sched, pool_np, region_np, first, count, mutate=True, grow=True,
                  slot_marks=True):
    """The oracle's run of slices [first, first+count) in issue order; the
    compute stand-in (KV growth, mutations) between slices where asked."""
    d = odesc(sched.shape)
    for s in range(first, first + count):
        if (s - first) % 10 == 0:
            say("oracle replay: slice", s)
        sl = sched.slices[s]
        out_off = [sched.slot_offsets[p] for p in sl.out_prompts]
        in_off = [sched.slot_offsets[p] for p in sl.in_prompts]
        assert oracle.swap_out(d, pool_np, sl.out_tables, region_np, out_off) == 0
        assert oracle.swap_in(d, pool_np, sl.in_tables, region_np, in_off) == 0
        if grow and sl.grow:
            wl.apply_growth(torch.from_numpy(pool_np), sched, s)
        if mutate and slot_marks:
            apply_mutations_host(sched, s, pool_np, region_np)
        elif mutate:
            apply_pool_mutations_host(sched, s, pool_np)


class _PointerAttributes(ctypes.Structure):
    _fields_ = [("type", ctypes.c_int), ("device", ctypes.c_int),
                ("devicePointer", ctypes.c_void_p), ("hostPointer", ctypes.c_void_p),
                ("isManaged", ctypes.c_int), ("allocationFlags", ctypes.c_uint)]


def _hip_runtime() -> ctypes.CDLL:
    """The HIP runtime that torch has loaded (the library binds to it too)."""
    for line in open("/proc/self/maps"):
        path = line.split()[-1]
        if "libamdhip64" in path:
            lib = ctypes.CDLL(path)
            break
    else:
        raise RuntimeError("the HIP runtime is not loaded")
    P = ctypes.c_void_p
    lib.hipExtMallocWithFlags.argtypes = [ctypes.POINTER(P), ctypes.c_size_t, ctypes.c_uint]
    lib.hipPointerGetAttributes.argtypes = [ctypes.POINTER(_PointerAttributes), P]
    lib.hipFree.argtypes = [P]
    lib.hipStreamWaitValue32.argtypes = [P, P, ctypes.c_uint32, ctypes.c_uint, ctypes.c_uint32]
    for f in (lib.hipExtMallocWithFlags, lib.hipPointerGetAttributes, lib.hipFree,
              lib.hipStreamWaitValue32):
        f.restype = ctypes.c_int
    return lib


class HostGate:
    """A 32-bit flag in the runtime's signal memory that holds a stream
    (hipStreamWaitValue32 until it equals 1) until the host opens it: the
    host decides when the held stream goes on.  A timer opens it after
    `failsafe` seconds whatever the test does, and close() opens it and waits
    for the device before freeing it, so no stream is left waiting."""

    SIGNAL_MEMORY = 0x2      # hipMallocSignalMemory
    WAIT_EQ = 0x1            # hipStreamWaitValueEq

    def __init__(self, failsafe: float = 30.0):
        self.hip = _hip_runtime()
        p = ctypes.c_void_p()
        assert self.hip.hipExtMallocWithFlags(ctypes.byref(p), 8, self.SIGNAL_MEMORY) == 0
        self.ptr = p.value
        attr = _PointerAttributes()
        assert self.hip.hipPointerGetAttributes(ctypes.byref(attr), self.ptr) == 0
        assert attr.hostPointer, "signal memory without a host address"
        self.flag = ctypes.c_uint32.from_address(attr.hostPointer)
        self.flag.value = 0
        self.timer = threading.Timer(failsafe, self.open)
        self.timer.start()

    def hold(self, stream: torch.cuda.Stream) -> None:
        rc = self.hip.hipStreamWaitValue32(ctypes.c_void_p(stream.cuda_stream),
                                           ctypes.c_void_p(self.ptr), 1, self.WAIT_EQ,
                                           0xFFFFFFFF)
        assert rc == 0, rc

    def open(self) -> None:
        self.flag.value = 1

    def close(self) -> None:
        self.open()
        self.timer.cancel()
        torch.cuda.synchronize()
        self.hip.hipFree(ctypes.c_void_p(self.ptr))
