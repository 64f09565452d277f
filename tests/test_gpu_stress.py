"""GPU parity under a random mix of calls: seeded swap-outs, swap-ins and
migrations (arena <-> a device region) on four streams with no host sync in
between, their images at random, often overlapping, offsets of one arena.
The arena is pinned host memory, staged through small HBM slots so that
every call is several copy-engine jobs, or swapped zero-copy; or it is in
HBM.  The library must behave as if the calls ran in issue order: pool,
arena and region at the end equal the oracle run call by call in that
order."""
import ctypes
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2407_21255_amd import aqua
from paper_2407_21255_amd import workload as wl
from tests.checkers import assert_bytes_equal
from tests.gpu_util import device_pool, host, odesc, say

ARENA = 4 << 20
REGION = 4 << 20
OPS = int(os.environ.get("AQUA_TEST_STRESS_OPS", "150"))   # calls per run


def _ops(shape, rng, count):
    """A seeded call list: (kind, stream, args)."""
    N, unit = shape.num_blocks, shape.num_layers * shape.chunk_bytes
    ops = []
    for _ in range(count):
        kind = rng.choice(["out", "out", "in", "in", "to_host", "to_device"])
        stream = int(rng.integers(0, 4))
        if kind in ("out", "in"):
            n = int(rng.integers(1, 25))
            if kind == "out" and rng.random() < 0.2:
                table = rng.integers(0, N, size=n)                 # repeats allowed
            else:
                table = rng.choice(N, size=n, replace=False)
            size = n * unit
            off = int(rng.integers(0, (ARENA - size) // 16 + 1)) * 16
            ops.append((kind, stream, ([int(b) for b in table], off, size)))
        else:
            k = int(rng.integers(1, 4))
            lens = [int(rng.integers(1, 16 << 10)) * 16 for _ in range(k)]
            total = sum(lens)

            def consecutive(limit):
                # Ranges one after another from a random base: never overlapping.
                pos = int(rng.integers(0, (limit - total) // 16 + 1)) * 16
                offs = []
                for ln in lens:
                    offs.append(pos)
                    pos += ln
                return offs

            # (arena offsets, region offsets, lengths)
            ops.append((kind, stream, (consecutive(ARENA), consecutive(REGION), lens)))
    return ops


@pytest.mark.gpu
@pytest.mark.parametrize("path,seed", [("staged", 1), ("staged", 2), ("zero_copy", 3),
                                       ("hbm", 4)])
def test_random_calls_on_four_streams(monkeypatch, path, seed):
    """`path`: where the arena lives and how host swaps move (staged on the
    copy engines, zero-copy kernels, or an arena in HBM, where migrations
    are device copies too)."""
    monkeypatch.setenv("AQUA_STAGE_SLOT_BYTES", str(64 << 10))
    shape = wl.KVShape(4, 256, 2, 16, 64, wl.BF16)                # 8 KiB chunks
    d = odesc(shape)
    rng = np.random.default_rng(seed)
    pool = device_pool(shape, 40 + seed)
    fill = torch.from_numpy(rng.integers(0, 256, size=ARENA, dtype=np.uint8))
    if path == "hbm":
        arena = fill.cuda()
    else:
        arena = torch.empty(ARENA, dtype=torch.uint8, pin_memory=True)
        arena.copy_(fill)
    region = torch.from_numpy(rng.integers(0, 256, size=REGION, dtype=np.uint8)).cuda()
    pool_h, arena_h, region_h = host(pool), host(arena).copy(), host(region)
    ops = _ops(shape, rng, OPS)
    say("stress", path, seed, {k: sum(1 for o in ops if o[0] == k)
                               for k in ("out", "in", "to_host", "to_device")})
    streams = [torch.cuda.Stream() for _ in range(4)]
    torch.cuda.synchronize()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        kv.set_host_path(aqua.AQUA_HOST_ZERO_COPY if path == "zero_copy"
                         else aqua.AQUA_HOST_STAGED)
        for kind, si, args in ops:
            s = streams[si]
            if kind == "out":
                table, off, size = args
                kv.swap_out([table], arena[off:off + size], stream=s)
            elif kind == "in":
                table, off, size = args
                kv.swap_in([table], arena[off:off + size], stream=s)
            elif kind == "to_host":
                ao, ro, lens = args
                kv.migrate(region, arena, ro, ao, lens, stream=s)
            else:
                ao, ro, lens = args
                kv.migrate(arena, region, ao, ro, lens, stream=s)
        st = kv.stats()
        kv.sync()
        say("carriers", [kv.link_engine(0), kv.link_engine(1)],
            "waits inserted", st["waits_inserted"], "elided", st["waits_elided"])
    finally:
        kv.close()
    for kind, _, args in ops:
        if kind == "out":
            table, off, size = args
            assert oracle.swap_out(d, pool_h, [table], arena_h[off:off + size]) == 0
        elif kind == "in":
            table, off, size = args
            assert oracle.swap_in(d, pool_h, [table], arena_h[off:off + size]) == 0
        elif kind == "to_host":
            ao, ro, lens = args
            assert oracle.migrate(region_h, arena_h, ro, ao, lens) == 0
        else:
            ao, ro, lens = args
            assert oracle.migrate(arena_h, region_h, ao, ro, lens) == 0
    assert_bytes_equal(host(pool), pool_h, "pool")
    assert_bytes_equal(host(arena), arena_h, "arena")
    assert_bytes_equal(host(region), region_h, "device region")


@pytest.mark.gpu
def test_random_calls_on_rotating_streams():
    """The stream set changes as the calls go: call i runs on one of the
    four streams of a window that moves on by one stream every five calls,
    over 64 streams made for the test (plain HIP streams, so every handle
    is new).  The library hands lanes whose calls have all completed to
    streams it has not seen, and must still order conflicting calls across
    them: pool, arena and region equal the oracle run in issue order."""
    from tests.gpu_util import _hip_runtime
    hip = _hip_runtime()
    hip.hipStreamCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    handles = []
    for _ in range(64):
        h = ctypes.c_void_p()
        assert hip.hipStreamCreateWithFlags(ctypes.byref(h), 1) == 0   # non-blocking
        handles.append(h.value)
    shape = wl.KVShape(4, 256, 2, 16, 64, wl.BF16)                # 8 KiB chunks
    d = odesc(shape)
    rng = np.random.default_rng(9)
    pool = device_pool(shape, 49)
    arena = torch.from_numpy(rng.integers(0, 256, size=ARENA, dtype=np.uint8)).cuda()
    region = torch.from_numpy(rng.integers(0, 256, size=REGION, dtype=np.uint8)).cuda()
    pool_h, arena_h, region_h = host(pool), host(arena).copy(), host(region)
    ops = _ops(shape, rng, 300)
    torch.cuda.synchronize()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        for i, (kind, si, args) in enumerate(ops):
            s = handles[(i // 5 + si) % len(handles)]
            if kind == "out":
                table, off, size = args
                kv.swap_out([table], arena[off:off + size], stream=s)
            elif kind == "in":
                table, off, size = args
                kv.swap_in([table], arena[off:off + size], stream=s)
            elif kind == "to_host":
                ao, ro, lens = args
                kv.migrate(region, arena, ro, ao, lens, stream=s)
            else:
                ao, ro, lens = args
                kv.migrate(arena, region, ao, ro, lens, stream=s)
        st = kv.stats()
        kv.sync()
        say("rotating streams: waits inserted", st["waits_inserted"], "elided",
            st["waits_elided"])
    finally:
        kv.close()
        torch.cuda.synchronize()
        for h in handles:
            hip.hipStreamDestroy(ctypes.c_void_p(h))
    for kind, _, args in ops:
        if kind == "out":
            table, off, size = args
            assert oracle.swap_out(d, pool_h, [table], arena_h[off:off + size]) == 0
        elif kind == "in":
            table, off, size = args
            assert oracle.swap_in(d, pool_h, [table], arena_h[off:off + size]) == 0
        elif kind == "to_host":
            ao, ro, lens = args
            assert oracle.migrate(region_h, arena_h, ro, ao, lens) == 0
        else:
            ao, ro, lens = args
            assert oracle.migrate(arena_h, region_h, ao, ro, lens) == 0
    assert_bytes_equal(host(pool), pool_h, "pool")
    assert_bytes_equal(host(arena), arena_h, "arena")
    assert_bytes_equal(host(region), region_h, "device region")
    assert st["waits_inserted"] > 0
