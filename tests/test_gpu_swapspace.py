"""GPU parity of the swap space: offload tensors placed in a device region or,
when it is full, in pinned host memory; reclaim moving them to host memory
and restore moving them back, on the pool's ordering, with no host sync
between the calls; each tensor's bytes checked against the oracle, read back
with the HIP runtime's own copy."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2407_21255_amd import aqua
from paper_2407_21255_amd import workload as wl
from tests.checkers import assert_bytes_equal
from tests.gpu_util import device_pool, host, odesc, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    aqua.load()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _read(ptr: int, nbytes: int) -> np.ndarray:
    """Bytes at a device or pinned host address, copied by the runtime."""
    torch.cuda.synchronize()
    hip = ctypes.CDLL("libamdhip64.so.7")
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    out = np.empty(nbytes, dtype=np.uint8)
    assert hip.hipMemcpy(out.ctypes.data, ptr, nbytes, 4) == 0     # hipMemcpyDefault
    return out


def test_swap_space_fallback_reclaim_and_restore():
    shape = wl.KVShape(8, 2048, 4, 16, 64, wl.BF16)      # 16 KiB chunks
    d = odesc(shape)
    case = wl.fragmented_case("space", shape, 41, 12, 40, 8)
    img = shape.image_bytes(40)                           # 5 MiB per prompt
    pool = device_pool(shape, case.seed, case.owner)
    pool_h = host(pool)
    sa, sb, sc = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    space = aqua.SwapSpace(kv, 3 * img + (1 << 20), 12 * img)
    try:
        hs = [space.alloc(img) for _ in case.out_tables]
        u = space.usage()
        assert (u["device_tensors"], u["host_tensors"]) == (3, 5), u
        assert [space.locate(h)[2] for h in hs] == [aqua.AQUA_TARGET_DEVICE] * 3 + \
            [aqua.AQUA_TARGET_HOST] * 5
        # Swap-outs into the tensors, then a reclaim of the device region and
        # new tensors in the vacated range, all without host syncs.  A bounded
        # spin ahead of them keeps the swap-outs pending while the reclaim is
        # issued, so the reclaim must wait for them on the device.
        for s in (sa, sb):
            with torch.cuda.stream(s):
                torch.cuda._sleep(20_000_000)
        for k, (h, t) in enumerate(zip(hs, case.out_tables)):
            kv.swap_out([t], space.buffer(h), stream=sa if k % 2 else sb)
        t_rec = space.reclaim(stream=sc)
        assert t_rec > 0
        u = space.usage()
        assert (u["device_tensors"], u["host_tensors"]) == (0, 8), u
        # Residents 8 and 9 go out into two new tensors, which reuse the
        # device range the reclaim is still reading from.
        extra_tables = [t for p, t in enumerate(_tables_of(case)) if p in (8, 9)]
        hx = [space.alloc(img) for _ in extra_tables]
        assert all(space.locate(h)[2] == aqua.AQUA_TARGET_DEVICE for h in hx)
        for h, t in zip(hx, extra_tables):
            kv.swap_out([t], space.buffer(h), stream=sa)
        # Swap the 8 preempted prompts back in from wherever they are now.
        for h, t in zip(hs, case.in_tables):
            kv.swap_in([t], space.buffer(h), stream=sb)
        kv.sync()
        st = kv.stats()
        say("swap space", st, space.usage())
        assert st["waits_inserted"] > 0
        # Oracle: images of the preempted and the two extra prompts, then
        # the swap-ins.
        want = []
        for t in case.out_tables:
            a = np.zeros(img, dtype=np.uint8)
            assert oracle.swap_out(d, pool_h, [t], a) == 0
            want.append(a)
        want_x = []
        for t in extra_tables:
            a = np.zeros(img, dtype=np.uint8)
            assert oracle.swap_out(d, pool_h, [t], a) == 0
            want_x.append(a)
        for t, a in zip(case.in_tables, want):
            assert oracle.swap_in(d, pool_h, [t], a) == 0
        assert_bytes_equal(host(pool), pool_h, "pool after swap-ins from reclaimed tensors")
        for h, a in zip(hs, want):
            ptr, nb, tg = space.locate(h)
            assert tg == aqua.AQUA_TARGET_HOST and nb == img
            assert_bytes_equal(_read(ptr, nb), a, f"reclaimed tensor {h}")
        for h, a in zip(hx, want_x):
            ptr, nb, _ = space.locate(h)
            assert_bytes_equal(_read(ptr, nb), a, f"new tensor {h} in the vacated range")
        # Restore: host tensors move back, oldest first, while the device
        # region has room.  With hx[0] freed, 5 MiB at offset 0 and 6 MiB at
        # 10 MiB are free: hs[0] and hs[1] move, hs[2] does not fit.
        space.free(hx[0])
        t_res = space.restore(stream=sc)
        assert t_res > 0
        u = space.usage()
        assert u["device_tensors"] == 3 and u["host_tensors"] == 6, u
        assert [space.locate(h)[2] for h in hs[:3]] == [aqua.AQUA_TARGET_DEVICE] * 2 + \
            [aqua.AQUA_TARGET_HOST]
        kv.stream_wait(t_res, torch.cuda.current_stream())
        for h, a in zip(hs, want):
            ptr, nb, _ = space.locate(h)
            assert_bytes_equal(_read(ptr, nb), a, f"restored tensor {h}")
        assert_bytes_equal(_read(*space.locate(hx[1])[:2]), want_x[1], "kept tensor")
    finally:
        space.close()
        kv.close()


def _tables_of(case):
    """Block table of every prompt of a fragmented case, by prompt."""
    by = {}
    for b, (p, i) in case.owner.items():
        by.setdefault(p, {})[i] = b
    return [[by[p][i] for i in range(len(by[p]))] for p in sorted(by)]


def test_swap_space_errors_leave_no_trace():
    shape = wl.KVShape(2, 64, 1, 2, 8, wl.BF16)
    pool = device_pool(shape, 3)
    kv = aqua.KVPool(shape.as_tuple(), pool)
    space = aqua.SwapSpace(kv, 4096, 8192)
    try:
        for nbytes, code in [(0, aqua.AQUA_ERR_INVALID), (24, aqua.AQUA_ERR_INVALID),
                             (16384, aqua.AQUA_ERR_CAPACITY)]:
            with pytest.raises(aqua.AquaError) as ei:
                space.alloc(nbytes)
            assert ei.value.status == code
        for fn in (space.free, space.locate):
            with pytest.raises(aqua.AquaError) as ei:
                fn(12345)
            assert ei.value.status == aqua.AQUA_ERR_INVALID
        a = space.alloc(4096)           # fills the device region
        b = space.alloc(8192)           # fills the host region
        assert space.locate(a)[2] == aqua.AQUA_TARGET_DEVICE
        assert space.locate(b)[2] == aqua.AQUA_TARGET_HOST
        before = space.usage()
        with pytest.raises(aqua.AquaError) as ei:
            space.reclaim()             # the host region has no room for `a`
        assert ei.value.status == aqua.AQUA_ERR_CAPACITY
        assert space.usage() == before and space.locate(a)[2] == aqua.AQUA_TARGET_DEVICE
        assert space.reclaim(0) == 0    # nothing needs to move
        assert space.restore() == 0     # the device region is full
        space.free(a)
        space.free(b)
        assert space.usage() == {"device_free": 4096, "host_free": 8192, "device_tensors": 0,
                                 "host_tensors": 0}
    finally:
        space.close()
        kv.close()


def test_fair_scheduling_images_in_a_swap_space_with_reclaim_and_restore():
    """The small fair-scheduling run with every prompt's image in its own
    swap-space tensor: a third of them fit the device region, the rest fall
    back to host memory.  After a third of the reschedules the device region
    is reclaimed (every tensor moves to host memory), after two thirds it is
    restored, and the swaps go on from wherever the tensors are.  Pool and
    tensors must equal the oracle's replay with images in fixed slots."""
    from paper_2407_21255_amd import cfs
    from paper_2407_21255_amd.cycle import run_slices_in_space
    from tests.gpu_util import apply_pool_mutations_device, oracle_replay
    cfg = wl.CFS_SMALL
    sh = cfg.shape
    tr = cfg.trace()
    log, _ = cfs.run_trace(tr, sh.num_blocks, sh.block_tokens, cfg.batch_tokens,
                           cfg.decode_slots(tr), cfg.k)
    sched = wl.cfs_swap_schedule(sh, cfg.seed, tr, log)
    n = len(sched.slices)
    sizes = [sh.image_bytes(nb) for nb in sched.nblocks]
    total = sum(sizes)
    pool = device_pool(sh, cfg.seed)
    pool_h = host(pool)
    region_h = np.full(sched.region_bytes, wl.GUARD_BYTE, dtype=np.uint8)
    sa, sb, sc = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(sh.as_tuple(), pool)
    space = aqua.SwapSpace(kv, total // 3 // 256 * 256, total + 256 * len(sizes))
    try:
        tensors = {p: space.alloc(sz) for p, sz in enumerate(sizes)}
        u0 = space.usage()
        assert u0["device_tensors"] > 0 and u0["host_tensors"] > 0, u0

        def between(k):
            wl.apply_growth(pool, sched, k)
            apply_pool_mutations_device(sched, k, pool)

        n1, n2 = n // 3, 2 * n // 3
        run_slices_in_space(kv, space, tensors, sched, 0, n1, sa, sb, between)
        assert space.reclaim(stream=sc) > 0
        assert space.usage()["device_tensors"] == 0
        run_slices_in_space(kv, space, tensors, sched, n1, n2 - n1, sa, sb, between)
        assert space.restore(stream=sc) > 0
        u2 = space.usage()
        assert u2["device_tensors"] > 0, u2
        run_slices_in_space(kv, space, tensors, sched, n2, n - n2, sa, sb, between)
        kv.sync()
        st = kv.stats()
        say("cfs in swap space", st, u0, u2)
        assert st["calls_migrate"] == 2
        oracle_replay(sched, pool_h, region_h, 0, n, slot_marks=False)
        assert_bytes_equal(host(pool), pool_h, "pool")
        last = {}
        for sl in sched.slices:
            for p, t in zip(sl.out_prompts, sl.out_tables):
                last[p] = len(t)
        assert last
        for p, m in last.items():
            ptr, _, _ = space.locate(tensors[p])
            nb = sh.image_bytes(m)
            o = sched.slot_offsets[p]
            assert_bytes_equal(_read(ptr, nb), region_h[o:o + nb], f"image of prompt {p}")
    finally:
        space.close()
        kv.close()


def test_partial_reclaim_and_restore_follow_handle_order():
    """reclaim(bytes) moves the oldest device tensors until that much of the
    region is free; restore moves host tensors back, oldest first, skipping
    those that do not fit.  Tensors allocated and freed in between reuse the
    vacated ranges, all without host syncs.  Placements follow that rule,
    and every tensor's bytes and the pool after swap-ins from wherever the
    tensors are equal the oracle's."""
    shape = wl.KVShape(2, 256, 1, 2, 8, wl.BF16)         # 64-byte chunks, 128 B per block
    d = odesc(shape)
    unit = shape.num_layers * shape.chunk_bytes
    pool = device_pool(shape, 23)
    pool_h = host(pool)
    perm = wl.permutation(shape.num_blocks, 23)
    # Image sizes (blocks): 2, 1, 3, 2 KiB fill the 8 KiB device region; the
    # fifth (2 KiB) falls back to host memory.
    sizes = [16, 8, 24, 16, 16]
    tables, k = [], 0
    for n in sizes:
        tables.append(perm[k:k + n])
        k += n
    kv = aqua.KVPool(shape.as_tuple(), pool)
    space = aqua.SwapSpace(kv, 8192, 65536)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    D, H = aqua.AQUA_TARGET_DEVICE, aqua.AQUA_TARGET_HOST
    try:
        hs = [space.alloc(n * unit) for n in sizes]
        assert [space.locate(h)[2] for h in hs] == [D, D, D, D, H]
        for h, t in zip(hs, tables):
            kv.swap_out([t], space.buffer(h), stream=sa)
        assert space.reclaim(2560, stream=sb) > 0        # 2 KiB is not enough: two move
        assert [space.locate(h)[2] for h in hs] == [H, H, D, D, H]
        t6 = perm[k:k + 24]
        k += 24
        h6 = space.alloc(24 * unit)                      # takes the vacated 3 KiB
        assert space.locate(h6)[2] == D
        kv.swap_out([t6], space.buffer(h6), stream=sa)
        assert space.restore(stream=sb) == 0             # nothing fits
        space.free(hs[2])                                # 3 KiB free again
        assert space.restore(stream=sb) > 0              # 2 KiB + 1 KiB fit, 2 KiB does not
        assert [space.locate(h)[2] for h in hs if h != hs[2]] == [D, D, D, H]
        live = [(h, t) for h, t in zip(hs, tables) if h != hs[2]] + [(h6, t6)]
        images = {h: space.locate(h) for h, _ in live}
        fresh = perm[k:]
        ins, j = [], 0
        for h, t in live:
            ins.append((h, fresh[j:j + len(t)]))
            j += len(t)
        for h, t in ins:
            kv.swap_in([t], space.buffer(h), stream=sb)
        kv.sync()
        got = {h: _read(images[h][0], images[h][1]) for h, _ in live}
    finally:
        space.close()
        kv.close()
    want = {}
    for h, t in live:
        want[h] = np.zeros(len(t) * unit, dtype=np.uint8)
        assert oracle.swap_out(d, pool_h, [t], want[h]) == 0
    for h, t in ins:
        assert oracle.swap_in(d, pool_h, [t], want[h]) == 0
    for h, _ in live:
        assert_bytes_equal(got[h], want[h], f"tensor {h}")
    assert_bytes_equal(host(pool), pool_h, "pool")
