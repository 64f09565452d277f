"""GPU parity: the HIP gather/scatter path against the CPU oracle, byte for
byte, through the C ABI.  Every input comes from the seeded generator; every
expected value from the oracle run on a host copy of the same input."""

import time

import numpy as np
import pytest
import torch

import oracle
from paper_2407_21255_amd import aqua
from paper_2407_21255_amd import workload as wl
from tests.checkers import assert_bytes_equal
from tests.gpu_util import (device_pool, guarded_buffer, host, odesc, say)

pytestmark = pytest.mark.gpu

G = 4096  # guard bytes on each side of an image


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    aqua.load()  # fails loudly when the library is missing
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _roundtrip(shape, seed, out_tables, in_tables, owner, img_offsets=None,
               buf_bytes=None, pinned=False, sentinel=True, stream=None, host_path=None,
               carrier=None, max_workgroups=None):
    """swap_out(out_tables) then swap_in(in_tables) on the GPU and in the
    oracle; compares the image, guards and the whole pool."""
    C = shape.chunk_bytes
    d = odesc(shape)
    pool = device_pool(shape, seed, owner)
    if sentinel:
        P = pool.view(shape.num_layers, shape.num_blocks, C)
        ids = torch.tensor(sorted({b for t in in_tables for b in t}), dtype=torch.long,
                           device="cuda")
        if len(ids):
            P[:, ids] = wl.SENTINEL_BYTE
    pool_h = host(pool)
    nb = sum(len(t) for t in out_tables)
    size = buf_bytes if buf_bytes is not None else shape.image_bytes(nb)
    buf = guarded_buffer(size, G, pinned)
    inner = buf[G:G + size]
    kv = aqua.KVPool(shape.as_tuple(), pool)
    if host_path is not None:
        kv.set_host_path(host_path)
    if max_workgroups is not None:
        kv.set_max_workgroups(aqua.AQUA_TARGET_HOST if pinned else aqua.AQUA_TARGET_DEVICE,
                              max_workgroups)
    if carrier is not None:
        for direction in (0, 1):
            kv.set_link_engine(direction, carrier)
    try:
        t1 = kv.swap_out(out_tables, inner, img_offsets, stream=stream)
        kv.sync(t1)
        img_h = host(buf)
        want = np.full(size + 2 * G, wl.GUARD_BYTE, dtype=np.uint8)
        assert oracle.swap_out(d, pool_h, out_tables, want[G:G + size], img_offsets) == 0
        assert_bytes_equal(img_h, want, f"{shape} image")
        assert_bytes_equal(host(pool), pool_h, "swap-out changed the pool")
        t2 = kv.swap_in(in_tables, inner, img_offsets, stream=stream)
        assert t2 == t1 + 1
        kv.sync(0)
        assert oracle.swap_in(d, pool_h, in_tables, want[G:G + size], img_offsets) == 0
        assert_bytes_equal(host(pool), pool_h, f"{shape} pool after swap-in")
        assert_bytes_equal(host(buf), want, "swap-in changed the image or guards")
        st = kv.stats()
        assert st["calls_out"] == 1 and st["calls_in"] == 1 and st["hip_error"] == 0
        if carrier is not None:
            used = [kv.link_engine(0), kv.link_engine(1)]
            say("link carriers", used)
            if carrier == aqua.AQUA_LINK_AUTO:
                assert all(u >= 0 or u == aqua.AQUA_LINK_RUNTIME for u in used)
            else:
                assert used == [carrier, carrier]
    finally:
        kv.close()
    return pool_h


def test_tiny_config_round_trip():
    """4 layers, 8 KV heads, head_dim 128, block 16, fp16; one 512-token
    prompt on a random block subset, back into a random free subset."""
    case = wl.tiny_case()
    say("tiny round trip", case.shape)
    pool_h = _roundtrip(case.shape, case.seed, case.out_tables, case.in_tables, case.owner)
    s = case.shape
    P = pool_h.reshape(s.num_layers, s.num_blocks, s.chunk_bytes)
    # Round trip identity: the new blocks hold the old blocks' bytes.
    fresh = np.empty(s.pool_bytes, dtype=np.uint8)
    wl.fill_pool(torch.from_numpy(fresh), s, case.seed, case.owner)
    F = fresh.reshape(P.shape)
    assert np.array_equal(P[:, case.in_tables[0]], F[:, case.out_tables[0]])


RAGGED = [
    # (L, N, H, T, D, dtype): 48-byte chunks, 8 KiB chunks, 32 KiB fp8, 64 KiB, and 1 MiB
    # chunks that the plan splits into 16 units of 64 KiB each.
    wl.KVShape(3, 300, 1, 3, 8, wl.FP8_E4M3),
    wl.KVShape(2, 64, 2, 16, 64, wl.BF16),
    wl.KVShape(2, 96, 8, 16, 128, wl.FP8_E4M3),
    wl.KVShape(3, 64, 8, 16, 128, wl.F16),
    wl.KVShape(2, 48, 32, 32, 256, wl.F16),
    # 24 and 40 KiB chunks end inside a workgroup's second and third rows of 1024
    # vectors; 96 KiB chunks split into a 64 KiB unit and a 32 KiB remainder.
    wl.KVShape(3, 80, 3, 16, 128, wl.F16),
    wl.KVShape(2, 64, 5, 16, 128, wl.BF16),
    wl.KVShape(2, 48, 12, 16, 128, wl.BF16),
]


@pytest.mark.parametrize("shape", RAGGED, ids=lambda s: f"C{s.chunk_bytes}")
def test_multi_sequence_ragged_and_coalesced(shape):
    """Several sequences per call: fragmented tables, contiguous runs that
    coalesce (and split at the unit size), an empty table, placed images
    with gaps between them."""
    N = shape.num_blocks
    perm = wl.permutation(N, 41)
    a = perm[:7]                                  # fragmented
    b = list(range(5, 5 + min(40, N // 3)))       # contiguous
    b = [x for x in b if x not in a]
    c = []                                        # empty
    e = [perm[-1]]                                # single block
    out_tables = [a, b, c, e]
    used = set(a) | set(b) | set(e)
    free = [x for x in perm if x not in used]
    in_tables, k = [], 0
    for t in out_tables:
        in_tables.append(free[k:k + len(t)])
        k += len(t)
    sizes = [shape.image_bytes(len(t)) for t in out_tables]
    offs, pos = [], 0
    for sz in sizes:
        pos += 4096 + 48  # gap, keeps 16-byte alignment
        pos = (pos + 15) // 16 * 16
        offs.append(pos)
        pos += sz
    say("ragged", shape, [len(t) for t in out_tables])
    _roundtrip(shape, 7, out_tables, in_tables, None, img_offsets=offs, buf_bytes=pos + 4096)


@pytest.mark.parametrize("unit", [16, 1 << 20])
def test_unit_size_extremes(unit, monkeypatch):
    """One chunk per workgroup, and runs long enough for several unrolled
    iterations plus a tail, give the same bytes."""
    monkeypatch.setenv("AQUA_UNIT_BYTES", str(unit))
    shape = wl.KVShape(2, 1024, 1, 3, 8, wl.FP8_E4M3)  # 48-byte chunks
    out_tables = [list(range(100, 400)), list(range(49, -1, -1))]
    in_tables = [list(range(400, 700)), list(range(700, 750))]
    say("unit", unit)
    _roundtrip(shape, 9, out_tables, in_tables, None)


@pytest.mark.parametrize("cap,pinned,chunk_kib", [(1, False, 8), (7, False, 8), (300, False, 8),
                                                (3, True, 8), (0, False, 32), (7, False, 32),
                                                (1000, False, 32)])
def test_capped_grids_loop_over_every_unit(cap, pinned, chunk_kib):
    """A grid capped below the number of (layer, run) units: each workgroup
    loops over units a grid apart, and every byte still moves once.  With
    32 KiB chunks the unsorted swap-out asks for the XCD unit order: used on
    the uncapped grid (cap 0), set aside on a capped one.
    The swap-ins cover 45 % of the pool, so their runs are sorted and dealt
    out to the XCDs."""
    if chunk_kib == 8:
        shape = wl.KVShape(3, 512, 2, 16, 64, wl.BF16)
    else:
        shape = wl.KVShape(3, 512, 8, 16, 128, wl.FP8_E4M3)
    assert shape.chunk_bytes == chunk_kib << 10
    perm = wl.permutation(shape.num_blocks, 61)
    out_tables = [perm[:150], perm[150:151], perm[151:233]]
    in_tables = [perm[233:383], perm[383:384], perm[384:466]]
    say("cap", cap, "pinned", pinned, "chunk", shape.chunk_bytes)
    _roundtrip(shape, 61, out_tables, in_tables, None, pinned=pinned,
               host_path=aqua.AQUA_HOST_ZERO_COPY if pinned else None,
               max_workgroups=cap or None)


def test_more_units_than_one_dispatch_can_count():
    """40 layers of a fragmented 131072-block table on a 262144-block pool of
    32-byte chunks: 5.2 million (layer, run) units, more workgroups than one
    dispatch can count (its 32-bit work-item count allows 4 194 303 of 1024
    lanes).  The grid is capped and each workgroup loops over units a grid
    apart; every byte still matches the oracle."""
    shape = wl.KVShape(40, 262144, 1, 1, 8, wl.BF16)          # 32-byte chunks
    perm = wl.permutation(shape.num_blocks, 67)
    out_tables = [perm[:131072]]
    in_tables = [perm[131072:]]
    say("units", shape.num_layers * len(out_tables[0]))
    _roundtrip(shape, 67, out_tables, in_tables, None)


def test_layer_ranges_of_32k_chunks_in_xcd_unit_order():
    """32 KiB chunks to an HBM buffer, 1.4 GiB each way: the swap-outs keep
    table order and run in the kernels' XCD unit order over the units of
    their layer range; the swap-ins cover 49 % of the pool, so their runs
    are sorted and dealt out to the XCDs.  Whole calls and layer ranges
    (1-7, 4-5, 9) match the oracle byte for byte, guard bytes included, and
    each call is one launch."""
    shape = wl.KVShape(10, 9216, 8, 16, 128, wl.FP8_E4M3)    # 32 KiB chunks, 2.8 GiB
    C = shape.chunk_bytes
    assert C == 32 << 10
    d = odesc(shape)
    perm = wl.permutation(shape.num_blocks, 71)
    out_t = [perm[:2500], perm[2500:4500]]
    in_t = [perm[4600:7100], perm[7100:9100]]
    n = 4500
    pool = device_pool(shape, 71)
    pool_h = host(pool)
    size = shape.image_bytes(n)
    buf = guarded_buffer(size, G)
    inner = buf[G:G + size]
    want = np.full(size + 2 * G, wl.GUARD_BYTE, dtype=np.uint8)
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        for l0, nl in [(0, 0), (1, 7), (4, 2), (9, 1)]:
            layers = None if nl == 0 else (l0, nl)
            say("32 KiB layer ranges, layers", layers)
            before = kv.stats()["launches"]
            kv.swap_out(out_t, inner, layers=layers)
            mid = kv.stats()["launches"]
            kv.swap_in(in_t, inner, layers=layers)
            kv.sync()
            after = kv.stats()["launches"]
            assert (mid - before, after - mid) == (1, 1)
            assert oracle.swap_out_ex(d, pool_h, out_t, want[G:G + size], None, None,
                                      l0, nl) == 0
            assert oracle.swap_in_ex(d, pool_h, in_t, want[G:G + size], None, None,
                                     l0, nl) == 0
            assert_bytes_equal(host(buf), want, f"image after layers {layers}")
            assert_bytes_equal(host(pool), pool_h, f"pool after layers {layers}")
    finally:
        kv.close()
        del pool, buf
        torch.cuda.empty_cache()


def test_pinned_host_zero_copy_round_trip():
    """The offload image in pinned host memory, written and read zero-copy."""
    case = wl.tiny_case(seed=11)
    say("host target zero-copy tiny")
    _roundtrip(case.shape, case.seed, case.out_tables, case.in_tables, case.owner,
               pinned=True, host_path=aqua.AQUA_HOST_ZERO_COPY)


def test_pinned_host_staged_round_trip():
    """The staged host path: gather into HBM slots, runtime copies over the
    link; same bytes as the oracle."""
    case = wl.tiny_case(seed=12)
    say("host target staged tiny")
    _roundtrip(case.shape, case.seed, case.out_tables, case.in_tables, case.owner,
               pinned=True, host_path=aqua.AQUA_HOST_STAGED)


@pytest.mark.parametrize("shape", RAGGED[:2], ids=lambda s: f"C{s.chunk_bytes}")
def test_pinned_host_staged_placed_images(shape):
    """Placed images with gaps in a pinned buffer on the staged path: the
    gaps and guards must stay untouched."""
    N = shape.num_blocks
    perm = wl.permutation(N, 43)
    out_tables = [perm[:5], perm[5:6], [], perm[6:20]]
    in_tables = [perm[20:25], perm[25:26], [], perm[26:40]]
    offs, pos = [], 0
    for t in out_tables:
        pos = (pos + 4096 + 48 + 15) // 16 * 16
        offs.append(pos)
        pos += shape.image_bytes(len(t))
    say("staged placed", shape)
    _roundtrip(shape, 8, out_tables, in_tables, None, img_offsets=offs, buf_bytes=pos + 4096,
               pinned=True, host_path=aqua.AQUA_HOST_STAGED)


@pytest.mark.parametrize("carrier", [aqua.AQUA_LINK_AUTO, aqua.AQUA_LINK_RUNTIME, 3],
                         ids=["auto", "runtime", "engine3"])
def test_staged_link_carriers_cycle_slots(carrier, monkeypatch):
    """Staged swaps through 1 MiB slots, so that every call refills both
    slots several times (one layer per slot fill), with the link copies on
    the automatic choice, on the runtime's copies and on engine 3."""
    monkeypatch.setenv("AQUA_STAGE_SLOT_BYTES", str(1 << 20))
    shape = wl.KVShape(8, 1024, 4, 16, 64, wl.BF16)       # 16 KiB chunks
    perm = wl.permutation(shape.num_blocks, 77)
    out_tables = [perm[0:100], perm[100:130], perm[130:300]]
    in_tables = [perm[300:400], perm[400:430], perm[430:600]]
    say("staged slot cycling", carrier)
    _roundtrip(shape, 21, out_tables, in_tables, None, pinned=True,
               host_path=aqua.AQUA_HOST_STAGED, carrier=carrier)


@pytest.mark.parametrize("carrier", [aqua.AQUA_LINK_AUTO, aqua.AQUA_LINK_RUNTIME],
                         ids=["auto", "runtime"])
def test_staged_calls_back_to_back_without_host_sync(carrier, monkeypatch):
    """Six staged calls with no host sync between them: out, in, out, in on
    one stream through two pinned images, then out and in on a second
    stream.  Each call cycles 1 MiB slots several times, so a call's first
    link job is queued while the previous call's last job may still be in
    flight.  The pool and all three images must equal the oracle's replay."""
    monkeypatch.setenv("AQUA_STAGE_SLOT_BYTES", str(1 << 20))
    shape = wl.KVShape(8, 1024, 4, 16, 64, wl.BF16)       # 16 KiB chunks
    d = odesc(shape)
    perm = wl.permutation(shape.num_blocks, 91)
    ta = [perm[0:100], perm[100:130], perm[130:300]]
    tb = [perm[300:400], perm[400:430], perm[430:600]]
    tc = [perm[600:700], perm[700:730], perm[730:900]]
    owner = {b: (p, i) for p, t in enumerate(ta) for i, b in enumerate(t)}
    pool = device_pool(shape, 31, owner)
    pool_h = host(pool)
    size = shape.image_bytes(300)
    imgs = [guarded_buffer(size, G, True) for _ in range(3)]
    want = [np.full(size + 2 * G, wl.GUARD_BYTE, dtype=np.uint8) for _ in range(3)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    kv.set_host_path(aqua.AQUA_HOST_STAGED)
    for direction in (0, 1):
        kv.set_link_engine(direction, carrier)
    calls = [("out", ta, 0, s1), ("in", tb, 0, s1), ("out", tb, 1, s1), ("in", ta, 1, s1),
             ("out", ta, 2, s2), ("in", tc, 2, s2)]
    say("staged back to back", carrier)
    try:
        for kind, t, k, st in calls:
            inner = imgs[k][G:G + size]
            (kv.swap_out if kind == "out" else kv.swap_in)(t, inner, stream=st)
        kv.sync()
        for kind, t, k, _ in calls:
            fn = oracle.swap_out if kind == "out" else oracle.swap_in
            assert fn(d, pool_h, t, want[k][G:G + size]) == 0
        assert_bytes_equal(host(pool), pool_h, "pool after six staged calls")
        for k in range(3):
            assert_bytes_equal(host(imgs[k]), want[k], f"image {k}")
        stt = kv.stats()
        say("link carriers", [kv.link_engine(0), kv.link_engine(1)], stt["waits_inserted"])
        assert stt["hip_error"] == 0 and stt["calls_out"] == 3 and stt["calls_in"] == 3
    finally:
        kv.close()


def _staged_case(seed):
    shape = wl.KVShape(8, 1024, 4, 16, 64, wl.BF16)       # 16 KiB chunks
    perm = wl.permutation(shape.num_blocks, seed)
    ta = [perm[0:100], perm[100:130], perm[130:300]]
    tb = [perm[300:400], perm[400:430], perm[430:600]]
    owner = {b: (p, i) for p, t in enumerate(ta) for i, b in enumerate(t)}
    return shape, ta, tb, owner


def test_staged_pool_closed_with_calls_in_flight(monkeypatch):
    """Closing a pool right after staged calls (no sync) waits for their
    link copies and stops the engine threads; the bytes are complete."""
    monkeypatch.setenv("AQUA_STAGE_SLOT_BYTES", str(1 << 20))
    shape, ta, tb, owner = _staged_case(97)
    d = odesc(shape)
    pool = device_pool(shape, 33, owner)
    pool_h = host(pool)
    size = shape.image_bytes(300)
    img = guarded_buffer(size, G, True)
    want = np.full(size + 2 * G, wl.GUARD_BYTE, dtype=np.uint8)
    s1 = torch.cuda.Stream()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    kv.set_host_path(aqua.AQUA_HOST_STAGED)
    kv.swap_out(ta, img[G:G + size], stream=s1)
    kv.swap_in(tb, img[G:G + size], stream=s1)
    kv.close()
    torch.cuda.synchronize()
    assert oracle.swap_out(d, pool_h, ta, want[G:G + size]) == 0
    assert oracle.swap_in(d, pool_h, tb, want[G:G + size]) == 0
    assert_bytes_equal(host(img), want, "image")
    assert_bytes_equal(host(pool), pool_h, "pool")


def test_link_carrier_switched_between_calls(monkeypatch):
    """The carrier changes between staged calls (automatic engine, engine 3,
    the runtime's copies); each switch waits for outstanding calls, and
    every call's bytes equal the oracle's."""
    monkeypatch.setenv("AQUA_STAGE_SLOT_BYTES", str(1 << 20))
    shape, ta, tb, owner = _staged_case(98)
    d = odesc(shape)
    pool = device_pool(shape, 34, owner)
    pool_h = host(pool)
    size = shape.image_bytes(300)
    imgs = [guarded_buffer(size, G, True) for _ in range(3)]
    want = [np.full(size + 2 * G, wl.GUARD_BYTE, dtype=np.uint8) for _ in range(3)]
    s1 = torch.cuda.Stream()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    kv.set_host_path(aqua.AQUA_HOST_STAGED)
    steps = [(aqua.AQUA_LINK_AUTO, ta, tb), (3, tb, ta), (aqua.AQUA_LINK_RUNTIME, ta, tb)]
    try:
        used = []
        for k, (carrier, out_t, in_t) in enumerate(steps):
            for direction in (0, 1):
                kv.set_link_engine(direction, carrier)
            kv.swap_out(out_t, imgs[k][G:G + size], stream=s1)
            kv.swap_in(in_t, imgs[k][G:G + size], stream=s1)
            used.append([kv.link_engine(0), kv.link_engine(1)])
        kv.sync()
        say("carriers used", used)
        assert used[1] == [3, 3] and used[2] == [aqua.AQUA_LINK_RUNTIME] * 2
        for k, (_, out_t, in_t) in enumerate(steps):
            assert oracle.swap_out(d, pool_h, out_t, want[k][G:G + size]) == 0
            assert oracle.swap_in(d, pool_h, in_t, want[k][G:G + size]) == 0
            assert_bytes_equal(host(imgs[k]), want[k], f"image {k}")
        assert_bytes_equal(host(pool), pool_h, "pool")
    finally:
        kv.close()


def test_two_pools_share_the_copy_engines(monkeypatch):
    """Two pools stage to pinned host memory at the same time, each on its
    own stream and both on the automatic engines: each pool's threads queue
    on the same engines, and each pool's bytes equal the oracle's."""
    monkeypatch.setenv("AQUA_STAGE_SLOT_BYTES", str(1 << 20))
    runs = []
    for seed in (61, 62):
        shape, ta, tb, owner = _staged_case(seed)
        pool = device_pool(shape, seed, owner)
        size = shape.image_bytes(300)
        runs.append(dict(shape=shape, ta=ta, tb=tb, pool=pool, pool_h=host(pool), size=size,
                         img=guarded_buffer(size, G, True), stream=torch.cuda.Stream(),
                         kv=aqua.KVPool(shape.as_tuple(), pool)))
    try:
        for r in runs:
            r["kv"].set_host_path(aqua.AQUA_HOST_STAGED)
        for kind in ("out", "in"):
            for r in runs:
                inner = r["img"][G:G + r["size"]]
                if kind == "out":
                    r["kv"].swap_out(r["ta"], inner, stream=r["stream"])
                else:
                    r["kv"].swap_in(r["tb"], inner, stream=r["stream"])
        for r in runs:
            r["kv"].sync()
        say("two pools", [[r["kv"].link_engine(0), r["kv"].link_engine(1)] for r in runs])
        for k, r in enumerate(runs):
            d = odesc(r["shape"])
            want = np.full(r["size"] + 2 * G, wl.GUARD_BYTE, dtype=np.uint8)
            assert oracle.swap_out(d, r["pool_h"], r["ta"], want[G:G + r["size"]]) == 0
            assert oracle.swap_in(d, r["pool_h"], r["tb"], want[G:G + r["size"]]) == 0
            assert_bytes_equal(host(r["img"]), want, f"pool {k} image")
            assert_bytes_equal(host(r["pool"]), r["pool_h"], f"pool {k}")
    finally:
        for r in runs:
            r["kv"].close()


@pytest.mark.parametrize("kind,fail_at", [("out", 3), ("in", 0), ("in", 3), ("migrate", 0)])
def test_failed_release_leaves_the_shared_engine_usable(monkeypatch, kind, fail_at):
    """A call that fails after queueing a job on a copy engine but before
    enqueueing the kernel that releases it (forced from the host with
    AQUA_FAIL_RELEASE_AT; every kernel still runs to its end) returns
    AQUA_ERR_HIP once its own work has ended, and the job still drains: a
    second pool on the same engine then moves its bytes as the oracle does,
    and the failed pool refuses further calls and closes promptly."""
    monkeypatch.setenv("AQUA_STAGE_SLOT_BYTES", str(1 << 20))
    engine = 3
    shape, ta, tb, owner = _staged_case(71)
    size = shape.image_bytes(300)
    pool_a = device_pool(shape, 71, owner)
    monkeypatch.setenv("AQUA_FAIL_RELEASE_AT", str(fail_at))
    kva = aqua.KVPool(shape.as_tuple(), pool_a)
    monkeypatch.delenv("AQUA_FAIL_RELEASE_AT")
    pool_b = device_pool(shape, 72, owner)
    pool_bh = host(pool_b)
    kvb = aqua.KVPool(shape.as_tuple(), pool_b)
    img_a = torch.zeros(size, dtype=torch.uint8, pin_memory=True)
    img_b = guarded_buffer(size, G, True)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    closed_a = False
    try:
        for kv in (kva, kvb):
            kv.set_host_path(aqua.AQUA_HOST_STAGED)
            kv.set_link_engine(0, engine)
            kv.set_link_engine(1, engine)
        say("forced release failure", kind, fail_at, "engine", engine)
        with pytest.raises(aqua.AquaError) as ei:
            if kind == "out":
                kva.swap_out(ta, img_a, stream=sa)
            elif kind == "in":
                kva.swap_in(tb, img_a, stream=sa)
            else:
                region = torch.zeros(size, dtype=torch.uint8, device="cuda")
                kva.migrate(region, img_a, [0], [0], [size], stream=sa)
        assert ei.value.status == aqua.AQUA_ERR_HIP
        assert kva.stats()["hip_error"] != 0
        with pytest.raises(aqua.AquaError) as ei:
            kva.swap_out(ta, img_a, stream=sa)
        assert ei.value.status == aqua.AQUA_ERR_STATE

        # The second pool queues behind the failed call's jobs on the engine.
        t0 = time.perf_counter()
        inner = img_b[G:G + size]
        kvb.swap_out(ta, inner, stream=sb)
        kvb.swap_in(tb, inner, stream=sb)
        kvb.sync()
        say("second pool done in", round(time.perf_counter() - t0, 3), "s")
        assert [kvb.link_engine(0), kvb.link_engine(1)] == [engine, engine]
        d = odesc(shape)
        want = np.full(size + 2 * G, wl.GUARD_BYTE, dtype=np.uint8)
        assert oracle.swap_out(d, pool_bh, ta, want[G:G + size]) == 0
        assert oracle.swap_in(d, pool_bh, tb, want[G:G + size]) == 0
        assert_bytes_equal(host(img_b), want, "second pool image")
        assert_bytes_equal(host(pool_b), pool_bh, "second pool")

        t0 = time.perf_counter()
        closed_a = True
        with pytest.raises(aqua.AquaError) as ei:
            kva.close()
        assert ei.value.status == aqua.AQUA_ERR_HIP
        assert time.perf_counter() - t0 < 10.0
    finally:
        if not closed_a:
            try:
                kva.close()
            except aqua.AquaError:
                pass
        kvb.close()


def test_link_engine_setter_rejects_bad_arguments():
    shape = wl.KVShape(2, 64, 1, 2, 8, wl.BF16)
    pool = device_pool(shape, 3)
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        assert kv.link_engine(0) == aqua.AQUA_LINK_AUTO      # nothing staged yet
        for direction, engine in [(2, 0), (-1, 0), (0, 16), (1, -3)]:
            with pytest.raises(aqua.AquaError) as ei:
                kv.set_link_engine(direction, engine)
            assert ei.value.status == aqua.AQUA_ERR_INVALID
        kv.set_link_engine(1, aqua.AQUA_LINK_RUNTIME)
        assert kv.link_engine(1) == aqua.AQUA_LINK_AUTO      # chosen on the next staged call
    finally:
        kv.close()


def test_errors_match_oracle_and_leave_no_trace():
    shape = wl.KVShape(2, 32, 1, 2, 8, wl.BF16)
    C = shape.chunk_bytes
    d = odesc(shape)
    pool = device_pool(shape, 3)
    pool_h = host(pool)
    buf = torch.zeros(shape.image_bytes(4), dtype=torch.uint8, device="cuda")
    hbuf = np.zeros(buf.numel(), dtype=np.uint8)
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        cases = [
            ("out", [[0, -1]], None), ("in", [[0, 32]], None),
            ("in", [[1, 2], [2]], None), ("out", [[1], [2]], [0, C]),
            ("out", [[1, 2, 3, 4, 5]], None), ("in", [[1]], [buf.numel() - C]),
            ("out", [[1]], [8]), ("in", [[32, 32]], [8]), ("in", [[32, 1, 1]], None),
            ("in", [[1, 1, 2, 3, 4]], None),
        ]
        for kind, tables, io in cases:
            fn = kv.swap_out if kind == "out" else kv.swap_in
            ofn = oracle.swap_out if kind == "out" else oracle.swap_in
            want = ofn(d, pool_h.copy(), tables, hbuf.copy(), io)
            assert want != 0
            with pytest.raises(aqua.AquaError) as ei:
                fn(tables, buf, io)
            assert ei.value.status == want, (kind, tables, io)
        # Target / pointer-class mismatches.
        for target, b in [(aqua.AQUA_TARGET_HOST, buf),
                          (aqua.AQUA_TARGET_DEVICE, torch.zeros(buf.numel(), dtype=torch.uint8,
                                                                pin_memory=True)),
                          (aqua.AQUA_TARGET_HOST, torch.zeros(buf.numel(), dtype=torch.uint8)),
                          (7, buf)]:
            with pytest.raises(aqua.AquaError) as ei:
                kv.swap_out([[1]], b, target=target)
            assert ei.value.status == aqua.AQUA_ERR_INVALID
        # A buffer size beyond its allocation is refused, not written.
        st, _ = aqua.aqua_swap_out(kv.handle, 1, np.array([1], np.int32).ctypes.data,
                                   np.array([0, 1], np.uint64).ctypes.data, buf.data_ptr(),
                                   1 << 40, None, 0, None)
        assert st == aqua.AQUA_ERR_INVALID
        torch.cuda.synchronize()
        assert_bytes_equal(host(pool), pool_h, "pool after failing calls")
        assert not host(buf).any()
        # No ticket was spent on the failures.
        t = kv.swap_out([[1]], buf)
        assert t == 1
        kv.sync()
        # Bad tickets.
        assert aqua.aqua_sync(kv.handle, 99) == aqua.AQUA_ERR_INVALID
        assert aqua.aqua_query(kv.handle, 0) == aqua.AQUA_ERR_INVALID
    finally:
        kv.close()
    # Pool creation checks.
    with pytest.raises(aqua.AquaError) as ei:
        aqua.KVPool(shape.as_tuple(), pool[:shape.pool_bytes - 16])
    assert ei.value.status == aqua.AQUA_ERR_CAPACITY
    with pytest.raises(aqua.AquaError) as ei:
        aqua.KVPool(shape.as_tuple(), pool[8:])
    assert ei.value.status == aqua.AQUA_ERR_INVALID
    with pytest.raises(aqua.AquaError) as ei:
        aqua.KVPool(shape.as_tuple(), torch.zeros(shape.pool_bytes, dtype=torch.uint8))
    assert ei.value.status == aqua.AQUA_ERR_INVALID


def test_empty_calls_issue_tickets():
    shape = wl.KVShape(2, 8, 1, 2, 8, wl.BF16)
    pool = device_pool(shape, 4)
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        t1 = kv.swap_out([], pool[:0])
        t2 = kv.swap_in([[], []], pool[:0])
        assert (t1, t2) == (1, 2)
        kv.sync(t2)
        assert kv.query(t1) and kv.query(t2)
    finally:
        kv.close()


def test_cross_stream_reuse_is_ordered():
    """A swap-in on stream B that reuses the blocks a swap-out on stream A
    reads must wait for it.  Stream A is held back by real work queued
    ahead of the swap-out, so without the library's wait B would overwrite
    the blocks first.  The result must equal the sequential oracle."""
    shape = wl.KVShape(8, 2048, 8, 16, 128, wl.BF16)
    C = shape.chunk_bytes
    d = odesc(shape)
    pool = device_pool(shape, 12)
    pool_h = host(pool)
    X = wl.permutation(shape.num_blocks, 5)[:256]
    other_img = torch.empty(shape.image_bytes(256), dtype=torch.uint8, device="cuda")
    wl.fill_chunks(other_img.view(-1, C), torch.arange(8 * 256, dtype=torch.int64) * 7919 + 3,
                   C, shape.dtype)
    other_h = host(other_img)
    img = torch.zeros(shape.image_bytes(256), dtype=torch.uint8, device="cuda")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    a = torch.randn(4096, 4096, device="cuda", dtype=torch.bfloat16)
    torch.cuda.synchronize()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        with torch.cuda.stream(sa):
            for _ in range(200):         # milliseconds of work ahead of the swap-out
                a = (a @ a).clamp_(-1, 1)
        kv.swap_out([X], img, stream=sa)
        kv.swap_in([X], other_img, stream=sb)
        st = kv.stats()
        kv.sync(0)
        assert st["waits_inserted"] == 1
        want_img = np.zeros(img.numel(), dtype=np.uint8)
        assert oracle.swap_out(d, pool_h, [X], want_img) == 0
        assert oracle.swap_in(d, pool_h, [X], other_h) == 0
        assert_bytes_equal(host(img), want_img, "image of the delayed swap-out")
        assert_bytes_equal(host(pool), pool_h, "pool after the reusing swap-in")
    finally:
        kv.close()


def test_stream_wait_orders_caller_work():
    shape = wl.KVShape(4, 256, 8, 16, 128, wl.F16)
    pool = device_pool(shape, 13)
    pool_h = host(pool)
    img = torch.zeros(shape.image_bytes(64), dtype=torch.uint8, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        bt = list(range(0, 128, 2))
        t = kv.swap_out([bt], img, stream=s1)
        kv.stream_wait(t, s2)
        with torch.cuda.stream(s2):
            snap = img.clone()
        s2.synchronize()
        want = np.zeros(img.numel(), dtype=np.uint8)
        assert oracle.swap_out(odesc(shape), pool_h, [bt], want) == 0
        assert_bytes_equal(host(snap), want, "copy made after aqua_stream_wait")
        assert kv.query(t)
    finally:
        kv.close()


def test_binding_keeps_call_buffers_alive_until_complete():
    """The binding holds the tensors a call names until the library reports
    the call complete, so that a caller may drop a temporary buffer right
    after the call; the hold ends with the call."""
    import gc
    import weakref

    shape = wl.KVShape(2, 64, 2, 16, 64, wl.BF16)
    pool = device_pool(shape, 5)
    kv = aqua.KVPool(shape.as_tuple(), pool)
    s = torch.cuda.Stream()
    try:
        with torch.cuda.stream(s):
            torch.cuda._sleep(200_000_000)            # a bounded spin: the call stays pending
        buf = torch.empty(shape.image_bytes(8), dtype=torch.uint8, device="cuda")
        ref = weakref.ref(buf)
        t = kv.swap_out([list(range(8))], buf, stream=s)
        assert not kv.query(t)
        del buf
        gc.collect()
        assert ref() is not None
        kv.sync(t)
        gc.collect()
        assert ref() is None
    finally:
        kv.close()


def test_host_gated_stream_forces_each_hazard_order():
    """Forced interleavings from the host.  Stream A is held by a wait on a
    host flag ahead of a swap-out, so that swap-out stays pending until the
    host opens the flag, after every later call has been issued.  Each later
    call on another stream that conflicts with it gets a device-side wait
    (counted by the library, none elided since A cannot have completed): a
    swap-in reading its image (read after write), a swap-in writing the
    blocks it reads (write after read), a swap-out writing the same image
    bytes again (write after write, and after the first swap-in's read).  A
    call that touches none of them gets no wait.  Once the host opens the
    gate, pool and images equal the oracle run in issue order.  (Whether an
    unrelated stream progresses meanwhile is the runtime's business: streams
    share a few hardware queues.)"""
    from tests.gpu_util import HostGate

    shape = wl.KVShape(4, 512, 8, 16, 128, wl.BF16)
    C = shape.chunk_bytes
    d = odesc(shape)
    pool = device_pool(shape, 19)
    pool_h = host(pool)
    perm = wl.permutation(shape.num_blocks, 17)
    X, Y, W, Z = perm[:32], perm[32:64], perm[64:96], perm[96:128]
    img = torch.zeros(shape.image_bytes(32), dtype=torch.uint8, device="cuda")
    img_e = torch.zeros_like(img)
    other = torch.empty(shape.image_bytes(16), dtype=torch.uint8, device="cuda")
    wl.fill_chunks(other.view(-1, C), torch.arange(4 * 16, dtype=torch.int64) * 104729 + 11,
                   C, shape.dtype)
    other_h = host(other)
    streams = [torch.cuda.Stream() for _ in range(5)]
    torch.cuda.synchronize()
    kv = aqua.KVPool(shape.as_tuple(), pool)
    gate = HostGate()
    try:
        gate.hold(streams[0])
        calls = [("A", lambda s: kv.swap_out([X], img, stream=s)),
                 ("B", lambda s: kv.swap_in([Y], img, stream=s)),           # reads A's image
                 ("C", lambda s: kv.swap_in([X[:16]], other, stream=s)),    # writes what A reads
                 ("D", lambda s: kv.swap_out([W], img, stream=s)),          # rewrites A's image
                 ("E", lambda s: kv.swap_out([Z], img_e, stream=s))]        # independent
        waits, elided, tickets = {}, {}, {}
        for (name, call), s in zip(calls, streams):
            before = kv.stats()
            tickets[name] = call(s)
            after = kv.stats()
            waits[name] = after["waits_inserted"] - before["waits_inserted"]
            elided[name] = after["waits_elided"] - before["waits_elided"]
        pending_a = not kv.query(tickets["A"])
        say("waits per call while the gate is shut:", waits, "elided:", elided)
        assert pending_a
        assert waits["A"] == 0 and waits["E"] == 0 and elided["E"] == 0
        assert waits["B"] == 1 and waits["C"] == 1 and waits["D"] >= 1
        assert sum(elided.values()) == 0
        gate.open()
        kv.sync()
    finally:
        gate.close()
        kv.close()
    want_img = np.zeros(img.numel(), dtype=np.uint8)
    want_e = np.zeros(img.numel(), dtype=np.uint8)
    assert oracle.swap_out(d, pool_h, [X], want_img) == 0
    assert oracle.swap_in(d, pool_h, [Y], want_img) == 0
    assert oracle.swap_in(d, pool_h, [X[:16]], other_h) == 0
    assert oracle.swap_out(d, pool_h, [W], want_img) == 0
    assert oracle.swap_out(d, pool_h, [Z], want_e) == 0
    assert_bytes_equal(host(img), want_img, "image rewritten last")
    assert_bytes_equal(host(img_e), want_e, "independent image")
    assert_bytes_equal(host(pool), pool_h, "pool")


@pytest.mark.parametrize("where", ["hbm", "staged"])
def test_descriptor_ring_wraps_and_grows(monkeypatch, where):
    """A 4 KiB descriptor ring (128 runs): calls of 100 runs wrap it and wait
    for the calls that used the space last, a call of 1000 runs makes it
    grow, and later calls use the grown ring.  No host sync between calls;
    every image and the pool equal the oracle run in issue order."""
    monkeypatch.setenv("AQUA_RING_BYTES", "4096")
    monkeypatch.setenv("AQUA_STAGE_SLOT_BYTES", str(256 << 10))
    shape = wl.KVShape(2, 4096, 1, 4, 16, wl.BF16)            # 256-byte chunks
    d = odesc(shape)
    pool = device_pool(shape, 31)
    pool_h = host(pool)
    perm = wl.permutation(shape.num_blocks, 31)
    sizes = [100, 100, 100, 1000, 100, 100]
    tables, k = [], 0
    for n in sizes:
        tables.append(perm[k:k + n])
        k += n
    fresh = perm[k:]
    pinned = where == "staged"
    imgs = [torch.zeros(shape.image_bytes(n), dtype=torch.uint8,
                        **({"pin_memory": True} if pinned else {"device": "cuda"}))
            for n in sizes]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    kv = aqua.KVPool(shape.as_tuple(), pool)
    try:
        kv.set_host_path(aqua.AQUA_HOST_STAGED)
        ins, j = [], 0
        for i, (t, img) in enumerate(zip(tables, imgs)):
            kv.swap_out([t], img, stream=streams[i % 2])
            dst = fresh[j:j + len(t)]
            j += len(t)
            kv.swap_in([dst], img, stream=streams[(i + 1) % 2])
            ins.append(dst)
        st = kv.stats()
        kv.sync()
        say("ring", where, "waits inserted", st["waits_inserted"],
            "host wait ms", round(st["wait_ns"] / 1e6, 3), "descriptors", st["descriptors"])
        # Random tables: almost every block is a run of its own.
        assert 1.9 * sum(sizes) <= st["descriptors"] <= 2 * sum(sizes)
    finally:
        kv.close()
    for t, dst, img in zip(tables, ins, imgs):
        want = np.zeros(img.numel(), dtype=np.uint8)
        assert oracle.swap_out(d, pool_h, [t], want) == 0
        assert_bytes_equal(host(img), want, "image")
        assert oracle.swap_in(d, pool_h, [dst], want) == 0
    assert_bytes_equal(host(pool), pool_h, "pool")
