"""Host core on the CPU: validation parity with the oracle, and the run plan."""
import numpy as np

import oracle
from tests import core_lib


def _desc(L, N, H, T, D, dt):
    return core_lib.Desc(L, N, H, T, D, dt)


def test_validation_status_matches_oracle_on_random_calls():
    """The library's validation gives the oracle's status for the same call,
    valid or not (same codes, same precedence)."""
    rng = np.random.default_rng(21)
    for case in range(4000):
        L = int(rng.integers(1, 3))
        N = int(rng.integers(1, 9))
        d = (L, N, 1, 2, 8, oracle.F16)
        C = 2 * 1 * 2 * 8 * 2
        S = int(rng.integers(0, 4))
        lens = rng.integers(0, 4, size=S)
        ids = rng.integers(-1, N + 1, size=int(lens.sum())).astype(np.int32)
        if rng.random() < 0.5:
            ids = np.clip(ids, 0, N - 1).astype(np.int32)
        offs = np.zeros(S + 1, dtype=np.uint64)
        offs[1:] = np.cumsum(lens)
        img_offsets = None
        if rng.random() < 0.5:
            img_offsets = (rng.integers(0, 6, size=S) * (L * C) +
                           (8 if rng.random() < 0.05 else 0)).astype(np.uint64)
        buf = np.zeros(int(rng.integers(0, 8)) * L * C + 16, dtype=np.uint8)
        pool = np.zeros(L * N * C, dtype=np.uint8)
        is_in = bool(rng.random() < 0.5)
        od = oracle.desc(*d)
        fn = oracle.swap_in if is_in else oracle.swap_out
        want = fn(od, pool, None, buf, img_offsets, ids=ids, offs=offs,
                  dst_bytes=buf.nbytes - 16) if not is_in else \
            fn(od, pool, None, buf, img_offsets, ids=ids, offs=offs,
               src_bytes=buf.nbytes - 16)
        got = core_lib.validate(_desc(*d), ids, offs, buf.ctypes.data, buf.nbytes - 16,
                                img_offsets, is_in)
        assert got == want, (case, d, ids, offs, img_offsets, is_in)


def test_shape_validation():
    ok = core_lib.validate(_desc(2, 4, 1, 2, 8, oracle.BF16), [], [0], 0, 0)
    assert ok == 0
    for bad in [(0, 4, 1, 2, 8, 2), (2, 0, 1, 2, 8, 2), (2, 4, 0, 2, 8, 2),
                (2, 4, 1, 0, 8, 2), (2, 4, 1, 2, 0, 2), (2, 4, 1, 2, 8, 7),
                (2, 4, 1, 1, 4, 3),                 # chunk of 8 bytes
                (2, 4, 1 << 17, 2, 8, 2),           # absurd head count
                (1 << 31, 1 << 30, 64, 64, 128, 2)]:  # pool beyond 2^62 bytes
        assert core_lib.validate(_desc(*bad), [], [0], 0, 0) == oracle.ERR_INVALID, bad


def test_capacity_arithmetic_cannot_wrap():
    d = _desc(80, 4096, 8, 16, 128, oracle.BF16)
    C = 64 * 1024
    # An image offset near 2^64 must be a capacity error, not a wrapped fit.
    big = np.array([(1 << 64) - 16], dtype=np.uint64)
    assert core_lib.validate(d, [1], [0, 1], 4096, 80 * C, big) == oracle.ERR_CAPACITY
    assert core_lib.validate(d, [1], [0, 1], 4096, 80 * C, [0]) == 0
    assert core_lib.validate(d, [1], [0, 1], 4096, 80 * C - 16, [0]) == oracle.ERR_CAPACITY


def _check_plan(desc_t, tables, img_offsets, unit_bytes):
    L, N, H, T, D, dt = desc_t
    e = 1 if dt == oracle.FP8_E4M3 else 2
    C = 2 * H * T * D * e
    ids = np.asarray([b for t in tables for b in t], dtype=np.int32)
    offs = np.zeros(len(tables) + 1, dtype=np.uint64)
    offs[1:] = np.cumsum([len(t) for t in tables])
    runs = core_lib.plan(_desc(*desc_t), ids, offs, img_offsets, unit_bytes)
    max_run = max(1, unit_bytes // C)
    k = 0
    packed = 0
    for s, t in enumerate(tables):
        n = len(t)
        base = packed if img_offsets is None else int(img_offsets[s])
        packed += L * n * C
        i = 0
        while i < n:
            r = runs[k]
            assert r["block"] == t[i]
            assert r["img_off"] == base + i * C
            assert r["img_lstride"] == n * C
            ln = int(r["nchunks"])
            assert 1 <= ln <= max_run
            assert list(t[i:i + ln]) == list(range(t[i], t[i] + ln))
            # Maximal: the next entry does not extend the run unless capped.
            if i + ln < n and ln < max_run:
                assert t[i + ln] != t[i + ln - 1] + 1
            i += ln
            k += 1
    assert k == len(runs)
    return runs


def test_plan_random_tables_cover_exactly_and_are_maximal():
    rng = np.random.default_rng(22)
    for case in range(500):
        N = 64
        S = int(rng.integers(0, 5))
        tables = []
        for _ in range(S):
            n = int(rng.integers(0, 12))
            if rng.random() < 0.5:
                start = int(rng.integers(0, N - n + 1))
                t = list(range(start, start + n))
                if n > 2 and rng.random() < 0.5:
                    t[n // 2] = int(rng.integers(0, N))
            else:
                t = [int(x) for x in rng.integers(0, N, size=n)]
            tables.append(t)
        dt = oracle.FP8_E4M3 if rng.random() < 0.5 else oracle.BF16
        unit = int(rng.choice([256, 512, 1024, 4096, 1 << 16]))
        io = None
        if rng.random() < 0.5:
            io = np.cumsum([0] + [3 * 64 * 4 * len(t) for t in tables])[:-1]
        _check_plan((3, N, 1, 4, 8, dt), tables, io, unit)


def test_plan_coalesces_contiguous_tables():
    # C = 2*8*16*128*1 = 32 KiB (fp8) and 64 KiB units: runs of two.
    runs = _check_plan((2, 100, 8, 16, 128, oracle.FP8_E4M3), [list(range(10, 20))], None,
                       64 << 10)
    assert len(runs) == 5 and all(runs["nchunks"] == 2)
    # bf16 (64 KiB chunks): one chunk per run whatever the table.
    runs = _check_plan((2, 100, 8, 16, 128, oracle.BF16), [list(range(10, 20))], None,
                       64 << 10)
    assert len(runs) == 10


def test_ex_validation_matches_oracle_on_random_calls():
    """Layer ranges and per-sequence image lengths: same status as the oracle."""
    rng = np.random.default_rng(23)
    for case in range(3000):
        L = int(rng.integers(1, 4))
        N = int(rng.integers(1, 9))
        d = (L, N, 1, 2, 8, oracle.F16)
        C = 64
        S = int(rng.integers(0, 4))
        lens = rng.integers(0, 4, size=S)
        ids = rng.integers(0, N, size=int(lens.sum())).astype(np.int32)
        if rng.random() < 0.2:
            ids = rng.integers(-1, N + 1, size=int(lens.sum())).astype(np.int32)
        offs = np.zeros(S + 1, dtype=np.uint64)
        offs[1:] = np.cumsum(lens)
        img_blocks = None
        if rng.random() < 0.7:
            img_blocks = (lens + rng.integers(-1 if rng.random() < 0.1 else 0, 3, size=S)).clip(0)
        img_offsets = None
        if rng.random() < 0.5:
            img_offsets = (rng.integers(0, 8, size=S) * (L * C)).astype(np.uint64)
        l0, nl = 0, 0
        if rng.random() < 0.6:
            l0 = int(rng.integers(0, L + 1))
            nl = int(rng.integers(0, L + 1))
        buf = np.zeros(int(rng.integers(0, 12)) * L * C + 16, dtype=np.uint8)
        pool = np.zeros(L * N * C, dtype=np.uint8)
        is_in = bool(rng.random() < 0.5)
        od = oracle.desc(*d)
        fn = oracle.swap_in_ex if is_in else oracle.swap_out_ex
        kw = {"src_bytes" if is_in else "dst_bytes": buf.nbytes - 16}
        want = fn(od, pool, None, buf, img_offsets, img_blocks, l0, nl, ids=ids, offs=offs, **kw)
        got = core_lib.validate_ex(_desc(*d), ids, offs, buf.ctypes.data, buf.nbytes - 16,
                                   img_offsets, img_blocks, l0, nl, is_in)
        assert got == want, (case, ids, offs, img_offsets, img_blocks, l0, nl, is_in)


def test_plan_with_longer_images_strides_by_image_length():
    d = _desc(3, 64, 1, 4, 8, oracle.BF16)
    C = 2 * 4 * 8 * 2
    runs = core_lib.plan_ex(d, [5, 9, 10, 11, 40], [0, 2, 5], None, [4, 7], unit_bytes=1 << 20)
    # Sequence 0: image of 4 blocks per layer at 0; sequence 1: 7 blocks at 3*4*C.
    assert list(runs["block"]) == [5, 9, 10, 40]
    assert list(runs["nchunks"]) == [1, 1, 2, 1]
    assert list(runs["img_lstride"]) == [4 * C, 4 * C, 7 * C, 7 * C]
    assert list(runs["img_off"]) == [0, C, 3 * 4 * C, 3 * 4 * C + 2 * C]


def test_migrate_validation_matches_oracle():
    rng = np.random.default_rng(24)
    for case in range(2000):
        src = np.zeros(4096, dtype=np.uint8)
        dst = src if rng.random() < 0.3 else np.zeros(4096, dtype=np.uint8)
        n = int(rng.integers(0, 4))
        g = 16 if rng.random() < 0.9 else 8
        so = rng.integers(0, 300, size=n) * g
        do = rng.integers(0, 300, size=n) * g
        ln = rng.integers(0, 40, size=n) * g
        want = oracle.migrate(src, dst, so, do, ln)
        got = core_lib.validate_migrate(src.ctypes.data, src.nbytes, dst.ctypes.data,
                                        dst.nbytes, so, do, ln)
        assert got == want, (case, so, do, ln, src is dst)


def test_launch_grid_stays_within_one_dispatch():
    """A dispatch counts its work-items in 32 bits: with 1024-lane
    workgroups at most 4 194 303 fit.  A call of 2^22 units (a fragmented
    131072-block table of 32 layers) and anything larger get a capped grid
    that the kernels' grid-stride loop covers."""
    from tests.core_lib import launch_grid
    assert launch_grid(1, 0) == 1
    assert launch_grid(32768, 0) == 32768
    assert launch_grid(32768, 16) == 16
    for units in (1 << 22, (1 << 31) - 1, 1 << 40):
        g = launch_grid(units, 0)
        assert g == 1 << 21 and g * 1024 < 1 << 32
    assert launch_grid(1 << 22, 4_000_000) == 1 << 21
    assert launch_grid(0, 0) == 0


def test_workgroup_is_sized_to_the_chunk():
    """Every lane holds 4 vectors of 16 bytes in flight: a 64 KiB chunk
    takes 1024 lanes, 32 KiB 512, 16 KiB 256; a larger chunk still 1024,
    and smaller ones never go below the minimum asked for (a power of two
    of at least one wave)."""
    from tests.core_lib import swap_threads
    assert swap_threads(64 << 10, 64) == 1024
    assert swap_threads(1 << 20, 64) == 1024
    assert swap_threads(32 << 10, 64) == 512
    assert swap_threads(16 << 10, 64) == 256
    assert swap_threads(4 << 10, 64) == 64
    assert swap_threads(48 << 10, 64) == 1024   # 768 lanes' worth rounds up
    assert swap_threads(32, 64) == 64
    assert swap_threads(16 << 10, 256) == 256
    assert swap_threads(4 << 10, 256) == 256
    assert swap_threads(4 << 10, 200) == 256
    assert swap_threads(32 << 10, 1024) == 1024
    for c in (16, 32, 4096, 12288, 65536, 1 << 30):
        t = swap_threads(c, 64)
        assert t in (64, 128, 256, 512, 1024)


def test_run_order_rule():
    """Chunks of 64 KiB or more: every swap-in sorted by pool block and
    dealt out to the XCDs; a swap-out dealt in table order when it covers at
    least 40 % of the pool or its sequences average at least 32 blocks.
    Smaller chunks: swap-ins that cover 40 % of the pool sorted and dealt;
    everything else keeps table order."""
    from tests.core_lib import SORTED_DEALT, TABLE, TABLE_DEALT, run_order
    K = 1 << 10
    # 64 KiB chunks.
    assert run_order(True, 64 * K, 2048, 4096) == SORTED_DEALT       # 70B scatter: half the pool
    assert run_order(False, 64 * K, 2048, 4096) == TABLE_DEALT       # 70B gather
    assert run_order(True, 64 * K, 1024, 16384, 8) == SORTED_DEALT   # 8B pair: a sixteenth
    assert run_order(False, 64 * K, 1024, 16384, 8) == TABLE_DEALT   # 128 blocks per prompt
    assert run_order(False, 64 * K, 1024, 16384, 64) == TABLE        # 16 blocks per prompt
    assert run_order(False, 64 * K, 2048, 16384, 64) == TABLE_DEALT  # 32 blocks per prompt
    assert run_order(False, 64 * K, 2047, 16384, 64) == TABLE
    assert run_order(True, 64 * K, 1024, 16384, 64) == SORTED_DEALT
    assert run_order(False, 1 << 20, 31, 4096, 1) == TABLE
    assert run_order(False, 1 << 20, 32, 4096, 1) == TABLE_DEALT
    assert run_order(False, 64 * K, 1639, 4096, 1000) == TABLE_DEALT # dense, short prompts
    assert run_order(False, 64 * K, 1638, 4096, 1000) == TABLE
    # Smaller chunks.
    assert run_order(True, 16 * K, 2048, 4096) == SORTED_DEALT       # TP4 scatter
    assert run_order(False, 32 * K, 2048, 4096) == TABLE             # TP2 gather
    assert run_order(True, 32 * K, 4168, 16384, 16) == TABLE         # preemption cycle: a quarter
    assert run_order(True, 32 * K, 1639, 4096) == SORTED_DEALT
    assert run_order(True, 32 * K, 1638, 4096) == TABLE
    # Nothing to order: no blocks, or fewer than two per XCD.
    assert run_order(True, 64 * K, 0, 0) == TABLE
    assert run_order(False, 64 * K, 0, 4096, 0) == TABLE
    assert run_order(True, 64 * K, 15, 4096) == TABLE
    assert run_order(True, 64 * K, 16, 4096) == SORTED_DEALT
    assert run_order(True, 64 * K, 15, 20) == TABLE


def test_sort_by_block_matches_a_stable_sort():
    """The counting sort gives the runs in ascending block order and keeps
    table order among runs that start at the same block (swap-outs may name
    a block twice), on random plans with and without repeats."""
    import numpy as np
    from tests.core_lib import RUN_DESC, sort_by_block
    rng = np.random.default_rng(5)
    for trial in range(200):
        n = int(rng.integers(0, 300))
        N = int(rng.integers(1, 400))
        d = np.zeros(n, dtype=RUN_DESC)
        d["block"] = rng.integers(0, N, n)
        d["img_off"] = np.arange(n) * 4096            # table order, to check stability
        d["nchunks"] = rng.integers(1, 5, n)
        got = sort_by_block(d, N)
        want = d[np.argsort(d["block"], kind="stable")]
        assert got.tobytes() == want.tobytes(), trial
    # Few runs on a large pool take the comparison sort, many the counting
    # sort: both stable.
    for n, N in ((3, 16384), (1023, 16384), (1024, 16384), (5000, 16384), (40, 40)):
        d = np.zeros(n, dtype=RUN_DESC)
        d["block"] = rng.integers(0, N, n)
        d["img_off"] = np.arange(n) * 4096
        want = d[np.argsort(d["block"], kind="stable")]
        assert sort_by_block(d, N).tobytes() == want.tobytes(), (n, N)
    assert len(sort_by_block(np.zeros(0, dtype=RUN_DESC), 7)) == 0


def test_interleave_runs_deals_eighths_to_the_xcds():
    """Sorted runs are dealt out 8 ways: position j holds run j // 8 of the
    (j % 8)-th contiguous eighth, so the units a round-robin dispatch sends
    to one XCD cover one contiguous eighth of the sorted range.  That holds
    for every length: the first n % 8 eighths hold one run more, so the
    last row, which is short, holds one run of each of them.  The result is
    a permutation of the input, and lists shorter than two runs per way
    stay as they are."""
    import numpy as np
    from tests.core_lib import RUN_DESC, interleave_runs, xcd_ways
    W = xcd_ways()
    assert W == 8
    # 2048 sorted runs (one 70B layer): XCD x (= position % 8) gets runs
    # 256x .. 256x + 255, in order.
    d = np.zeros(2048, dtype=RUN_DESC)
    d["block"] = np.arange(2048)
    got = interleave_runs(d, W)["block"]
    for x in range(W):
        assert list(got[x::W]) == list(range(256 * x, 256 * x + 256))
    # A worked case: 19 runs, eighths of 3, 3, 3, 2, 2, 2, 2, 2 (0-2, 3-5,
    # 6-8, 9-10, 11-12, 13-14, 15-16, 17-18).
    d = np.zeros(19, dtype=RUN_DESC)
    d["block"] = np.arange(19)
    assert list(interleave_runs(d, W)["block"]) == [
        0, 3, 6, 9, 11, 13, 15, 17, 1, 4, 7, 10, 12, 14, 16, 18, 2, 5, 8]
    rng = np.random.default_rng(9)
    for n in list(range(0, 40)) + [int(x) for x in rng.integers(40, 5000, 30)]:
        d = np.zeros(n, dtype=RUN_DESC)
        d["block"] = rng.permutation(n)
        d["img_off"] = np.arange(n) * 64
        got = interleave_runs(d, W)
        assert sorted(got.tobytes()[i:i + 32] for i in range(0, 32 * n, 32)) == \
            sorted(d.tobytes()[i:i + 32] for i in range(0, 32 * n, 32)), n
        if n < 2 * W:
            assert got.tobytes() == d.tobytes(), n
        else:
            # Eighths as contiguous index ranges; position j must hold
            # element j // 8 of eighth j % 8.
            q, r = divmod(n, W)
            starts = [s * q + min(s, r) for s in range(W)]
            order = [starts[j % W] + j // W for j in range(n)]
            assert got.tobytes() == d[order].tobytes(), n
            sizes = [q + (s < r) for s in range(W)]
            assert sum(sizes) == n and all(j // W < sizes[j % W] for j in range(n)), n
    d = np.zeros(100, dtype=RUN_DESC)
    d["block"] = np.arange(100)
    assert interleave_runs(d, 1).tobytes() == d.tobytes()


def test_xcd_unit_order_gives_each_xcd_a_contiguous_eighth():
    """On a one-pass launch, workgroup b goes to XCD b % 8 and takes unit
    xcd_unit(b, units): a bijection on the units in which each XCD's
    workgroups, in dispatch order, take consecutive units of one contiguous
    eighth (the first units % 8 eighths one unit longer).  Only calls of
    chunks between 16 and 64 KiB whose runs are not dealt out use it."""
    from tests.core_lib import xcd_unit, xcd_unit_order
    for units in list(range(1, 70)) + [163840, 16384, 4168 * 3, 2 ** 21 - 1, 1000003]:
        got = [xcd_unit(b, units) for b in range(units)]
        assert sorted(got) == list(range(units)), units
        q, r = divmod(units, 8)
        for x in range(8):
            mine = got[x::8]
            start = x * q + min(x, r)
            assert mine == list(range(start, start + len(mine))), (units, x)
            assert len(mine) == q + (1 if x < r else 0)
    # Worked case: 19 units, eighths of 3, 3, 3, 2, 2, 2, 2, 2.
    assert [xcd_unit(b, 19) for b in range(19)] == [
        0, 3, 6, 9, 11, 13, 15, 17, 1, 4, 7, 10, 12, 14, 16, 18, 2, 5, 8]
    K = 1 << 10
    assert xcd_unit_order(32 * K, False) and xcd_unit_order(48 * K, False)
    assert not xcd_unit_order(32 * K, True)   # runs dealt out on the host instead
    assert not xcd_unit_order(16 * K, False) and not xcd_unit_order(64 * K, False)
    assert not xcd_unit_order(48, False) and not xcd_unit_order(1 << 20, False)


def test_launch_size_rule():
    """A call goes out in launches of whole layers of fewer than 2^31 units
    each: one launch for every workload here, several only where one layer
    holds a large share of 2^31 runs."""
    from tests.core_lib import layers_per_launch
    assert layers_per_launch(2048) == (1 << 31) // 2048          # 70B or TP2: all 80 layers
    assert layers_per_launch(4168) == (1 << 31) // 4168          # preemption cycle call
    assert layers_per_launch(131072) == 16384                     # 131072 runs per layer
    assert layers_per_launch((1 << 31) - 1) == 1
    assert layers_per_launch(1 << 31) == 1
    assert layers_per_launch(0) == 1 << 31
