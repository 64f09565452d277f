"""The library's fair batch partitioner (``aqua_cfs_partition``, C ABI) and
the rescheduler built on it, against the oracle, on the CPU: the partition
is host code, so this is its parity test proper (bit-exact: it is integer
work).  Also checks the block-level swap schedules derived from a run."""
import ctypes

import numpy as np
import pytest

from oracle import cfs as ocfs
from paper_2407_21255_amd import aqua
from paper_2407_21255_amd import cfs
from paper_2407_21255_amd import workload as wl


def _c_partition(reqs, b, d, cap, T, reserved=0):
    req = np.ascontiguousarray(np.asarray(reqs, dtype=np.uint32).reshape(-1, 4))
    n = len(req)
    idx = np.full(max(n, 1), 0xFFFFFFFF, dtype=np.uint32)
    tok = np.full(max(n, 1), 0xFFFFFFFF, dtype=np.uint32)
    prm = aqua.aqua_cfs_params(b, d, T, reserved, cap)
    st, size, taken = aqua.aqua_cfs_partition(req, prm, idx, tok)
    return st, [[int(i), int(x)] for i, x in zip(idx[:size], tok[:size])], taken, idx, tok


def _random_reqs(rng, n, T, big=False):
    out = []
    hi = (1 << 32) - 1 if big else 500
    for _ in range(n):
        P = int(rng.integers(1, hi, endpoint=True))
        kind = rng.random()
        if kind < 0.45:
            c, g = P, int(rng.integers(0, (hi - P) + 1))
        elif kind < 0.9:
            c, g = int(rng.integers(0, P)), 0
        else:                                   # invalid now and then
            c, g = int(rng.integers(0, P + 2)), int(rng.integers(0, 3))
            c = min(c, hi)
        held = int(rng.integers(0, -(-(c + g) // T) + 2)) if rng.random() < 0.5 else 0
        out.append((P, c, g, min(held, hi)))
    return out


@pytest.mark.parametrize("big", [False, True])
def test_partition_matches_oracle_on_random_states(big):
    rng = np.random.default_rng(700 + big)
    for case in range(3000):
        n = int(rng.integers(0, 40))
        T = int(rng.choice([1, 2, 16, 4096]))
        reqs = _random_reqs(rng, n, T, big)
        b = int(rng.integers(0, 3000)) if not big else int(rng.integers(0, 1 << 32))
        d = int(rng.integers(0, 60)) if not big else int(rng.integers(0, 1 << 32))
        cap = int(rng.integers(0, 400)) if not big else int(rng.integers(0, 1 << 63))
        if rng.random() < 0.02:
            T = 0
        st, batch, taken, idx, tok = _c_partition(reqs, b, d, cap, T)
        ost, obatch, otaken = ocfs.partition(reqs, b, d, cap, T)
        assert st == ost, (case, reqs, b, d, cap, T)
        if st == 0:
            assert batch == obatch and taken == otaken, (case, reqs, b, d, cap, T)
        else:
            assert (idx == 0xFFFFFFFF).all() and (tok == 0xFFFFFFFF).all(), "wrote on error"


def test_partition_argument_errors():
    L = aqua.load()
    prm = aqua.aqua_cfs_params(16, 2, 16, 0, 100)
    size, taken = ctypes.c_uint32(7), ctypes.c_uint64(7)
    req = np.asarray([[8, 0, 0, 0]], dtype=np.uint32)
    out = np.zeros(1, dtype=np.uint32)
    P = req.ctypes.data
    O = out.ctypes.data
    assert L.aqua_cfs_partition(None, 1, ctypes.byref(prm), O, O, ctypes.byref(size),
                                ctypes.byref(taken)) == aqua.AQUA_ERR_INVALID
    assert L.aqua_cfs_partition(P, 1, None, O, O, ctypes.byref(size),
                                ctypes.byref(taken)) == aqua.AQUA_ERR_INVALID
    assert L.aqua_cfs_partition(P, 1, ctypes.byref(prm), None, O, ctypes.byref(size),
                                ctypes.byref(taken)) == aqua.AQUA_ERR_INVALID
    assert L.aqua_cfs_partition(P, 1, ctypes.byref(prm), O, O, None,
                                ctypes.byref(taken)) == aqua.AQUA_ERR_INVALID
    assert size.value == 7 and taken.value == 7
    assert _c_partition([[8, 0, 0, 0]], 16, 2, 100, 16, reserved=1)[0] == aqua.AQUA_ERR_INVALID
    # blocks_taken may be NULL; no request needs no arrays.
    assert L.aqua_cfs_partition(P, 1, ctypes.byref(prm), O, ctypes.c_void_p(O + 0),
                                ctypes.byref(size), None) == aqua.AQUA_OK
    assert L.aqua_cfs_partition(None, 0, ctypes.byref(prm), None, None,
                                ctypes.byref(size), ctypes.byref(taken)) == aqua.AQUA_OK
    assert size.value == 0 and taken.value == 0


def _trace(rng, n, T, pool):
    tr = []
    for _ in range(n):
        while True:
            P, O = int(rng.integers(1, 300)), int(rng.integers(1, 80))
            if -(-(P + O) // T) <= pool:
                break
        tr.append((int(rng.integers(0, 60)), P, O))
    return tr


def test_rescheduler_matches_oracle_on_random_traces():
    rng = np.random.default_rng(710)
    for _ in range(150):
        T = int(rng.choice([1, 4, 16]))
        pool = int(rng.integers(20, 200))
        tr = _trace(rng, int(rng.integers(1, 40)), T, pool)
        args = (pool, T, int(rng.integers(1, 400)), int(rng.integers(1, 20)),
                int(rng.integers(1, 20)))
        log, _ = cfs.run_trace(tr, *args)
        assert log == ocfs.simulate(tr, *args)


@pytest.mark.parametrize("cfg", [wl.CFS_SMALL, wl.CFS_LLAMA8B], ids=lambda c: c.name)
def test_rescheduler_matches_oracle_on_workloads(cfg):
    tr = cfg.trace()
    d = cfg.decode_slots(tr)
    args = (cfg.shape.num_blocks, cfg.shape.block_tokens, cfg.batch_tokens, d, cfg.k)
    log, s = cfs.run_trace(tr, *args)
    assert log == ocfs.simulate(tr, *args)
    assert s.partition_calls >= len(log)
    assert sum(len(e["out"]) for e in log) > len(tr), "workload pages prompts out"


@pytest.mark.parametrize("cfg", [wl.CFS_SMALL, wl.CFS_LLAMA8B], ids=lambda c: c.name)
def test_swap_schedule_conserves_blocks(cfg):
    """Every pool block is free or in exactly one resident's table; a
    resident holds ceil(ctx / T) blocks; a prompt swaps back in as many
    blocks as it swapped out; slots do not overlap."""
    sh = cfg.shape
    T, N = sh.block_tokens, sh.num_blocks
    tr = cfg.trace()
    log, _ = cfs.run_trace(tr, N, T, cfg.batch_tokens, cfg.decode_slots(tr), cfg.k)
    sc = wl.cfs_swap_schedule(sh, cfg.seed, tr, log)
    assert len(sc.slices) == sum(e["resched"] for e in log)
    ends = [sh.image_bytes(n) + o for o, n in zip(sc.slot_offsets, sc.nblocks)]
    assert all(e + 4096 <= o for e, o in zip(ends, sc.slot_offsets[1:]))
    ctx = [0] * len(tr)
    image = {}
    e_it = iter(log)
    tables = {}
    e = next(e_it)
    for sl in sc.slices:
        assert e["resched"]
        for p, t in zip(sl.out_prompts, sl.out_tables):
            assert tables.pop(p) == t
            image[p] = len(t)
        for p, t in zip(sl.in_prompts, sl.in_tables):
            assert len(t) == image.pop(p) > 0
        while True:                       # the slice's iterations
            for p, x in e["batch"]:
                ctx[p] += x if ctx[p] < tr[p][1] else 1
            e = next(e_it, None)
            if e is None or e["resched"]:
                break
        held = [b for p in sl.resident_after for b in sl.tables_after[p]]
        assert len(held) == len(set(held)) and all(0 <= b < N for b in held)
        for p in sl.resident_after:
            assert len(sl.tables_after[p]) == -(-ctx[p] // T)
        tables = {p: list(t) for p, t in sl.tables_after.items()}
    assert e is None
    assert all(c == p + o for c, (_, p, o) in zip(ctx, tr))


def test_rescheduler_fails_loudly_when_a_context_outgrows_the_pool():
    """A request that keeps generating past what the pool holds can never be
    admitted again; the scheduler raises instead of spinning."""
    s = cfs.CfsScheduler(pool_blocks=4, block_tokens=4, batch_tokens=8, decode_slots=2, k=4)
    s.add(8)
    now = 0
    with pytest.raises(RuntimeError, match="outgrown"):
        for _ in range(100):
            st = s.step(now)
            s.advance(st, [])
            now += 1
    assert s.generated[0] >= 8       # it ran until its context filled the pool


def test_scheduler_rejects_bad_settings_and_prompts():
    with pytest.raises(ValueError):
        cfs.CfsScheduler(0, 16, 64, 2, 4)
    s = cfs.CfsScheduler(4, 4, 8, 2, 4)
    with pytest.raises(ValueError):
        s.add(0)
    with pytest.raises(ValueError):
        s.add(17)                     # 5 blocks > 4
    with pytest.raises(ValueError):
        cfs.run_trace([(0, 4, 13)], 4, 4, 8, 2, 4)    # prompt + output > pool
