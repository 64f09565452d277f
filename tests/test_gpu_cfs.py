"""GPU parity of the swaps that fair scheduling issues (Aqua, section 7):
the rescheduler's page-outs and page-ins become block-level swap calls,
the slice's compute stand-in grows the residents' KV between them.

* small pool: the whole run, then the pool and offload region bit for bit
  against the oracle's replay of the same schedule;
* Llama-3-8B-shaped pool at full size: the first slices of the run, then a
  sample of resident chunks and swapped-out image chunks against the values
  the generator defines for them (no other write touches them).
"""
import os
import time

import numpy as np
import pytest
import torch

from oracle import cfs as ocfs
from paper_2407_21255_amd import aqua
from paper_2407_21255_amd import cfs
from paper_2407_21255_amd import workload as wl
from paper_2407_21255_amd.cycle import run_slices, slice_tables
from tests.checkers import assert_bytes_equal
from tests.gpu_util import apply_mutations_device, device_pool, host, oracle_replay, \
    region_for, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    aqua.load()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _schedule(cfg):
    tr = cfg.trace()
    sh = cfg.shape
    args = (sh.num_blocks, sh.block_tokens, cfg.batch_tokens, cfg.decode_slots(tr), cfg.k)
    log, _ = cfs.run_trace(tr, *args)
    assert log == ocfs.simulate(tr, *args), "rescheduler differs from the oracle's"
    return tr, wl.cfs_swap_schedule(sh, cfg.seed, tr, log)


@pytest.mark.parametrize("where", ["hbm", "staged", "zero_copy"])
def test_cfs_schedule_small_whole_run(where):
    cfg = wl.CFS_SMALL
    sh = cfg.shape
    tr, sched = _schedule(cfg)
    n = len(sched.slices)
    say("cfs small:", n, "slices,", where)
    pool = device_pool(sh, cfg.seed)
    region = region_for(sched)
    if where != "hbm":
        pinned = torch.empty(region.numel(), dtype=torch.uint8, pin_memory=True)
        pinned.copy_(region.cpu())
        region = pinned
    pool_h, region_h = host(pool), host(region)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(sh.as_tuple(), pool)
    if where != "hbm":
        kv.set_host_path(aqua.AQUA_HOST_STAGED if where == "staged" else aqua.AQUA_HOST_ZERO_COPY)

    def between(k):
        wl.apply_growth(pool, sched, k)
        apply_mutations_device(sched, k, pool, region)

    try:
        run_slices(kv, region, sched, 0, n, sa, sb, between=between)
        torch.cuda.synchronize()
        st = kv.stats()
        say("cfs small on GPU", st)
        oracle_replay(sched, pool_h, region_h, 0, n)
        assert_bytes_equal(host(region), region_h, "offload region")
        assert_bytes_equal(host(pool), pool_h, "pool")
        assert st["calls_out"] == n and st["calls_in"] == n
        assert st["bytes_out"] == sum(len(t) for sl in sched.slices for t in sl.out_tables) * \
            sh.num_layers * sh.chunk_bytes
    finally:
        kv.close()


def test_cfs_schedule_small_without_host_syncs():
    """Every reschedule's swaps issued back to back on two streams with no
    host synchronisation and no compute in between: the swap-ins of one
    reschedule reuse blocks that its own and earlier swap-outs still read,
    and only the library's waits keep the end state equal to the oracle's
    sequential replay."""
    cfg = wl.CFS_SMALL
    sh = cfg.shape
    tr, sched = _schedule(cfg)
    n = len(sched.slices)
    pool = device_pool(sh, cfg.seed)
    region = region_for(sched)
    pool_h, region_h = host(pool), host(region)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(sh.as_tuple(), pool)
    try:
        for k in range(n):
            out, out_off, inn, in_off = slice_tables(sched, k)
            kv.swap_out(out, region, out_off, stream=sa)
            kv.swap_in(inn, region, in_off, stream=sb)
        kv.sync(0)
        st = kv.stats()
        say("cfs small unsynchronised", st)
        oracle_replay(sched, pool_h, region_h, 0, n, mutate=False, grow=False)
        assert_bytes_equal(host(region), region_h, "offload region")
        assert_bytes_equal(host(pool), pool_h, "pool")
        assert st["waits_inserted"] > 0
    finally:
        kv.close()


def _expected(sh, seed, keys):
    k = torch.from_numpy(np.ascontiguousarray(keys, dtype=np.uint64).view(np.int64))
    return wl.chunk_values(k, sh.chunk_bytes, sh.dtype).numpy()


def _sample_check(sched, cfg, pool, region, k, rng):
    """Resident chunks and swapped-out image chunks after reschedule k hold
    the generator's values for their (prompt, layer, logical block).
    Returns the number of chunks each sample could draw from."""
    sh = cfg.shape
    L, N, C = sh.num_layers, sh.num_blocks, sh.chunk_bytes
    last = sched.slices[k]
    res = [(p, i) for p in last.resident_after for i in range(len(last.tables_after[p]))]
    if res:
        pick = rng.choice(len(res), size=min(384, len(res)), replace=False)
        lay = rng.integers(0, L, size=len(pick))
        pi = np.asarray([res[j] for j in pick], dtype=np.int64)
        blocks = np.asarray([last.tables_after[p][i] for p, i in pi], dtype=np.int64)
        want = _expected(sh, cfg.seed, wl.chunk_keys_np(cfg.seed, wl.TAG_LIVE, pi[:, 0], lay,
                                                        pi[:, 1]))
        P = pool.view(L, N, C)
        got = P[torch.from_numpy(lay).cuda(), torch.from_numpy(blocks).cuda()].cpu().numpy()
        assert_bytes_equal(got, want, f"resident chunks after reschedule {k}")
    # Swapped-out images: the last image each such prompt wrote.
    image = {}
    for sl in sched.slices[:k + 1]:
        for p, t in zip(sl.out_prompts, sl.out_tables):
            image[p] = len(t)
        for p in sl.in_prompts:
            image.pop(p)
    finished = {p for sl in sched.slices[:k + 1] for p in sl.finished}
    out = [(p, i) for p, m in image.items() if p not in finished and p not in
           last.tables_after for i in range(m)]
    if out:
        pick = rng.choice(len(out), size=min(384, len(out)), replace=False)
        po = np.asarray([out[j] for j in pick], dtype=np.int64)
        lay = rng.integers(0, L, size=len(pick))
        offs = np.asarray([sched.slot_offsets[p] + (l * image[p] + i) * C
                           for (p, i), l in zip(po, lay)], dtype=np.int64)
        idx = torch.from_numpy(offs).cuda().reshape(-1, 1) + torch.arange(C, device="cuda")
        got = region[idx.reshape(-1)].view(-1, C).cpu().numpy()
        want = _expected(sh, cfg.seed, wl.chunk_keys_np(cfg.seed, wl.TAG_LIVE, po[:, 0], lay,
                                                        po[:, 1]))
        assert_bytes_equal(got, want, f"swapped-out image chunks after reschedule {k}")
    return len(res), len(out)


def test_cfs_schedule_llama8b_sampled():
    """The 8B burst at full size, in segments of 60 reschedules (60 by
    default, the whole run of 349 with AQUA_TEST_CFS_SLICES=349), with a
    sampled check after each segment."""
    cfg = wl.CFS_LLAMA8B
    sh = cfg.shape
    tr, sched = _schedule(cfg)
    n = min(len(sched.slices), int(os.environ.get("AQUA_TEST_CFS_SLICES", "60")))
    t0 = time.time()
    pool = device_pool(sh, cfg.seed)
    region = region_for(sched)
    torch.cuda.synchronize()
    say("cfs llama8b inputs ready", round(time.time() - t0, 1), "s; running", n, "of",
        len(sched.slices), "slices")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(sh.as_tuple(), pool)
    rng = np.random.default_rng(720)
    try:
        checked = 0
        for a in range(0, n, 60):
            b = min(n, a + 60)
            prepared = {k: slice_tables(sched, k) for k in range(a, b)}
            run_slices(kv, region, sched, a, b - a, sa, sb,
                       between=lambda k: wl.apply_growth(pool, sched, k),
                       prepared=[prepared.get(k) for k in range(b)])
            torch.cuda.synchronize()
            nres, nout = _sample_check(sched, cfg, pool, region, b - 1, rng)
            checked += bool(nres) + bool(nout)
            say("cfs llama8b after reschedule", b - 1, round(time.time() - t0, 1), "s:",
                nres, "resident chunks,", nout, "image chunks sampled from")
        st = kv.stats()
        say("cfs llama8b on GPU", st)
        assert st["bytes_out"] > 100 * 2 ** 30, "the sampled slices must page real volume"
        assert checked >= 2
    finally:
        kv.close()
        del pool, region
        torch.cuda.empty_cache()
