"""GPU parity at the full workload sizes, in the launch configuration the
bench times (default unit size and grid), element by element against the
oracle run on host copies of the same generated pools."""
import os
import time

import numpy as np
import pytest
import torch

import oracle
from paper_2407_21255_amd import aqua
from paper_2407_21255_amd import workload as wl
from paper_2407_21255_amd.cycle import run_slices, slice_tables
from tests.checkers import assert_bytes_equal
from tests.gpu_util import (apply_mutations_device, device_pool, host, odesc,
                            oracle_replay, region_for, say, schedule_owner)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    aqua.load()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _full_round_trip(case: wl.SwapCase, pinned: bool, gemm: bool = False,
                     host_path=None):
    s = case.shape
    d = odesc(s)
    t0 = time.time()
    pool = device_pool(s, case.seed, case.owner)
    say(case.name, "pool filled", round(time.time() - t0, 1), "s")
    pool_h = host(pool)
    say(case.name, "pool on host", round(time.time() - t0, 1), "s")
    size = case.payload_bytes
    if pinned:
        img = torch.empty(size, dtype=torch.uint8, pin_memory=True)
    else:
        img = torch.empty(size, dtype=torch.uint8, device="cuda")
    img.fill_(wl.GUARD_BYTE)
    torch.cuda.synchronize()  # fills ran on the current stream; swaps use another
    swap = torch.cuda.Stream()
    comp = torch.cuda.Stream()
    kv = aqua.KVPool(s.as_tuple(), pool)
    if host_path is not None:
        kv.set_host_path(host_path)
    try:
        if gemm:  # a compute stream busy with bf16 GEMMs while the swap runs
            a = torch.randn(4096, 4096, device="cuda", dtype=torch.bfloat16)
            torch.cuda.synchronize()
            with torch.cuda.stream(comp):
                for _ in range(20):
                    a = (a @ a).clamp_(-1, 1)
        kv.swap_out(case.out_tables, img, stream=swap)
        kv.sync(0)
        say(case.name, "swap-out done")
        want = np.empty(size, dtype=np.uint8)
        assert oracle.swap_out(d, pool_h, case.out_tables, want) == 0
        assert_bytes_equal(host(img), want, f"{case.name} image")
        del want
        if gemm:
            with torch.cuda.stream(comp):
                for _ in range(20):
                    a = (a @ a).clamp_(-1, 1)
        kv.swap_in(case.in_tables, img, stream=swap)
        kv.sync(0)
        say(case.name, "swap-in done")
        img_h = host(img)
        assert oracle.swap_in(d, pool_h, case.in_tables, img_h) == 0
        assert_bytes_equal(host(pool), pool_h, f"{case.name} pool")
        say(case.name, "compared", round(time.time() - t0, 1), "s")
        torch.cuda.synchronize()
    finally:
        kv.close()
        del pool, img
        torch.cuda.empty_cache()


def test_llama8b_hbm_full():
    """32 layers x 8 KV heads x 128, bf16, 16384-block pool; 8 of 16
    fragmented 2048-token prompts out to the HBM region and back."""
    _full_round_trip(wl.llama8b_hbm_case(), pinned=False)


@pytest.mark.parametrize("path", ["zero_copy", "staged"])
def test_llama8b_pinned_host_full_with_gemm(path):
    """8 x 4096-token prompts out to pinned host memory and back while a
    second stream runs bf16 GEMMs."""
    _full_round_trip(wl.llama8b_host_case(), pinned=True, gemm=True,
                     host_path={"staged": aqua.AQUA_HOST_STAGED,
                                "zero_copy": aqua.AQUA_HOST_ZERO_COPY}[path])


def test_llama70b_hbm_full():
    """80 layers, one 32768-token prompt (10 GiB) to the HBM region."""
    _full_round_trip(wl.llama70b_case(), pinned=False)


@pytest.mark.parametrize("shape", [wl.LLAMA70B_TP2, wl.LLAMA70B_TP4, wl.LLAMA8B_FP8],
                         ids=["70b_tp2", "70b_tp4", "8b_fp8"])
def test_smaller_chunks_hbm_full(shape):
    """One tensor-parallel rank's share of the 70B pool (32 and 16 KiB
    chunks) and the fp8 8B pool (32 KiB chunks): a workgroup's 64 KiB pass
    covers one chunk partly, so the ragged tail path carries the copy."""
    if shape.num_layers == 80:
        case = wl.llama70b_case(shape=shape)
    else:
        case = wl.llama8b_hbm_case(shape=shape)
    _full_round_trip(case, pinned=False)


@pytest.mark.parametrize("path", ["zero_copy", "staged"])
def test_llama70b_pinned_host_full(path):
    """The 10 GiB image of one 32768-token prompt in pinned host memory."""
    _full_round_trip(wl.llama70b_case(seed=14), pinned=True,
                     host_path={"staged": aqua.AQUA_HOST_STAGED,
                                "zero_copy": aqua.AQUA_HOST_ZERO_COPY}[path])


def test_preemption_cycle_full():
    """64 prompts of 128..8192 tokens on the fp8 8B-shaped pool; every slice
    swaps 16 out on one stream and 16 in on another, then the host mutates
    the residents and the consumed slots.  The whole pool and offload region
    must equal the oracle's replay."""
    # The configuration runs 100 slices; AQUA_TEST_SLICES shortens a quick run.
    n = int(os.environ.get("AQUA_TEST_SLICES", "100"))
    sched = wl.preemption_schedule(n_slices=n)
    s = sched.shape
    t0 = time.time()
    pool = device_pool(s, sched.seed, schedule_owner(sched))
    region = region_for(sched)
    pool_h, region_h = host(pool), host(region)
    say("cycle inputs ready", round(time.time() - t0, 1), "s")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(s.as_tuple(), pool)
    try:
        prepared = [slice_tables(sched, k) for k in range(n)]
        run_slices(kv, region, sched, 0, n, sa, sb,
                   between=lambda k: apply_mutations_device(sched, k, pool, region),
                   prepared=prepared)
        torch.cuda.synchronize()
        st = kv.stats()
        say("cycle on GPU done", round(time.time() - t0, 1), "s", st)
        oracle_replay(sched, pool_h, region_h, 0, n)
        say("oracle replay done", round(time.time() - t0, 1), "s")
        assert_bytes_equal(host(region), region_h, "offload region")
        assert_bytes_equal(host(pool), pool_h, "pool")
        assert st["calls_out"] == n and st["calls_in"] == n
    finally:
        kv.close()
        del pool, region
        torch.cuda.empty_cache()


@pytest.mark.parametrize("path", ["staged", "zero_copy"])
def test_preemption_cycle_pinned_host(path):
    """The preemption cycle with the offload region in pinned host memory
    (17.7 GB): every slice swaps 16 prompts out on one stream and 16 in on
    another, both directions of the link at once (staged: one copy engine
    per direction), then the host mutates the residents and the consumed
    slots.  Pool and region must equal the oracle's replay."""
    n = int(os.environ.get("AQUA_TEST_HOST_SLICES", "6"))
    sched = wl.preemption_schedule(n_slices=n)
    s = sched.shape
    t0 = time.time()
    pool = device_pool(s, sched.seed, schedule_owner(sched))
    region = torch.empty(sched.region_bytes, dtype=torch.uint8, pin_memory=True)
    staging = region_for(sched)
    region.copy_(staging)
    del staging
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    pool_h = host(pool)
    region_h = region.numpy().copy()
    say("host cycle inputs ready", path, round(time.time() - t0, 1), "s")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(s.as_tuple(), pool)
    kv.set_host_path({"staged": aqua.AQUA_HOST_STAGED,
                      "zero_copy": aqua.AQUA_HOST_ZERO_COPY}[path])
    try:
        prepared = [slice_tables(sched, k) for k in range(n)]
        run_slices(kv, region, sched, 0, n, sa, sb,
                   between=lambda k: apply_mutations_device(sched, k, pool, region),
                   prepared=prepared)
        torch.cuda.synchronize()
        st = kv.stats()
        say("host cycle on GPU done", path, round(time.time() - t0, 1), "s",
            [kv.link_engine(0), kv.link_engine(1)], st)
        oracle_replay(sched, pool_h, region_h, 0, n)
        say("oracle replay done", round(time.time() - t0, 1), "s")
        assert_bytes_equal(region.numpy(), region_h, "pinned offload region")
        del region_h
        assert_bytes_equal(host(pool), pool_h, "pool")
        assert st["calls_out"] == n and st["calls_in"] == n and st["hip_error"] == 0
    finally:
        kv.close()
        del pool, region
        torch.cuda.empty_cache()


def test_preemption_cycle_without_host_syncs():
    """The same schedule issued slice after slice with no host
    synchronisation (no mutations in between): blocks that one slice frees
    are reused by later swap-ins while earlier swap-outs may still read
    them, and only the library's waits keep the result equal to the
    oracle's sequential replay."""
    n = 24
    sched = wl.preemption_schedule(n_slices=n, seed=15)
    s = sched.shape
    pool = device_pool(s, sched.seed, schedule_owner(sched))
    region = region_for(sched)
    pool_h, region_h = host(pool), host(region)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    kv = aqua.KVPool(s.as_tuple(), pool)
    try:
        for k in range(n):
            out, out_off, inn, in_off = slice_tables(sched, k)
            kv.swap_out(out, region, out_off, stream=sa)
            kv.swap_in(inn, region, in_off, stream=sb)
        kv.sync(0)
        st = kv.stats()
        say("unsynchronised cycle", st)
        oracle_replay(sched, pool_h, region_h, 0, n, mutate=False)
        assert_bytes_equal(host(region), region_h, "offload region")
        assert_bytes_equal(host(pool), pool_h, "pool")
        assert st["waits_inserted"] > 0
    finally:
        kv.close()
        del pool, region
        torch.cuda.empty_cache()
