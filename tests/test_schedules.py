"""The generated swap schedules never alias a live block: at every point in
issue order each physical block belongs to at most one live table, swap-ins
take only free blocks, blocks are conserved, and offload slots are disjoint.
(The GPU parity tests take these schedules as given.)"""
import pytest

from paper_2407_21255_amd import workload as wl


def _check_case(case: wl.SwapCase):
    N = case.shape.num_blocks
    live = {}
    for b, (p, i) in case.owner.items():
        assert 0 <= b < N and b not in live
        live[b] = (p, i)
    out_blocks = [b for t in case.out_tables for b in t]
    in_blocks = [b for t in case.in_tables for b in t]
    assert len(set(out_blocks)) == len(out_blocks), "a swap-out table repeats a block"
    assert all(b in live for b in out_blocks), "swap-out of a block nobody owns"
    assert len(set(in_blocks)) == len(in_blocks), "a swap-in names one block twice"
    assert all(0 <= b < N for b in in_blocks)
    assert [len(t) for t in case.in_tables] == [len(t) for t in case.out_tables]
    # Fresh blocks: not owned by any prompt still resident.
    resident = set(live) - set(out_blocks)
    assert not set(in_blocks) & resident, "swap-in overwrites a resident prompt's block"


@pytest.mark.parametrize("make", [wl.tiny_case, wl.llama8b_hbm_case, wl.llama8b_host_case,
                                  wl.llama70b_case,
                                  lambda: wl.llama70b_case(shape=wl.LLAMA70B_TP4),
                                  lambda: wl.llama8b_hbm_case(shape=wl.LLAMA8B_FP8)])
def test_single_swap_cases_are_valid(make):
    _check_case(make())


def _check_schedule(sched: wl.Schedule):
    N = sched.shape.num_blocks
    tables = {p: list(t) for p, t in sched.initial_tables.items()}
    held = [b for t in tables.values() for b in t]
    assert len(set(held)) == len(held)
    # Prompts whose image is in the region (the others have not run yet).
    swapped = (set(sched.initial_swapped) if sched.initial_swapped is not None
               else set(range(len(sched.nblocks))) - set(tables))
    # Slots: disjoint, in order, each large enough for its prompt's largest image.
    ends = [o + sched.shape.image_bytes(n) for o, n in zip(sched.slot_offsets, sched.nblocks)]
    assert all(e <= o for e, o in zip(ends, sched.slot_offsets[1:]))
    assert ends[-1] <= sched.region_bytes
    for sl in sched.slices:
        # Swap-out: the prompts' current tables, which then become free.
        for p, t in zip(sl.out_prompts, sl.out_tables):
            assert tables.pop(p) == t
            assert len(t) <= sched.nblocks[p]
            swapped.add(p)
        busy = {b for t in tables.values() for b in t}
        # Swap-in: only prompts that were out, into blocks nobody holds.
        for p, t in zip(sl.in_prompts, sl.in_tables):
            assert p in swapped and p not in tables
            assert not set(t) & busy, f"slice {sl.index}: swap-in into a live block"
            assert len(set(t)) == len(t) and all(0 <= b < N for b in t)
            busy |= set(t)
            tables[p] = list(t)
            swapped.discard(p)
        # Growth: new blocks are free ones, appended to the prompt's table.
        # A prompt that runs for the first time has no image and starts
        # with an empty table.
        for p, first, new in sl.grow:
            if p not in tables:
                assert first == 0 and p not in swapped, f"slice {sl.index}: prompt {p}"
                tables[p] = []
            assert first == len(tables[p])
            assert not set(new) & busy, f"slice {sl.index}: growth into a live block"
            busy |= set(new)
            tables[p] = tables[p] + list(new)
        for p in sl.finished:
            del tables[p]
        nonempty = {p: t for p, t in sl.tables_after.items() if t}
        assert tables == nonempty
        assert set(tables) <= set(sl.resident_after)
        held = [b for t in tables.values() for b in t]
        assert len(set(held)) == len(held) <= N


def test_preemption_schedule_never_aliases_a_live_block():
    _check_schedule(wl.preemption_schedule(n_slices=100))


@pytest.mark.parametrize("cfg", [wl.CFS_SMALL, wl.CFS_LLAMA8B], ids=lambda c: c.name)
def test_fair_scheduling_swap_schedule_never_aliases_a_live_block(cfg):
    from paper_2407_21255_amd import cfs
    sh = cfg.shape
    tr = cfg.trace()
    log, _ = cfs.run_trace(tr, sh.num_blocks, sh.block_tokens, cfg.batch_tokens,
                           cfg.decode_slots(tr), cfg.k)
    _check_schedule(wl.cfs_swap_schedule(sh, cfg.seed, tr, log))
