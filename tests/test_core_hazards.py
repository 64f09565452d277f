"""Hazard tracker on the CPU, driven by a fake device clock.

Calls on one pool must behave as if run in issue order.  The fake device
runs each lane's tickets in order, starts a ticket only after the tickets
it was told to wait for, and completes runnable tickets in random
(adversarial) order; the tracker learns of completions late.  For every
pair of conflicting calls i < j the test requires that i happens before j:
through lane order, inserted waits, or a completion the tracker had been
told of before j was issued.
"""
import numpy as np

from tests.core_lib import Tracker


def _conflict(a, b):
    """Do two calls touch the same block or bytes with at least one write?"""
    # a, b: (is_in, blocks, ranges)
    ai, ab, ar = a
    bi, bb, br = b
    a_w_blocks = set(ab) if ai else set()
    a_r_blocks = set() if ai else set(ab)
    b_w_blocks = set(bb) if bi else set()
    b_r_blocks = set() if bi else set(bb)
    if a_w_blocks & (b_w_blocks | b_r_blocks) or b_w_blocks & a_r_blocks:
        return True
    a_writes_r, b_writes_r = not ai, not bi
    if a_writes_r or b_writes_r:
        for lo, hi in ar:
            for lo2, hi2 in br:
                if lo < hi2 and lo2 < hi:
                    return True
    return False


def _overlap(ra, rb):
    return any(lo < hi2 and lo2 < hi for lo, hi in ra for lo2, hi2 in rb)


def _conflict_rw(a, b):
    """a, b: (blocks_r, blocks_w, ranges_r, ranges_w)."""
    br, bw, rr, rw = a
    cr, cw, sr, sw = b
    if set(bw) & (set(cr) | set(cw)) or set(cw) & set(br):
        return True
    return _overlap(rw, sr + sw) or _overlap(sw, rr)


def _run_sequence(rng, n_calls, n_blocks, n_lanes, inform_prob, complete_steps,
                  general=False):
    tr = Tracker(n_blocks)
    calls = []          # (is_in, blocks, ranges, lane)
    waits = {}          # ticket -> list of dep tickets
    informed_at_issue = {}
    done = set()
    informed = {m: 0 for m in range(n_lanes)}
    lane_tickets = {m: [] for m in range(n_lanes)}

    def runnable(t):
        is_in, blocks, ranges, m = calls[t - 1]
        idx = lane_tickets[m].index(t)
        if idx and lane_tickets[m][idx - 1] not in done:
            return False
        return all(d in done for d in waits[t])

    for t in range(1, n_calls + 1):
        m = int(rng.integers(0, n_lanes))
        is_in = bool(rng.random() < 0.5)
        k = int(rng.integers(0, min(4, n_blocks + 1)))
        if is_in:
            blocks = [int(x) for x in rng.choice(n_blocks, size=k, replace=False)]
        else:
            blocks = [int(x) for x in rng.integers(0, n_blocks, size=k)]
        ranges = []
        for _ in range(int(rng.integers(0, 3))):
            lo = int(rng.integers(0, 64)) * 16
            ranges.append((lo, lo + int(rng.integers(1, 8)) * 16))
        if not is_in:  # a swap-out's images never overlap each other
            ranges.sort()
            ranges = [r for i, r in enumerate(ranges) if i == 0 or r[0] >= ranges[i - 1][1]]
        if general:
            # Arbitrary read and write sets: distinct written blocks, read
            # blocks possibly repeated, ranges read and written (migration).
            kw = int(rng.integers(0, min(3, n_blocks + 1)))
            bw = [int(x) for x in rng.choice(n_blocks, size=kw, replace=False)]
            br = [int(x) for x in rng.integers(0, n_blocks, size=int(rng.integers(0, 3)))]
            br = [b for b in br if b not in bw]
            rr, rw = [], []
            for _ in range(int(rng.integers(0, 3))):
                lo = int(rng.integers(0, 64)) * 16
                (rr if rng.random() < 0.5 else rw).append(
                    (lo, lo + int(rng.integers(1, 8)) * 16))
            acc = (br, bw, rr, rw)
            deps = tr.issue_rw(t, m, br, bw, rr, rw)
        else:
            acc = (([] if is_in else blocks), (blocks if is_in else []),
                   (ranges if is_in else []), ([] if is_in else ranges))
            deps = tr.issue(t, m, is_in, blocks, ranges)
        for lane, dt in deps:
            assert lane != m and calls[dt - 1][3] == lane
        calls.append((acc, None, None, m))
        waits[t] = [dt for _, dt in deps]
        informed_at_issue[t] = dict(informed)
        lane_tickets[m].append(t)
        # The device makes progress in a random order among runnable tickets.
        for _ in range(int(rng.integers(0, complete_steps))):
            cand = [u for u in range(1, t + 1) if u not in done and runnable(u)]
            if not cand:
                break
            done.add(int(rng.choice(cand)))
        # The host learns of completions late and only in lane order.
        for lane in range(n_lanes):
            if rng.random() < inform_prob:
                w = informed[lane]
                for u in lane_tickets[lane]:
                    if u <= w:
                        continue
                    if u in done:
                        w = u
                    else:
                        break
                if w > informed[lane]:
                    informed[lane] = w
                    tr.complete(lane, w)

    # Happens-before: lane order, waits, and completions known at issue.
    n = len(calls)
    pred = {t: set(waits[t]) for t in range(1, n + 1)}
    for lane, ts in lane_tickets.items():
        for a, b in zip(ts, ts[1:]):
            pred[b].add(a)
    for t in range(1, n + 1):
        for lane, w in informed_at_issue[t].items():
            for u in lane_tickets[lane]:
                if u <= w and u < t:
                    pred[t].add(u)
    reach = {}
    for t in range(1, n + 1):
        r = set()
        for p in pred[t]:
            r.add(p)
            r |= reach[p]
        reach[t] = r
    for j in range(1, n + 1):
        for i in range(1, j):
            if _conflict_rw(calls[i - 1][0], calls[j - 1][0]):
                assert i in reach[j], (i, j, calls[i - 1], calls[j - 1], waits[j])
    return calls, waits


def test_random_sequences_are_sequentially_consistent():
    rng = np.random.default_rng(31)
    for trial in range(300):
        _run_sequence(rng, n_calls=int(rng.integers(5, 40)), n_blocks=int(rng.integers(2, 12)),
                      n_lanes=int(rng.integers(1, 4)), inform_prob=float(rng.random()),
                      complete_steps=int(rng.integers(1, 4)))


def test_random_read_write_sets_are_sequentially_consistent():
    rng = np.random.default_rng(32)
    for trial in range(300):
        _run_sequence(rng, n_calls=int(rng.integers(5, 40)), n_blocks=int(rng.integers(2, 12)),
                      n_lanes=int(rng.integers(1, 4)), inform_prob=float(rng.random()),
                      complete_steps=int(rng.integers(1, 4)), general=True)


def test_waits_only_where_needed():
    tr = Tracker(16)
    # Swap-out on lane 0 reads blocks 1, 2 and writes bytes [0, 100).
    assert tr.issue(1, 0, False, [1, 2], [(0, 96)]) == []
    # Swap-in on lane 1 into unrelated blocks from unrelated bytes: no wait.
    assert tr.issue(2, 1, True, [5, 6], [(1000, 1096)]) == []
    # Swap-in on lane 1 reusing block 2 (write after read): waits on 1.
    assert tr.issue(3, 1, True, [2, 7], [(2000, 2096)]) == [(0, 1)]
    # Swap-in on lane 2 reading bytes the swap-out wrote (read after write).
    assert tr.issue(4, 2, True, [9], [(48, 64)]) == [(0, 1)]
    # Another reader of the same bytes on lane 1: still only the writer.
    assert tr.issue(5, 1, True, [10], [(0, 32)]) == [(0, 1)]
    # A swap-out on lane 0 overwriting those bytes waits for both readers.
    assert sorted(tr.issue(6, 0, False, [11], [(0, 96)])) == [(1, 5), (2, 4)]
    # Same-lane conflicts are ordered by the stream: no event wait.
    assert tr.issue(7, 0, False, [11], [(0, 96)]) == []
    # A swap-out reading block 2 on lane 2 waits for its writer (ticket 3).
    assert tr.issue(8, 2, False, [2], [(5000, 5096)]) == [(1, 3)]
    # Once lane 1 is known complete, nothing of it is waited on.
    tr.complete(1, 5)
    tr.complete(0, 7)
    assert tr.issue(9, 2, True, [2], [(7000, 7096)]) == []  # waits on 8 via lane 2 order
    assert tr.issue(10, 0, True, [2], [(9000, 9096)]) == [(2, 9)]


def test_block_read_on_several_streams_at_once():
    """Readers of one block on several lanes at once: a later write waits
    for the newest live reader of every other lane, a lane that reads again
    replaces its own entry, and finished readers are forgotten when another
    lane joins."""
    tr = Tracker(8)
    # Swap-outs on lanes 0, 1 and 2 all read block 5 (and nothing else).
    assert tr.issue_rw(1, 0, [5], [], [], []) == []
    assert tr.issue_rw(2, 1, [5], [], [], []) == []
    assert tr.issue_rw(3, 2, [5], [], [], []) == []
    # Lane 1 reads block 5 again: its entry moves to ticket 4.
    assert tr.issue_rw(4, 1, [5, 6], [], [], []) == []
    # A swap-in on lane 3 writing block 5 waits for the newest reader of
    # each of the three lanes.
    assert sorted(tr.issue_rw(5, 3, [], [5], [], [])) == [(0, 1), (1, 4), (2, 3)]
    # After the write, a reader on lane 0 waits only for the writer.
    assert tr.issue_rw(6, 0, [5], [], [], []) == [(3, 5)]
    # Lanes 0 and 3 complete up to 6; readers join on lanes 1 and 2, and a
    # write on lane 0 waits for those two only.
    tr.complete(3, 5)
    tr.complete(0, 6)
    assert tr.issue_rw(7, 1, [5], [], [], []) == []
    assert tr.issue_rw(8, 2, [5], [], [], []) == []
    assert sorted(tr.issue_rw(9, 0, [], [5], [], [])) == [(1, 7), (2, 8)]
    # Block 6, read once by lane 1 (ticket 4), is still owed a wait.
    assert tr.issue_rw(10, 2, [], [6], [], []) == [(1, 4)]


def test_finished_ranges_are_forgotten():
    tr = Tracker(4)
    for t in range(1, 101):
        tr.issue(t, 0, False, [t % 4], [(t * 4096, t * 4096 + 4096)])
    assert tr.live_ranges() == 100
    tr.complete(0, 100)
    tr.issue(101, 1, False, [0], [(0, 16)])
    assert tr.live_ranges() == 1


def test_tracker_memory_stays_bounded_over_a_million_calls():
    """A serving loop issues 10^6 swaps over streams that are replaced by
    new handles every 1000 calls, with at most 8 calls in flight: the
    tracker keeps the lanes of the in-flight tickets only, and the stream
    map reuses idle lanes instead of growing by one per stream handle."""
    from tests.core_lib import tracker_soak
    kept, lanes = tracker_soak(1_000_000, 16384, streams=4, rotate=1000, depth=8)
    assert kept <= 9            # the in-flight tickets plus the one being issued
    assert lanes <= 4 + 8 + 1   # the streams in use, plus those still in flight


def test_completed_tickets_are_dropped_and_still_done():
    """Once every ticket up to t is complete its lane is forgotten, and done()
    still answers for it; a ticket of a lane that is behind keeps the ones
    after it."""
    tr = Tracker(64)
    for t in range(1, 11):
        tr.issue(t, t % 2, False, [t], [])
    assert tr.tickets_kept() == 10
    tr.complete(1, 9)                      # lane 1: tickets 1, 3, ..., 9
    assert tr.tickets_kept() == 9          # ticket 1 goes; ticket 2 (lane 0) holds the rest
    assert tr.done(9) and not tr.done(2)
    tr.complete(0, 6)
    assert tr.tickets_kept() == 3          # tickets 8..10 are kept
    assert all(tr.done(t) for t in range(1, 8)) and not tr.done(8)
    tr.complete(0, 10)
    assert tr.tickets_kept() == 0 and all(tr.done(t) for t in range(1, 11))
    # A later call on a forgotten block's ticket is not held back by it.
    assert tr.issue(11, 2, True, [3], []) == []


def test_skipped_tickets_count_as_complete():
    tr = Tracker(16)
    tr.issue(5, 0, False, [1], [])
    assert tr.done(2) and not tr.done(5)
    assert tr.issue(9, 1, True, [1], []) == [(0, 5)]
    tr.complete(0, 5)
    assert tr.tickets_kept() == 1          # ticket 9 only


def test_lane_map_reuses_idle_lanes_only():
    from tests.core_lib import LaneMap
    tr, lm = Tracker(16), LaneMap()
    a = lm.lane_for(0xA, tr)
    tr.issue(1, a, False, [1], [])
    b = lm.lane_for(0xB, tr)
    assert b != a                            # lane a is busy
    tr.issue(2, b, False, [2], [])
    assert lm.lane_for(0xA, tr) == a         # a stream keeps its lane
    tr.complete(a, 1)
    c = lm.lane_for(0xC, tr)
    assert c == a and lm.size() == 2         # the idle lane is handed over
    tr.issue(3, c, True, [1], [])
    assert lm.lane_for(0xA, tr) not in (b, c)  # stream A comes back: a new lane
    assert lm.size() == 3
