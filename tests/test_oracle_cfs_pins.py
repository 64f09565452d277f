"""Pins of the fair-scheduling oracle (Aqua, section 7) against facts that do
not come from the oracle itself:

* hand-worked partitions and a hand-worked rescheduler run
  (``golden/cfs_partition.json``, each case with its derivation);
* closed forms: decodes only -> the d least-generated (a stable argsort);
  prefills only with memory to spare -> a water fill of the b tokens in
  least-computed order (a cumulative sum);
* invariants on random states: budget, one token per decode, least-served
  prefixes, memory, and that more memory only extends the batch (filling
  stops at the first prompt that does not fit, it does not skip it);
* rescheduler: every request finishes with its exact token counts, memory
  never overflows, reschedules are at most k iterations apart, equal decode
  requests are served within k tokens of each other, and with no
  contention nothing is ever paged out.
"""
import json
import os

import numpy as np
import pytest

from oracle import cfs

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "cfs_partition.json")))


def _part(reqs, b, d, cap, T):
    return cfs.partition([tuple(int(v) for v in r) for r in reqs], b, d, cap, T)


@pytest.mark.parametrize("case", GOLDEN["partition"], ids=lambda c: c["name"])
def test_hand_worked_partitions(case):
    p = case["params"]
    st, batch, taken = _part(case["requests"], p["batch_tokens"], p["decode_slots"],
                             p["capacity_blocks"], p["block_tokens"])
    assert st == cfs.OK
    assert batch == case["batch"]
    assert taken == case["blocks_taken"]


@pytest.mark.parametrize("case", GOLDEN["invalid"], ids=lambda c: c["why"])
def test_invalid_states_are_rejected(case):
    p = case["params"]
    st, batch, taken = _part(case["requests"], p["batch_tokens"], p["decode_slots"],
                             p["capacity_blocks"], p["block_tokens"])
    assert st == cfs.ERR_INVALID and batch == [] and taken == 0


@pytest.mark.parametrize("s", GOLDEN["simulate"], ids=lambda s: s["name"])
def test_hand_worked_reschedules(s):
    p = s["params"]
    log = cfs.simulate([tuple(x) for x in s["trace"]], p["pool_blocks"], p["block_tokens"],
                       p["batch_tokens"], p["decode_slots"], p["k"])
    assert log == s["log"]


def _random_state(rng, n, T, decode_frac=0.5):
    reqs = []
    for _ in range(n):
        P = int(rng.integers(1, 200))
        if rng.random() < decode_frac:
            reqs.append((P, P, int(rng.integers(0, 50)), 0))
        else:
            reqs.append((P, int(rng.integers(0, P)), 0, 0))
    return reqs


def test_decodes_only_take_the_least_generated():
    rng = np.random.default_rng(600)
    for _ in range(300):
        n = int(rng.integers(0, 30))
        T = int(rng.choice([1, 4, 16]))
        reqs = _random_state(rng, n, T, decode_frac=1.0)
        b = int(rng.integers(1, 40))
        d = int(rng.integers(1, 40))
        st, batch, _ = _part(reqs, b, d, 10 ** 9, T)
        assert st == 0
        gen = np.asarray([r[2] for r in reqs], dtype=np.int64)
        want = np.argsort(gen, kind="stable")[:min(d, b, n)]
        assert [i for i, _ in batch] == [int(i) for i in want]
        assert all(x == 1 for _, x in batch)


def test_prefills_only_water_fill_the_whole_budget():
    """With no decode prompt every decode slot is left over, so all b tokens
    go to prefill chunks in least-computed order."""
    rng = np.random.default_rng(601)
    for _ in range(300):
        n = int(rng.integers(0, 20))
        reqs = _random_state(rng, n, 16, decode_frac=0.0)
        b = int(rng.integers(1, 1500))
        d = int(rng.integers(1, 64))
        st, batch, _ = _part(reqs, b, d, 10 ** 9, 16)
        assert st == 0
        order = sorted(range(n), key=lambda i: (reqs[i][1], i))
        rem = np.asarray([reqs[i][0] - reqs[i][1] for i in order], dtype=np.int64)
        before = np.concatenate([[0], np.cumsum(rem)[:-1]]) if n else rem
        x = np.clip(b - before, 0, rem)
        want = [[order[j], int(x[j])] for j in range(n) if x[j] > 0]
        assert batch == want


def test_shares_with_memory_to_spare():
    """d decodes (or all there are) take one token each; prefill gets p plus
    the unused decode slots, as far as the prompts have tokens left."""
    rng = np.random.default_rng(602)
    for _ in range(500):
        n = int(rng.integers(0, 30))
        reqs = _random_state(rng, n, 8)
        b = int(rng.integers(1, 600))
        dslots = int(rng.integers(1, 50))
        st, batch, _ = _part(reqs, b, dslots, 10 ** 9, 8)
        d = min(dslots, b)
        n_dec_avail = sum(1 for r in reqs if r[1] == r[0])
        n_dec = sum(1 for i, _ in batch if reqs[i][1] == reqs[i][0])
        pre = sum(x for i, x in batch if reqs[i][1] < reqs[i][0])
        rem = sum(r[0] - r[1] for r in reqs)
        assert n_dec == min(d, n_dec_avail)
        assert pre == min(rem, (b - d) + (d - n_dec))


def _takes(r, x, T):
    P, c, g, h = r
    return max(0, -(-(c + g + x) // T) - h)


def _check_invariants(reqs, b, dslots, cap, T, batch, taken):
    d = min(dslots, b)
    idx = [i for i, _ in batch]
    assert len(set(idx)) == len(idx)
    assert sum(x for _, x in batch) <= b
    dec = [i for i in idx if reqs[i][1] == reqs[i][0]]
    pre = [i for i in idx if reqs[i][1] < reqs[i][0]]
    assert len(dec) <= d
    tok = dict(batch)
    for i in dec:
        assert tok[i] == 1
    for i in pre:
        assert 1 <= tok[i] <= reqs[i][0] - reqs[i][1]
    # Least served first: the admitted prompts of each kind are a prefix of
    # that kind's order, and only the last prefill may be cut short.
    dorder = sorted([i for i, r in enumerate(reqs) if r[1] == r[0]], key=lambda i: (reqs[i][2], i))
    porder = sorted([i for i, r in enumerate(reqs) if r[1] < r[0]], key=lambda i: (reqs[i][1], i))
    assert sorted(dec, key=dorder.index) == dorder[:len(dec)]
    assert sorted(pre, key=porder.index) == porder[:len(pre)]
    ps = sorted(pre, key=porder.index)
    for i in ps[:-1]:
        assert tok[i] == reqs[i][0] - reqs[i][1]
    # Memory.
    assert taken == sum(_takes(reqs[i], x, T) for i, x in batch)
    assert taken <= cap


def test_invariants_and_memory_monotonicity_on_random_states():
    rng = np.random.default_rng(603)
    for _ in range(600):
        n = int(rng.integers(0, 25))
        T = int(rng.choice([1, 2, 16]))
        reqs = _random_state(rng, n, T)
        if rng.random() < 0.5:        # inside a slice: some blocks are held
            reqs = [(P, c, g, int(rng.integers(0, -(-(c + g) // T) + 1))) for P, c, g, _ in reqs]
        b = int(rng.integers(1, 400))
        dslots = int(rng.integers(1, 30))
        caps = sorted(int(v) for v in rng.integers(0, 200, size=4))
        prev = None
        for cap in caps:
            st, batch, taken = _part(reqs, b, dslots, cap, T)
            assert st == 0
            _check_invariants(reqs, b, dslots, cap, T, batch, taken)
            if prev is not None:
                # More memory extends the admission sequence; it never
                # admits a different prompt in place of one it stopped at.
                pi = [i for i, _ in prev]
                assert [i for i, _ in batch][:len(pi)] == pi
                for (i, x0), (j, x1) in zip(prev, batch):
                    assert x0 <= x1
            prev = batch


def test_relabelling_requests_relabels_the_batch():
    """Service decides the order, not the position in the input (states
    without ties, so that the index tie-break plays no part)."""
    rng = np.random.default_rng(604)
    for _ in range(200):
        n = int(rng.integers(1, 20))
        served = rng.permutation(1000)[:n]
        reqs = []
        for k in range(n):
            if rng.random() < 0.5:          # prefill, keyed by tokens computed
                reqs.append((int(served[k]) + int(rng.integers(1, 50)), int(served[k]), 0, 0))
            else:                           # decode, keyed by tokens generated
                P = int(rng.integers(1, 100))
                reqs.append((P, P, int(served[k]), 0))
        perm = rng.permutation(n)
        shuffled = [reqs[j] for j in perm]
        b, dslots, cap = int(rng.integers(1, 500)), int(rng.integers(1, 20)), int(rng.integers(0, 300))
        _, b1, t1 = _part(reqs, b, dslots, cap, 16)
        _, b2, t2 = _part(shuffled, b, dslots, cap, 16)
        assert [[int(perm[i]), x] for i, x in b2] == b1 and t1 == t2


def _random_trace(rng, n, T, pool):
    tr = []
    for _ in range(n):
        while True:
            P, O = int(rng.integers(1, 120)), int(rng.integers(1, 40))
            if -(-(P + O) // T) <= pool:
                break
        tr.append((int(rng.integers(0, 30)), P, O))
    return tr


def _replay_checks(trace, log, pool, T, k):
    n = len(trace)
    c, g = [0] * n, [0] * n
    resident, done = set(), set()
    since = None
    for j, e in enumerate(log):
        if j and log[j - 1]["done"]:
            assert e["resched"], "a completion re-forms the batch"
        if e["resched"]:
            assert since is None or since <= k
            assert set(e["out"]) <= resident
            assert not set(e["in"]) & resident
            resident = (resident - set(e["out"])) | set(e["in"])
            since = 0
            for i, _ in e["batch"]:
                assert trace[i][0] <= e["t"], "scheduled before its arrival"
        for i, x in e["batch"]:
            assert i in resident and i not in done
            if c[i] < trace[i][1]:
                c[i] += x
                assert c[i] <= trace[i][1]
            else:
                assert x == 1
                g[i] += 1
        assert sum(-(-(c[i] + g[i]) // T) for i in resident) <= pool, "pool overflow"
        for i in e["done"]:
            assert g[i] == trace[i][2]
            resident.discard(i)
            done.add(i)
        since += 1
    assert done == set(range(n))
    assert c == [p for _, p, _ in trace] and g == [o for _, _, o in trace]


def test_rescheduler_runs_every_request_to_completion_within_memory():
    rng = np.random.default_rng(605)
    for _ in range(60):
        T = int(rng.choice([1, 4, 16]))
        pool = int(rng.integers(8, 60))
        trace = _random_trace(rng, int(rng.integers(1, 25)), T, pool)
        b, dslots, k = int(rng.integers(1, 200)), int(rng.integers(1, 12)), int(rng.integers(1, 8))
        log = cfs.simulate(trace, pool, T, b, dslots, k)
        _replay_checks(trace, log, pool, T, k)


def test_equal_decode_requests_are_served_within_k_tokens():
    """CFS fairness: n equal requests, memory for m of them; once every
    prompt is prefilled, at every reschedule the generated counts of the
    requests differ by at most k (each slice serves the m least-generated
    for k tokens)."""
    for n, m, k in [(10, 3, 4), (12, 5, 1), (9, 4, 7)]:
        T, P, O = 4, 4, 200
        pool = m * (-(-(P + O) // T))
        trace = [(0, P, O)] * n
        log = cfs.simulate(trace, pool, T, 64, m, k)
        c, g = [0] * n, [0] * n
        checked = 0
        for e in log:
            if e["resched"] and min(c) == P and not e["done"] and max(g) < O:
                assert max(g) - min(g) <= k, (n, m, k, e["t"], g)
                checked += 1
            for i, x in e["batch"]:
                if c[i] < P:
                    c[i] += x
                else:
                    g[i] += 1
        assert g == [O] * n and checked > 10


def test_no_contention_means_no_paging():
    """Memory and decode slots for everyone: nothing is paged out, every
    prompt is prefilled at its first iteration and request i finishes at
    iteration O_i (all arrive together)."""
    rng = np.random.default_rng(606)
    T = 16
    trace = [(0, int(rng.integers(1, 300)), int(rng.integers(1, 50))) for _ in range(20)]
    pool = sum(-(-(P + O) // T) for _, P, O in trace)
    b = sum(P for _, P, _ in trace) + 20
    log = cfs.simulate(trace, pool, T, b, 20, 8)
    assert all(e["out"] == [] for e in log)
    fin = {i: e["t"] for e in log for i in e["done"]}
    assert fin == {i: O for i, (_, _, O) in enumerate(trace)}
