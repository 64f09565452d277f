"""CPU oracle for Aqua's fair batch partitioner and its k-iteration
rescheduler -- TEST INFRASTRUCTURE ONLY (Aqua, section 7, "Fair scheduling
prompts with Aqua").

Plain Python loops, written from the paper's description of the algorithm
and taken in its order; only the tests, the smoke check and the bench's
CPU-baseline leg may import this module.  It shares nothing with the
library's partitioner.

Partition (one inference iteration's batch of ``b`` tokens):

1. The decode share ``d`` is set to its upper bound, the number of prompts
   that fit in GPU memory (the caller's ``decode_slots``; at most ``b``); the
   prefill share is ``p = b - d``.
2. ``p`` is filled with prompts still in prefill, those with the fewest
   prompt tokens computed first; each takes a chunk of as many of its
   remaining prompt tokens as the share has left (chunked prefill).
3. ``d`` is filled with prompts in decode, those with the fewest generated
   tokens first, one token each.
4. Decode slots left over go to the prefill prompts, continuing the order of
   step 2 (first the chunk that step 2 cut short, then further prompts).
5. Filling stops -- for the whole batch -- at the first prompt whose KV
   blocks would not fit in the memory left.

Readings where the paper is silent (each a choice of this implementation):

* Equal service is broken by request index (arrival order).
* Memory is counted in KV blocks of ``block_tokens`` tokens.  A prompt with
  ``ctx`` cached tokens that computes ``x`` more needs ``ceil((ctx + x) / T)``
  blocks after the iteration; ``held`` of them are already its own and not
  part of ``capacity``, so it takes ``max(0, ceil((ctx + x)/T) - held)``.
  At a reschedule nothing is held (prompts left out are paged out) and the
  capacity is the whole pool; inside a time slice the residents hold their
  blocks and the capacity is the pool's free blocks.
* ``ctx`` is prompt tokens computed plus tokens generated; a prefill chunk
  does not itself produce a token; each decode iteration produces one.

Status codes are the library's: 0 ok, -1 invalid.
"""
from __future__ import annotations

OK, ERR_INVALID = 0, -1


def _blocks(tokens, T):
    return -(-tokens // T)


def partition(reqs, batch_tokens, decode_slots, capacity_blocks, block_tokens):
    """One iteration's batch.

    ``reqs`` is a sequence of ``(prompt_tokens, prefill_done, generated,
    held_blocks)``.  Returns ``(status, batch, blocks_taken)`` where ``batch``
    is a list of ``[request index, tokens]`` in admission order."""
    if block_tokens < 1 or batch_tokens < 1 or decode_slots < 1 or capacity_blocks < 0:
        return ERR_INVALID, [], 0
    for P, c, g, h in reqs:
        if P < 1 or c > P or (g > 0 and c < P) or min(P, c, g, h) < 0:
            return ERR_INVALID, [], 0
    T = block_tokens

    def takes(i, x):
        P, c, g, h = reqs[i]
        return max(0, _blocks(c + g + x, T) - h)

    d = min(decode_slots, batch_tokens)
    p = batch_tokens - d
    # Least served first: prefill by prompt tokens computed, decode by tokens
    # generated; ties by request index.
    prefills = sorted([i for i, r in enumerate(reqs) if r[1] < r[0]],
                      key=lambda i: (reqs[i][1], i))
    decodes = sorted([i for i, r in enumerate(reqs) if r[1] == r[0]],
                     key=lambda i: (reqs[i][2], i))

    batch = []              # [index, tokens], admission order
    where = {}              # index -> position in batch
    mem_left = capacity_blocks
    stopped = False
    cursor = 0              # next position in ``prefills``

    def fill_prefill(budget):
        nonlocal mem_left, stopped, cursor
        while budget > 0 and cursor < len(prefills):
            i = prefills[cursor]
            have = batch[where[i]][1] if i in where else 0
            rem = reqs[i][0] - reqs[i][1] - have
            x = min(rem, budget)
            extra = takes(i, have + x) - (takes(i, have) if i in where else 0)
            if extra > mem_left:
                stopped = True
                return budget
            mem_left -= extra
            if i in where:
                batch[where[i]][1] = have + x
            else:
                where[i] = len(batch)
                batch.append([i, x])
            budget -= x
            if x == rem:
                cursor += 1
        return budget

    # Step 2: the prefill share.
    p_left = fill_prefill(p)
    # Step 3: the decode share.
    n_dec = 0
    if not stopped:
        for i in decodes:
            if n_dec == d:
                break
            extra = takes(i, 1)
            if extra > mem_left:
                stopped = True
                break
            mem_left -= extra
            where[i] = len(batch)
            batch.append([i, 1])
            n_dec += 1
    # Step 4: decode slots left over go to prefill.
    if not stopped:
        fill_prefill(p_left + (d - n_dec))
    return OK, batch, capacity_blocks - mem_left


def simulate(trace, pool_blocks, block_tokens, batch_tokens, decode_slots, k,
             max_iterations=10 ** 7):
    """Run a trace to completion under the rescheduler (section 7: the batch
    is re-formed every ``k`` iterations or when a request completes; prompts
    outside the new batch are paged out, those joining it paged in).

    ``trace`` is a sequence of ``(arrival iteration, prompt tokens, output
    tokens)``.  Returns a list with one entry per executed iteration::

        {"t": iteration, "resched": bool, "out": [...], "in": [...],
         "batch": [[index, tokens], ...], "done": [...]}

    ``out``/``in`` (in increasing index order) are the prompts paged out and
    in at a reschedule.  Additional readings: a request is seen by the first
    reschedule at or after its arrival; when an iteration inside a slice can
    admit no resident (memory), the batch is re-formed at once instead; with
    nothing arrived and nothing resident, time skips to the next arrival."""
    n = len(trace)
    T = block_tokens
    arr = [a for a, _, _ in trace]
    P = [q for _, q, _ in trace]
    O = [o for _, _, o in trace]
    c = [0] * n
    g = [0] * n
    done = [False] * n
    resident = []           # indices, increasing
    log = []
    t = 0
    since = 0               # iterations since the last reschedule
    resched = True
    n_done = 0
    for a, q, o in trace:
        assert q >= 1 and o >= 1 and _blocks(q + o, T) <= pool_blocks
    while n_done < n:
        assert len(log) < max_iterations, "simulation does not terminate"
        cands = [i for i in range(n) if arr[i] <= t and not done[i]]
        if not cands:
            t = min(arr[i] for i in range(n) if not done[i])
            resched = True
            continue
        entry = {"t": t, "resched": False, "out": [], "in": [], "batch": [], "done": []}
        if not resched:
            reqs = [(P[i], c[i], g[i], _blocks(c[i] + g[i], T)) for i in resident]
            free = pool_blocks - sum(r[3] for r in reqs)
            st, b, _ = partition(reqs, batch_tokens, decode_slots, free, T)
            assert st == OK
            if not b:
                resched = True          # nothing resident can grow: re-form now
                continue
            batch = [[resident[j], x] for j, x in b]
        else:
            reqs = [(P[i], c[i], g[i], 0) for i in cands]
            st, b, _ = partition(reqs, batch_tokens, decode_slots, pool_blocks, T)
            assert st == OK and b
            batch = [[cands[j], x] for j, x in b]
            members = sorted(i for i, _ in batch)
            entry["resched"] = True
            entry["out"] = [i for i in resident if i not in members]
            entry["in"] = [i for i in members if i not in resident]
            resident = members
            since = 0
            resched = False
        for i, x in batch:
            if c[i] < P[i]:
                c[i] += x
            else:
                g[i] += 1
        fin = [i for i, _ in batch if g[i] == O[i]]
        for i in fin:
            done[i] = True
            n_done += 1
        resident = [i for i in resident if not done[i]]
        entry["batch"] = batch
        entry["done"] = sorted(fin)
        log.append(entry)
        t += 1
        since += 1
        if fin or since == k:
            resched = True
    return log
