"""Fair time-sliced scheduling of prompts with KV paging (Aqua, section 7).

``CfsScheduler`` is the engine-facing half of the scheme: it decides, for
every inference iteration, which prompts compute how many tokens, and, at
every reschedule, which prompts leave the GPU (page-out) and which come
back (page-in).  The partition of one iteration is the library's
``aqua_cfs_partition`` (C ABI); this module keeps the per-request state and
applies the rescheduling rule:

* the batch is re-formed every ``k`` iterations, when a request completes,
  and when no resident prompt can grow inside the current slice (memory);
* at a reschedule the partition runs over every request that has arrived
  and not completed, holding nothing and with the whole pool as capacity;
  its prompts are the residents of the next slice, everybody else is paged
  out;
* inside a slice each iteration partitions the residents only, with their
  own blocks held and the pool's free blocks as capacity.

The page-out / page-in sets feed ``aqua_swap_out`` / ``aqua_swap_in``; the
swaps of one reschedule are issued together so that the library overlaps
them (section 7, "Efficient context switching").
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Sequence, Tuple

import numpy as np

from . import aqua


@dataclass
class Step:
    """One iteration's decision."""
    t: int
    resched: bool
    page_out: List[int] = field(default_factory=list)
    page_in: List[int] = field(default_factory=list)
    index: np.ndarray = None            # request ids, admission order
    tokens: np.ndarray = None           # tokens each computes

    def as_log(self, done: Sequence[int]) -> dict:
        return {"t": self.t, "resched": self.resched, "out": list(self.page_out),
                "in": list(self.page_in),
                "batch": [[int(i), int(x)] for i, x in zip(self.index, self.tokens)],
                "done": sorted(int(i) for i in done)}


class CfsScheduler:
    """Scheduler state for one KV pool of ``pool_blocks`` blocks."""

    def __init__(self, pool_blocks: int, block_tokens: int, batch_tokens: int,
                 decode_slots: int, k: int):
        if min(pool_blocks, block_tokens, batch_tokens, decode_slots, k) < 1:
            raise ValueError("pool_blocks, block_tokens, batch_tokens, decode_slots "
                             "and k must be positive")
        self.pool_blocks = pool_blocks
        self.T = block_tokens
        self.b = batch_tokens
        self.d = decode_slots
        self.k = k
        self.prompt = np.zeros(0, dtype=np.int64)
        self.computed = np.zeros(0, dtype=np.int64)
        self.generated = np.zeros(0, dtype=np.int64)
        self.arrival = np.zeros(0, dtype=np.int64)
        self.live = np.zeros(0, dtype=bool)         # arrived or not, not completed
        self.resident = np.zeros(0, dtype=np.int64)  # ids, increasing
        self.since = 0
        self.pending = True
        self.partition_calls = 0

    # -- requests --------------------------------------------------------
    def add(self, prompt_tokens: int, arrival: int = 0) -> int:
        if prompt_tokens < 1:
            raise ValueError("empty prompt")
        if -(-prompt_tokens // self.T) > self.pool_blocks:
            raise ValueError("prompt larger than the pool")
        rid = len(self.prompt)
        self.prompt = np.append(self.prompt, prompt_tokens)
        self.computed = np.append(self.computed, 0)
        self.generated = np.append(self.generated, 0)
        self.arrival = np.append(self.arrival, arrival)
        self.live = np.append(self.live, True)
        return rid

    def blocks(self, ids) -> np.ndarray:
        ids = np.asarray(ids, dtype=np.int64)
        return -(-(self.computed[ids] + self.generated[ids]) // self.T)

    def _partition(self, ids: np.ndarray, held: np.ndarray, capacity: int):
        req = np.stack([self.prompt[ids], self.computed[ids], self.generated[ids], held],
                       axis=1).astype(np.uint32)
        self.partition_calls += 1
        j, x, _ = aqua.cfs_partition(req, self.b, self.d, capacity, self.T)
        return ids[j.astype(np.int64)], x.astype(np.int64)

    # -- one iteration ---------------------------------------------------
    def next_arrival(self) -> int:
        waiting = self.arrival[self.live]
        return int(waiting.min()) if len(waiting) else -1

    def step(self, now: int) -> Step:
        """The batch of iteration ``now`` (None when nothing has arrived)."""
        cands = np.flatnonzero(self.live & (self.arrival <= now))
        if len(cands) == 0:
            self.pending = True
            return None
        if not self.pending:
            held = self.blocks(self.resident)
            idx, tok = self._partition(self.resident, held, self.pool_blocks - int(held.sum()))
            if len(idx):
                return Step(now, False, index=idx, tokens=tok)
            self.pending = True          # no resident can grow: re-form now
        idx, tok = self._partition(cands, np.zeros(len(cands), dtype=np.int64),
                                   self.pool_blocks)
        if len(idx) == 0:
            # Only a prompt whose context no longer fits the whole pool can
            # block every admission; the engine must bound context lengths.
            raise RuntimeError("no request fits the pool: a context has outgrown it")
        members = np.sort(idx)
        out = np.setdiff1d(self.resident, members, assume_unique=True)
        inn = np.setdiff1d(members, self.resident, assume_unique=True)
        self.resident = members
        self.pending = False
        self.since = 0
        return Step(now, True, [int(i) for i in out], [int(i) for i in inn], idx, tok)

    def advance(self, st: Step, completed: Sequence[int]) -> None:
        """Record that ``st`` ran; ``completed`` produced their last token."""
        pre = self.computed[st.index] < self.prompt[st.index]
        self.computed[st.index[pre]] += st.tokens[pre]
        self.generated[st.index[~pre]] += 1
        if len(completed):
            done = np.asarray(completed, dtype=np.int64)
            self.live[done] = False
            self.resident = self.resident[~np.isin(self.resident, done)]
            self.pending = True
        self.since += 1
        if self.since >= self.k:
            self.pending = True


def run_trace(trace: Sequence[Tuple[int, int, int]], pool_blocks: int, block_tokens: int,
              batch_tokens: int, decode_slots: int, k: int):
    """Runs a synthetic trace of (arrival iteration, prompt tokens, output
    tokens) to completion; a request completes after its output tokens.
    Returns (log, scheduler): one log entry per executed iteration, with
    ``out``/``in`` the prompts paged out / in at a reschedule."""
    s = CfsScheduler(pool_blocks, block_tokens, batch_tokens, decode_slots, k)
    outputs = np.asarray([o for _, _, o in trace], dtype=np.int64)
    for a, p, o in trace:
        if o < 1 or -(-(p + o) // block_tokens) > pool_blocks:
            raise ValueError("each request needs at least one output token and must fit the pool")
        s.add(p, a)
    log = []
    now = 0
    while s.live.any():
        st = s.step(now)
        if st is None:
            now = s.next_arrival()
            continue
        dec = st.index[s.computed[st.index] >= s.prompt[st.index]]
        completed = dec[s.generated[dec] + 1 == outputs[dec]]
        s.advance(st, completed)
        log.append(st.as_log(completed))
        now += 1
    return log, s
