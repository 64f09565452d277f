"""Time-sliced preemption cycle on one GPU.

Every slice of a preemptive scheduler pages out the prompts that leave the
batch and pages in those that join it (Aqua, section 7: the batch is
rescheduled every k iterations or when a request completes).  Here each
slice issues one batched swap-out of the leaving prompts on one stream and
one batched swap-in of the joining prompts on a second stream, so the two
overlap; the library orders them only where a joining prompt reuses blocks
that a leaving prompt is still being read from.  The slice ends with
``aqua_sync`` and the caller's between-slice work.
"""
from __future__ import annotations

from typing import Callable, Optional

import numpy as np
import torch

from . import aqua
from .workload import Schedule


def slice_tables(sched: Schedule, s: int):
    """(out CSR, out image offsets, in CSR, in image offsets) of slice s."""
    sl = sched.slices[s]
    out = aqua._csr(sl.out_tables)
    out_off = np.asarray([sched.slot_offsets[p] for p in sl.out_prompts], dtype=np.uint64)
    inn = aqua._csr(sl.in_tables)
    in_off = np.asarray([sched.slot_offsets[p] for p in sl.in_prompts], dtype=np.uint64)
    return out, out_off, inn, in_off


def run_slices(pool: aqua.KVPool, region: torch.Tensor, sched: Schedule,
               first: int, count: int, out_stream, in_stream,
               between: Optional[Callable[[int], None]] = None,
               prepared=None) -> None:
    """Runs slices [first, first+count) of the schedule."""
    for s in range(first, first + count):
        out, out_off, inn, in_off = prepared[s] if prepared else slice_tables(sched, s)
        pool.swap_out(out, region, out_off, stream=out_stream)
        pool.swap_in(inn, region, in_off, stream=in_stream)
        pool.sync(0)
        if between is not None:
            between(s)
            # The caller's writes ran on its current stream: the next
            # slice's swaps must not start before them.
            cur = torch.cuda.current_stream()
            out_stream.wait_stream(cur)
            in_stream.wait_stream(cur)


def run_slices_in_space(pool: aqua.KVPool, space: aqua.SwapSpace, tensors: dict,
                        sched: Schedule, first: int, count: int, out_stream, in_stream,
                        between: Optional[Callable[[int], None]] = None) -> None:
    """Runs slices [first, first+count) with every prompt's image in its own
    swap-space tensor (``tensors``: prompt -> handle), wherever the tensor
    lives now (device region or host fallback).  One call per prompt, since
    the tensors of one slice may sit in different places."""
    for s in range(first, first + count):
        sl = sched.slices[s]
        for p, t in zip(sl.out_prompts, sl.out_tables):
            pool.swap_out([t], space.buffer(tensors[p]), stream=out_stream)
        for p, t in zip(sl.in_prompts, sl.in_tables):
            pool.swap_in([t], space.buffer(tensors[p]), stream=in_stream)
        pool.sync(0)
        if between is not None:
            between(s)
            cur = torch.cuda.current_stream()
            out_stream.wait_stream(cur)
            in_stream.wait_stream(cur)
