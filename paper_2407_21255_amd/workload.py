"""Seeded synthetic inputs for the KV page-swap path.

This module generates *inputs* only: pool contents, block tables, free lists,
image placements and the time-sliced preemption schedule.  It holds none of
the swap arithmetic, imports nothing else from this package, and serves both
the GPU path (tests, bench) and the CPU oracle.

Generator (counter based, identical on any device and thread count):

* ``mix`` is the SplitMix64 finaliser (Steele, Lea and Flood, "Fast
  splittable pseudorandom number generators", OOPSLA 2014).
* A host stream ``Rng(seed)`` is SplitMix64: state += 0x9E3779B97F4A7C15,
  output = mix(state).
* Every (layer, block) chunk carries a 64-bit key; a live or initial-image
  chunk is keyed by (prompt, layer, logical block) with tag 1, a free chunk
  by (layer, physical block) with tag 2:
  ``key = mix(mix(mix(mix(seed) ^ tag) ^ a) ^ l) ^ i``.
* Element k of a chunk draws ``u = mix(key ^ k)``.  fp16/bf16:
  ``x = (u >> 40) * 2**-23 - 1`` (exact in fp32, uniform in [-1, 1)), rounded
  to the 16-bit format by round-to-nearest-even.  fp8 e4m3: the byte
  ``u & 0xFF`` with the NaN codes (low seven bits all ones) moved to a
  neighbouring finite code by flipping bit 0.

The element functions are written with torch integer ops so that the same
code fills a host tensor for the oracle and a device tensor for the GPU.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
_C1 = 0xBF58476D1CE4E5B9
_C2 = 0x94D049BB133111EB

F16, BF16, FP8_E4M3 = 1, 2, 3
ELEM_BYTES = {F16: 2, BF16: 2, FP8_E4M3: 1}
DTYPE_NAME = {F16: "f16", BF16: "bf16", FP8_E4M3: "fp8_e4m3"}

TAG_LIVE = 1
TAG_FREE = 2
GUARD_BYTE = 0xCD        # guard bands around offload images
SENTINEL_BYTE = 0xEE     # pool chunks that are about to be overwritten
CONSUMED_BYTE = 0xA5     # offload slots whose image has been swapped back in


def mix(z: int) -> int:
    """SplitMix64 finaliser on a Python int (taken mod 2**64)."""
    z &= M64
    z = ((z ^ (z >> 30)) * _C1) & M64
    z = ((z ^ (z >> 27)) * _C2) & M64
    return z ^ (z >> 31)


class Rng:
    """SplitMix64 stream."""

    def __init__(self, seed: int):
        self.state = seed & M64

    def next(self) -> int:
        self.state = (self.state + GAMMA) & M64
        return mix(self.state)

    def below(self, m: int) -> int:
        """An integer in [0, m) (plain modulo reduction)."""
        return self.next() % m


def permutation(n: int, seed: int) -> List[int]:
    """Fisher-Yates shuffle of 0..n-1 driven by ``Rng(seed)``."""
    rng = Rng(seed)
    p = list(range(n))
    for i in range(n - 1, 0, -1):
        j = rng.below(i + 1)
        p[i], p[j] = p[j], p[i]
    return p


def chunk_key(seed: int, tag: int, a: int, layer: int, i: int) -> int:
    return mix(mix(mix(mix(seed) ^ tag) ^ a) ^ layer) ^ i


def _signed(v: int) -> int:
    v &= M64
    return v - (1 << 64) if v >= (1 << 63) else v


_S1, _S2 = _signed(_C1), _signed(_C2)


def mix_t(z: torch.Tensor) -> torch.Tensor:
    """SplitMix64 finaliser on an int64 tensor holding uint64 bit patterns.

    Right shifts are made logical by masking off the sign-extended bits;
    int64 multiplication wraps modulo 2**64 on both CPU and GPU."""
    z = z ^ ((z >> 30) & ((1 << 34) - 1))
    z = z * _S1
    z = z ^ ((z >> 27) & ((1 << 37) - 1))
    z = z * _S2
    return z ^ ((z >> 31) & ((1 << 33) - 1))


def chunk_values(keys: torch.Tensor, chunk_bytes: int, dtype: int) -> torch.Tensor:
    """Bytes of ``len(keys)`` chunks, shape [n, chunk_bytes] uint8, on keys' device."""
    e = ELEM_BYTES[dtype]
    n_el = chunk_bytes // e
    k = torch.arange(n_el, dtype=torch.int64, device=keys.device)
    u = mix_t(keys.reshape(-1, 1) ^ k.reshape(1, -1))
    if dtype == FP8_E4M3:
        b = u & 0xFF
        b = torch.where((b & 0x7F) == 0x7F, b ^ 1, b)
        return b.to(torch.uint8)
    x = ((u >> 40) & 0xFFFFFF).to(torch.float32) * (2.0 ** -23) - 1.0
    tdt = torch.float16 if dtype == F16 else torch.bfloat16
    return x.to(tdt).contiguous().view(torch.uint8).reshape(len(keys), chunk_bytes)


def fill_chunks(dst: torch.Tensor, keys: torch.Tensor, chunk_bytes: int,
                dtype: int, slab_bytes: int = 1 << 28) -> None:
    """Write generated chunks into ``dst`` ([n, chunk_bytes] uint8 view)."""
    n = dst.shape[0]
    per = max(1, slab_bytes // (chunk_bytes * 8 // ELEM_BYTES[dtype]))
    keys = keys.to(dst.device)
    for s in range(0, n, per):
        dst[s:s + per].copy_(chunk_values(keys[s:s + per], chunk_bytes, dtype))


# --------------------------------------------------------------------------
# Shapes

@dataclass(frozen=True)
class KVShape:
    num_layers: int
    num_blocks: int
    num_kv_heads: int
    block_tokens: int
    head_dim: int
    dtype: int

    @property
    def chunk_bytes(self) -> int:
        return 2 * self.num_kv_heads * self.block_tokens * self.head_dim * \
            ELEM_BYTES[self.dtype]

    @property
    def bytes_per_token(self) -> int:
        return self.num_layers * 2 * self.num_kv_heads * self.head_dim * \
            ELEM_BYTES[self.dtype]

    @property
    def pool_bytes(self) -> int:
        return self.num_layers * self.num_blocks * self.chunk_bytes

    def image_bytes(self, nblocks: int) -> int:
        return self.num_layers * nblocks * self.chunk_bytes

    def as_tuple(self):
        return (self.num_layers, self.num_blocks, self.num_kv_heads,
                self.block_tokens, self.head_dim, self.dtype)


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


# --------------------------------------------------------------------------
# Pool fills

def mix_np(z: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser on a uint64 numpy array (wrapping arithmetic)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(_C1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(_C2)
    return z ^ (z >> np.uint64(31))


def chunk_keys_np(seed: int, tag: int, a, layer, i) -> np.ndarray:
    """Vectorised ``chunk_key`` over broadcastable integer arrays."""
    base = np.uint64(mix(mix(seed) ^ tag))
    a = np.asarray(a, dtype=np.uint64)
    layer = np.asarray(layer, dtype=np.uint64)
    i = np.asarray(i, dtype=np.uint64)
    return mix_np(mix_np(base ^ a) ^ layer) ^ i


def pool_keys(shape: KVShape, seed: int, owner: Optional[dict] = None) -> torch.Tensor:
    """Key of every (layer, block) chunk, int64 [L*N] (layer-major).

    ``owner`` maps physical block -> (prompt, logical block) for live chunks;
    every other chunk is keyed as free."""
    L, N = shape.num_layers, shape.num_blocks
    lay = np.arange(L, dtype=np.uint64).reshape(L, 1)
    keys = chunk_keys_np(seed, TAG_FREE, 0, lay,
                         np.arange(N, dtype=np.uint64).reshape(1, N))
    if owner:
        b = np.fromiter(owner.keys(), dtype=np.int64, count=len(owner))
        pi = np.array(list(owner.values()), dtype=np.int64).reshape(-1, 2)
        keys[:, b] = chunk_keys_np(seed, TAG_LIVE, pi[:, 0].reshape(1, -1), lay,
                                   pi[:, 1].reshape(1, -1))
    return torch.from_numpy(np.ascontiguousarray(keys).reshape(-1).view(np.int64))


def image_keys(shape: KVShape, seed: int, prompt: int, nblocks: int) -> torch.Tensor:
    """Keys of an initial offload image of ``prompt``, layer-major [L*n]."""
    lay = np.arange(shape.num_layers, dtype=np.uint64).reshape(-1, 1)
    i = np.arange(nblocks, dtype=np.uint64).reshape(1, -1)
    keys = chunk_keys_np(seed, TAG_LIVE, prompt, lay, i)
    return torch.from_numpy(np.ascontiguousarray(keys).reshape(-1).view(np.int64))


def fill_pool(pool: torch.Tensor, shape: KVShape, seed: int,
              owner: Optional[dict] = None) -> None:
    """Fill a flat uint8 pool tensor (host or device) from the generator."""
    C = shape.chunk_bytes
    assert pool.dtype == torch.uint8 and pool.numel() >= shape.pool_bytes
    fill_chunks(pool[:shape.pool_bytes].view(-1, C),
                pool_keys(shape, seed, owner), C, shape.dtype)


# --------------------------------------------------------------------------
# Block tables

def alloc_round_robin(free: List[int], sizes: List[int]) -> List[List[int]]:
    """Take blocks from the head of ``free`` one at a time, cycling over the
    requests, until request r holds sizes[r] blocks (fragmented tables)."""
    tables: List[List[int]] = [[] for _ in sizes]
    need = list(sizes)
    pos = 0
    while any(need):
        for r in range(len(sizes)):
            if need[r]:
                tables[r].append(free[pos])
                pos += 1
                need[r] -= 1
    del free[:pos]
    return tables


def csr(tables: List[List[int]]):
    """(int32 ids, uint64 offsets) of a list of tables."""
    ids = np.asarray([b for t in tables for b in t], dtype=np.int32)
    offs = np.zeros(len(tables) + 1, dtype=np.uint64)
    if tables:
        offs[1:] = np.cumsum([len(t) for t in tables])
    return ids, offs


@dataclass
class SwapCase:
    """One swap-out / swap-in round: the tables of the preempted prompts,
    the fresh tables they are swapped back into, and the chunk owners."""
    name: str
    shape: KVShape
    seed: int
    out_tables: List[List[int]]
    in_tables: List[List[int]]
    owner: dict = field(default_factory=dict)

    @property
    def nblocks(self) -> int:
        return sum(len(t) for t in self.out_tables)

    @property
    def payload_bytes(self) -> int:
        return self.shape.image_bytes(self.nblocks)


# The five workloads.  Shapes follow the public Llama-3 8B and 70B
# configurations (32 / 80 layers, 8 KV heads, head_dim 128, grouped-query
# attention); KV bytes per token are then 128 KiB and 320 KiB in bf16.
TINY = KVShape(4, 256, 8, 16, 128, F16)
LLAMA8B = KVShape(32, 16384, 8, 16, 128, BF16)
LLAMA70B = KVShape(80, 4096, 8, 16, 128, BF16)
LLAMA8B_FP8 = KVShape(32, 16384, 8, 16, 128, FP8_E4M3)
# One tensor-parallel rank's share of the 70B pool: H/TP KV heads per rank.
LLAMA70B_TP2 = KVShape(80, 4096, 4, 16, 128, BF16)
LLAMA70B_TP4 = KVShape(80, 4096, 2, 16, 128, BF16)
# Yi-34B (public configuration: 60 layers, 8 KV heads, head_dim 128), bf16:
# 240 KiB of KV per token; an 8192-block pool holds 131072 tokens.
YI34B = KVShape(60, 8192, 8, 16, 128, BF16)


def tiny_case(seed: int = 1, shape: KVShape = TINY, nblocks: int = 32) -> SwapCase:
    """One 512-token prompt (32 blocks) drawn as a random subset of the pool,
    swapped back into a random subset of the complement."""
    perm = permutation(shape.num_blocks, seed)
    bt = perm[:nblocks]
    rest = perm[nblocks:]
    p2 = permutation(len(rest), seed + 1000)
    bt2 = [rest[j] for j in p2[:nblocks]]
    owner = {b: (0, i) for i, b in enumerate(bt)}
    return SwapCase("tiny", shape, seed, [bt], [bt2], owner)


def fragmented_case(name: str, shape: KVShape, seed: int, n_prompts: int,
                    blocks_per_prompt: int, n_preempt: int) -> SwapCase:
    """``n_prompts`` prompts allocated round-robin from a shuffled free list
    (fragmented tables); the first ``n_preempt`` are swapped out and then back
    into fresh blocks taken from the head of the free list."""
    free = permutation(shape.num_blocks, seed)
    tables = alloc_round_robin(free, [blocks_per_prompt] * n_prompts)
    owner = {b: (p, i) for p, t in enumerate(tables) for i, b in enumerate(t)}
    out_t = tables[:n_preempt]
    in_t = alloc_round_robin(free, [len(t) for t in out_t])
    return SwapCase(name, shape, seed, out_t, in_t, owner)


def llama8b_hbm_case(seed: int = 2, shape: KVShape = LLAMA8B) -> SwapCase:
    """16 prompts x 2048 tokens resident; 8 preempted to the HBM region."""
    return fragmented_case("llama8b_hbm", shape, seed, 16, 2048 // shape.block_tokens, 8)


def llama8b_host_case(seed: int = 3, shape: KVShape = LLAMA8B) -> SwapCase:
    """8 prompts x 4096 tokens preempted to pinned host memory."""
    return fragmented_case("llama8b_host", shape, seed, 8, 4096 // shape.block_tokens, 8)


def llama70b_case(seed: int = 4, shape: KVShape = LLAMA70B,
                  tokens: int = 32768) -> SwapCase:
    """One long prompt on a random block subset; swapped back into a random
    permutation of the complement."""
    n = tokens // shape.block_tokens
    perm = permutation(shape.num_blocks, seed)
    bt = perm[:n]
    rest = perm[n:]
    p2 = permutation(len(rest), seed + 1000)
    bt2 = [rest[j] for j in p2[:n]]
    owner = {b: (0, i) for i, b in enumerate(bt)}
    return SwapCase("llama70b", shape, seed, [bt], [bt2], owner)


def image_offsets(nblocks: List[int], shape: KVShape, guard: int = 4096):
    """Offsets of images placed one after another, each preceded and the last
    followed by ``guard`` bytes; returns (offsets, total bytes)."""
    offs, pos = [], guard
    for n in nblocks:
        offs.append(pos)
        pos += shape.image_bytes(n) + guard
    return offs, pos


# --------------------------------------------------------------------------
# Time-sliced preemption schedule (resident FIFO out, swapped FIFO in)

@dataclass
class Slice:
    index: int
    out_prompts: List[int]
    out_tables: List[List[int]]
    in_prompts: List[int]
    in_tables: List[List[int]]
    resident_after: List[int]       # resident prompts after the slice (FIFO order)
    tables_after: dict              # prompt -> table, for residents
    # Written by the compute of the slice's iterations, after its swaps:
    # (prompt, first logical block, new physical blocks), in order.
    grow: List[tuple] = field(default_factory=list)
    finished: List[int] = field(default_factory=list)   # blocks freed, no swap


@dataclass
class Schedule:
    shape: KVShape
    seed: int
    lengths: List[int]              # tokens per prompt
    nblocks: List[int]              # blocks per prompt
    slot_offsets: List[int]         # byte offset of each prompt's offload slot
    region_bytes: int
    initial_resident: List[int]
    initial_tables: dict            # prompt -> table
    slices: List[Slice]
    # Prompts whose generated image is in the region at the start (None:
    # every prompt that is not initially resident).
    initial_swapped: Optional[List[int]] = None

    def mutation(self, s: int, p: int) -> int:
        """64-bit word written twice at the start of the last logical block
        of resident prompt p, in layer s mod L, after slice s."""
        return mix(self.seed ^ (s << 32) ^ p)


def preemption_schedule(shape: KVShape = LLAMA8B_FP8, seed: int = 5,
                        n_prompts: int = 64, n_resident: int = 32,
                        per_slice: int = 16, n_slices: int = 100,
                        min_tokens: int = 128, max_tokens: int = 8192,
                        guard: int = 4096) -> Schedule:
    """Deterministic context-switch schedule.

    Each slice preempts the ``per_slice`` longest-resident prompts and resumes
    the ``per_slice`` longest-waiting ones (time slices of equal cost make the
    least-served-first rule a FIFO).  Freed blocks go to the tail of a free
    list that starts as a shuffled permutation; resumed prompts take blocks
    from its head round-robin.  Every prompt owns a fixed offload slot."""
    rng = Rng(mix(seed ^ 0x5EED))
    lengths = [min_tokens + rng.below(max_tokens - min_tokens + 1)
               for _ in range(n_prompts)]
    nblocks = [ceil_div(t, shape.block_tokens) for t in lengths]
    slot_offsets, region = image_offsets(nblocks, shape, guard)
    free = permutation(shape.num_blocks, seed)
    resident = list(range(n_resident))
    swapped = list(range(n_resident, n_prompts))
    if sum(nblocks[p] for p in resident) > shape.num_blocks:
        raise ValueError("initial resident set does not fit the pool")
    init = alloc_round_robin(free, [nblocks[p] for p in resident])
    tables = {p: t for p, t in zip(resident, init)}
    initial_tables = {p: list(t) for p, t in tables.items()}
    slices = []
    for s in range(n_slices):
        outs = resident[:per_slice]
        ins = swapped[:per_slice]
        out_tables = [tables.pop(p) for p in outs]
        for t in out_tables:
            free.extend(t)
        in_tables = alloc_round_robin(free, [nblocks[p] for p in ins])
        for p, t in zip(ins, in_tables):
            tables[p] = t
        resident = resident[per_slice:] + ins
        swapped = swapped[per_slice:] + outs
        slices.append(Slice(s, outs, out_tables, ins, in_tables, list(resident),
                            {p: list(t) for p, t in tables.items()}))
    return Schedule(shape, seed, lengths, nblocks, slot_offsets, region,
                    list(range(n_resident)), initial_tables, slices)


def mutation_writes(sched: Schedule, s: int):
    """Host writes after slice s, so that a stale image cannot pass as a
    fresh one: (pool byte offsets, 16-byte payloads) for every resident
    prompt -- two copies of a 64-bit word at the start of its last logical
    block in layer s mod L -- and the offload slots just swapped back in,
    which are overwritten with CONSUMED_BYTE: [(offset, length)]."""
    sh = sched.shape
    C = sh.chunk_bytes
    l = s % sh.num_layers
    sl = sched.slices[s]
    offs, words = [], []
    for p in sl.resident_after:
        if not sl.tables_after[p]:
            continue
        b = sl.tables_after[p][-1]
        offs.append((l * sh.num_blocks + b) * C)
        w = sched.mutation(s, p)
        words.append(np.frombuffer(w.to_bytes(8, "little") * 2, dtype=np.uint8))
    slots = [(sched.slot_offsets[p], sh.image_bytes(len(t)))
             for p, t in zip(sl.in_prompts, sl.in_tables)]
    return (np.asarray(offs, dtype=np.int64),
            np.stack(words) if words else np.zeros((0, 16), np.uint8), slots)


def apply_growth(pool: torch.Tensor, sched: Schedule, s: int) -> None:
    """The KV that slice s's iterations compute: every new block of a
    resident prompt, all layers, keyed as live chunk (prompt, layer,
    logical block).  ``pool`` is the flat uint8 pool (host or device)."""
    sh = sched.shape
    L, N, C = sh.num_layers, sh.num_blocks, sh.chunk_bytes
    P = pool[:sh.pool_bytes].view(L, N, C)
    lay = np.arange(L, dtype=np.uint64).reshape(L, 1)
    step = max(1, (64 << 20) // (L * C))          # bounds the temporaries
    for p, first, blocks in sched.slices[s].grow:
        for j in range(0, len(blocks), step):
            part = blocks[j:j + step]
            i = np.arange(first + j, first + j + len(part), dtype=np.uint64).reshape(1, -1)
            keys = torch.from_numpy(np.ascontiguousarray(
                chunk_keys_np(sched.seed, TAG_LIVE, p, lay, i)).reshape(-1).view(np.int64))
            vals = chunk_values(keys.to(pool.device), C, sh.dtype).view(L, len(part), C)
            P[:, torch.as_tensor(part, dtype=torch.long, device=pool.device)] = vals


def fill_region(region: torch.Tensor, sched: Schedule) -> None:
    """Offload region of a preemption schedule: guard bytes everywhere, and
    the generated initial images of the prompts that start swapped out."""
    region.fill_(GUARD_BYTE)
    sh = sched.shape
    C = sh.chunk_bytes
    swapped = sched.initial_swapped
    if swapped is None:
        swapped = [p for p in range(len(sched.nblocks)) if p not in sched.initial_resident]
    for p in swapped:
        o, n = sched.slot_offsets[p], sched.nblocks[p]
        fill_chunks(region[o:o + sh.image_bytes(n)].view(-1, C),
                    image_keys(sh, sched.seed, p, n), C, sh.dtype)


def schedule_owner(sched: Schedule) -> dict:
    """Physical block -> (prompt, logical block) of the initial residents."""
    return {b: (p, i) for p, t in sched.initial_tables.items() for i, b in enumerate(t)}


# --------------------------------------------------------------------------
# Fair-scheduling traces and the swap schedules they produce

def burst_trace(seed: int, n: int, burst: int, gap: int, prompt_range, output_range):
    """Synthetic serving burst: ``burst`` requests at iteration 0, then one
    every ``gap`` iterations; prompt and output lengths uniform in the
    closed ranges.  Returns [(arrival, prompt tokens, output tokens)]."""
    rng = Rng(mix(seed ^ 0xC0F5))
    out = []
    for r in range(n):
        a = 0 if r < burst else (r - burst + 1) * gap
        p = prompt_range[0] + rng.below(prompt_range[1] - prompt_range[0] + 1)
        o = output_range[0] + rng.below(output_range[1] - output_range[0] + 1)
        out.append((a, p, o))
    return out


def cfs_swap_schedule(shape: KVShape, seed: int, trace, log, guard: int = 4096) -> Schedule:
    """Block-level swap schedule of a rescheduler run.

    ``log`` has one entry per iteration (``resched``, ``out``, ``in``,
    ``batch``, ``done``).  Each reschedule opens a slice: the prompts paged
    out are swapped out from their tables into their slots and their blocks
    go to the tail of the free list (a seeded permutation at the start);
    the prompts paged in that have an image get fresh blocks from its head,
    round-robin.  The slice's iterations then grow the residents' tables as
    their tokens need blocks, and completed prompts free theirs.  Slot p
    holds prompt p's largest image (prompt plus output tokens)."""
    T = shape.block_tokens
    lengths = [p + o for _, p, o in trace]
    nblocks = [ceil_div(x, T) for x in lengths]
    slot_offsets, region = image_offsets(nblocks, shape, guard)
    free = permutation(shape.num_blocks, seed)
    ctx = [0] * len(trace)
    tables: dict = {}
    image = {}                       # prompt -> blocks in its offload image
    slices: List[Slice] = []
    for e in log:
        if e["resched"]:
            outs, out_t = [], []
            for p in e["out"]:
                t = tables.pop(p)
                if t:
                    outs.append(p)
                    out_t.append(t)
                    free.extend(t)
                image[p] = len(t)
            ins = [p for p in e["in"] if image.get(p, 0) > 0]
            in_t = alloc_round_robin(free, [image[p] for p in ins])
            for p in e["in"]:
                tables[p] = []
            for p, t in zip(ins, in_t):
                tables[p] = t
            slices.append(Slice(len(slices), outs, out_t, ins, in_t, [], {}))
        sl = slices[-1]
        for p, x in e["batch"]:
            ctx[p] += x if ctx[p] < trace[p][1] else 1
            need = ceil_div(ctx[p], T) - len(tables[p])
            if need > 0:
                new = free[:need]
                del free[:need]
                sl.grow.append((p, len(tables[p]), new))
                tables[p] = tables[p] + new
        for p in e["done"]:
            free.extend(tables.pop(p))
            sl.finished.append(p)
        sl.resident_after = sorted(tables)
        sl.tables_after = {p: list(t) for p, t in tables.items()}
    return Schedule(shape, seed, lengths, nblocks, slot_offsets, region, [], {}, slices, [])


@dataclass
class CfsConfig:
    """A fair-scheduling workload: pool shape, burst trace and scheduler
    settings.  ``decode_slots`` -- the number of prompts that fit in the
    pool -- is the pool's blocks over the blocks of a mean-length request."""
    name: str
    shape: KVShape
    seed: int
    n: int
    burst: int
    gap: int
    prompt_range: tuple
    output_range: tuple
    batch_tokens: int
    k: int

    def trace(self):
        return burst_trace(self.seed, self.n, self.burst, self.gap, self.prompt_range,
                           self.output_range)

    def decode_slots(self, trace=None) -> int:
        tr = self.trace() if trace is None else trace
        total = sum(p + o for _, p, o in tr)
        mean_blocks = ceil_div(total, len(tr) * self.shape.block_tokens)
        return max(1, self.shape.num_blocks // mean_blocks)


# Small enough for a whole-schedule oracle replay: 48 requests on a
# 1024-block pool of 8 KiB chunks, about 4x oversubscribed.
CFS_SMALL = CfsConfig("small", KVShape(4, 1024, 2, 16, 64, BF16), 11, 48, 24, 2,
                      (64, 1024), (64, 512), 1024, 8)
# Llama-3-8B-shaped pool (32 GiB); 192 requests, 96 at once then one every
# second iteration, prompts 512-4096 and outputs 512-2048 tokens, 8192-token
# iterations, rescheduled every 16 iterations: the pool is about 2x
# oversubscribed at the peak.
CFS_LLAMA8B = CfsConfig("llama8b", LLAMA8B, 7, 192, 96, 2, (512, 4096), (512, 2048), 8192, 16)
