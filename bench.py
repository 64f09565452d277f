"""KV page-swap throughput on one MI355X.

A step is one context switch of the hot path: a batched swap-out (gather)
of the preempted prompts' KV blocks into the offload image, then a batched
swap-in (scatter) of that image into fresh pool blocks -- validation, run
planning, cross-stream ordering, both kernels and completion.  Steps
alternate between two disjoint block sets, so every step moves the whole
payload both ways.  The pool and the offload buffer are resident (HBM, or
pinned host for the host-target workloads) before the timed region starts.

Prints one JSON line.  The default workload is the largest single-GPU
configuration: the Llama-3-70B-shaped pool (80 layers, 8 KV heads, head_dim
128, block 16, bf16, 4096 blocks) with one 32768-token prompt (10 GiB each
way) preempted to an HBM offload region, the long-prompt regime.
"""
from __future__ import annotations

import argparse
import contextlib
import ctypes
import gc
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, read + write combined
HIP_MEMCPY_D2D_NO_CU = 1024  # hipMemcpyDeviceToDeviceNoCU: a copy engine, no compute units
HOST_LINK_PEAK_GBS = 63.0    # PCIe 5.0 x16, one direction, after encoding

# HBM bytes per launch of the dominant kernel from rocprofv3 --pmc
# (FETCH_SIZE, WRITE_SIZE), each scaled by the same counters' reading for a
# plain copy of known size (a call split into several launches: per launch).  Keyed by _kernel_hash(): a change to the kernels
# or to how they are launched reports null until measured again.
# Recorded with the profile summary of the same kernel under profiles/.
MEASURED_TRAFFIC = {
    ("llama70b_hbm", "13417f258857070b"): {
        "gather (swap-out)": 21478084809, "scatter (swap-in)": 21476892772},
    ("llama8b_hbm", "13417f258857070b"): {
        "gather (swap-out)": 4296124199, "scatter (swap-in)": 4295530800},
    ("llama70b_tp2_hbm", "13417f258857070b"): {
        "gather (swap-out)": 10739621776, "scatter (swap-in)": 10739296865},
    ("llama70b_tp4_hbm", "13417f258857070b"): {
        "gather (swap-out)": 5369594663, "scatter (swap-in)": 5369299960},
    ("llama8b_fp8_hbm", "13417f258857070b"): {
        "gather (swap-out)": 2148315120, "scatter (swap-in)": 2149326387},
}

# Every source that decides what the swap kernels do and how they are
# launched: the kernels, the per-launch store rule, the workgroup size and
# grid rules, the run planning (unit size) and the launch set-up.
KERNEL_SOURCES = ("swap_kernels.hip", "swap_kernels.h", "aqua_core.h", "aqua_core.cpp",
                  "aqua_capi.hip")
# Run-time settings that change the launches.
KERNEL_ENV = ("AQUA_UNIT_BYTES", "AQUA_RING_BYTES", "AQUA_STAGE_SLOT_BYTES")


def _kernel_hash(root: str = ROOT, max_workgroups: int = 0) -> str:
    """Hash of the launch-defining sources and settings (16 hex digits)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        h.update(name.encode() + b"\0")
        h.update(open(os.path.join(root, "paper_2407_21255_amd", "csrc", name), "rb").read())
    for name in KERNEL_ENV:
        h.update(f"{name}={os.environ.get(name, '')}\0".encode())
    h.update(f"max_workgroups={max_workgroups}".encode())
    return h.hexdigest()[:16]


WORKLOADS = {
    "llama8b_hbm": "Llama-3-8B-shaped KV (32 layers, 8 KV heads, head_dim 128, block 16, "
                   "bf16, 16384-block pool): 8 of 16 fragmented 2048-token prompts "
                   "swapped out to an HBM offload region and back into fresh blocks",
    "llama8b_host": "Llama-3-8B-shaped KV, bf16: 8 x 4096-token prompts swapped out to "
                    "pinned host memory (zero copy) and back",
    "llama70b_hbm": "Llama-3-70B-shaped KV (80 layers, bf16, 4096-block pool): one "
                    "32768-token prompt swapped out to an HBM offload region and back",
    "llama70b_host": "Llama-3-70B-shaped KV, bf16: one 32768-token prompt swapped out to "
                     "pinned host memory and back",
    "llama70b_tp2_hbm": "one tensor-parallel rank of a TP2 Llama-3-70B (80 layers, 4 KV heads, "
                        "bf16, 32 KiB chunks, 4096-block pool): one 32768-token prompt "
                        "swapped out to an HBM offload region and back",
    "llama70b_tp4_hbm": "one tensor-parallel rank of a TP4 Llama-3-70B (80 layers, 2 KV heads, "
                        "bf16, 16 KiB chunks, 4096-block pool): one 32768-token prompt "
                        "swapped out to an HBM offload region and back",
    "llama8b_fp8_hbm": "Llama-3-8B-shaped fp8 e4m3 KV (32 KiB chunks, 16384-block pool): 8 of "
                       "16 fragmented 2048-token prompts swapped out to an HBM offload region "
                       "and back into fresh blocks",
    "tiny": "4 layers, 8 KV heads, head_dim 128, block 16, fp16, 256-block pool: one "
            "512-token prompt out to an HBM buffer and back",
    "prefix": "prefill caching on a Yi-34B-shaped pool (60 layers, 8 KV heads, head_dim 128, "
              "bf16, 8192 blocks): the KV of a 100000-token prompt is cached once in an HBM "
              "region; each step swaps its prefix (all but the last 256 tokens) back in "
              "from the cached image",
    "prefix_host": "the same prefix cache held in pinned host memory",
    "prefix_mixed": "the same prefix loaded (from HBM) once per ten iterations of other swap "
                    "traffic on the same pool: two prompts of 448 blocks swapped out and back "
                    "into another block set each iteration, on two more streams",
    "layered": "Llama-3-70B-shaped KV, one 32768-token prompt swapped in from an HBM region "
               "in 10 layer groups of 8, one ticket each",
    "layered_host": "the same layer-group swap-in from pinned host memory",
    "migrate": "Llama-3-70B-shaped KV: the 10 GiB image of one 32768-token prompt migrated "
               "from the HBM region to pinned host memory and back",
    "elastic": "the first 30 reschedules of the fair-scheduling burst with every prompt's "
               "image in its own swap-space tensor (58 prompts, 25.3 GB): reschedules 0-19 "
               "with the tensors in the device region, then the region reclaimed (tensors "
               "moved to pinned host memory), reschedules 20-24 over the host link, the "
               "region restored, reschedules 25-29",
    "cfs": "fair scheduling (least-served first, rescheduled every 16 iterations or on a "
           "completion) of a 192-request burst on a Llama-3-8B-shaped bf16 pool (16384 "
           "blocks, 2x oversubscribed): each reschedule swaps the prompts leaving the batch "
           "out and those rejoining it in",
    "cycle_host": "the preemption cycle with pinned host memory as swap space: each slice "
                  "swaps 16 prompts out to host memory on one stream and 16 in on another",
    "sizes": "swap rate against payload size on the Llama-3-8B-shaped bf16 pool (64 KiB "
             "chunks, 2 MiB per block over 32 layers): one fragmented prompt of 2 to 2048 blocks "
             "(4 MiB to 4 GiB) out to an HBM region and back, and to pinned host memory and "
             "back, beside one runtime copy of the same bytes and one runtime copy per chunk",
    "cycle": "time-sliced preemption on a Llama-3-8B-shaped fp8 e4m3 pool (16384 blocks): "
             "64 prompts of 128..8192 tokens, each slice swaps the 16 longest-resident out "
             "on one stream and the 16 longest-waiting in on another",
}


def _case(name):
    from paper_2407_21255_amd import workload as wl
    return {
        "llama8b_hbm": lambda: (wl.llama8b_hbm_case(), False),
        "llama8b_host": lambda: (wl.llama8b_host_case(), True),
        "llama70b_hbm": lambda: (wl.llama70b_case(), False),
        "llama70b_host": lambda: (wl.llama70b_case(), True),
        "llama70b_tp2_hbm": lambda: (wl.llama70b_case(shape=wl.LLAMA70B_TP2), False),
        "llama70b_tp4_hbm": lambda: (wl.llama70b_case(shape=wl.LLAMA70B_TP4), False),
        "llama8b_fp8_hbm": lambda: (wl.llama8b_hbm_case(shape=wl.LLAMA8B_FP8), False),
        "tiny": lambda: (wl.tiny_case(), False),
    }[name]()


def cpu_baseline(shape, target_seconds: float):
    """The CPU oracle on a bounded sample of the same workload: the same
    chunk shape on a 512-block pool, one 128-block (2048-token) prompt out
    to a host image and back into other blocks, repeated for
    ``target_seconds``; single thread."""
    import numpy as np

    import oracle
    from paper_2407_21255_amd import workload as wl

    L, H, T, D, dt = (shape.num_layers, shape.num_kv_heads, shape.block_tokens,
                      shape.head_dim, shape.dtype)
    small = wl.KVShape(L, 512, H, T, D, dt)
    d = oracle.desc(*small.as_tuple())
    rng = np.random.default_rng(2)
    pool = rng.integers(0, 256, size=small.pool_bytes, dtype=np.uint8)
    perm = wl.permutation(512, 2)
    a, b = perm[:128], perm[128:256]
    img = np.zeros(small.image_bytes(128), dtype=np.uint8)
    assert oracle.swap_out(d, pool, [a], img) == 0  # touch every page once
    assert oracle.swap_in(d, pool, [b], img) == 0
    # One core for the timing (this thread only), restored afterwards.
    try:
        prev = os.sched_getaffinity(0)
        os.sched_setaffinity(0, {min(prev)})
        pinned = f"pinned to core {min(prev)}"
    except (AttributeError, OSError):
        prev, pinned = None, "not pinned"
    reps, moved = 0, 0
    try:
        t0 = time.perf_counter()
        while True:
            src, dst = (a, b) if reps % 2 == 0 else (b, a)
            assert oracle.swap_out(d, pool, [src], img) == 0
            assert oracle.swap_in(d, pool, [dst], img) == 0
            reps += 1
            moved += 2 * img.nbytes
            el = time.perf_counter() - t0
            if el >= target_seconds:
                break
    finally:
        if prev is not None:
            os.sched_setaffinity(0, prev)
    return {
        "value": round(moved / el / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
        "sample": f"{L}-layer chunks of {small.chunk_bytes} B on a 512-block pool: one "
                  f"128-block prompt ({img.nbytes >> 20} MiB per direction) out and back in, "
                  f"{reps} round trips in {el:.1f} s, single thread {pinned}",
    }


def gemm_run(stream, a, iters, per_kernel=True):
    """Enqueues ``iters`` 4096^3 bf16 GEMMs on ``stream``; returns the event
    pairs bracketing each GEMM (or the whole run)."""
    import torch
    evs = []
    with torch.cuda.stream(stream):
        if not per_kernel:
            e0 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
        for _ in range(iters):
            if per_kernel:
                e0 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
            c = a @ a
            if per_kernel:
                e1 = torch.cuda.Event(enable_timing=True)
                e1.record(stream)
                evs.append((e0, e1))
        if not per_kernel:
            e1 = torch.cuda.Event(enable_timing=True)
            e1.record(stream)
            evs.append((e0, e1))
    del c
    return evs


class GemmCompanion:
    """4096^3 bf16 GEMMs on a compute stream beside the timed steps: about
    one step's worth per step (estimated from the warm-up), first timed
    alone, after a warm-up, so that both figures cover the same span of
    sustained work."""

    def __init__(self, step_s, steps):
        import torch
        self.comp = torch.cuda.Stream()
        self.a = torch.randn(4096, 4096, device="cuda", dtype=torch.bfloat16)
        gemm_run(self.comp, self.a, 20)
        torch.cuda.synchronize()
        est = gemm_run(self.comp, self.a, 20, per_kernel=False)
        torch.cuda.synchronize()
        self.per_step = max(1, int(step_s * 1e3 / (gemm_ms(est) / 20)))
        self.n = self.per_step * steps
        alone = gemm_run(self.comp, self.a, self.n)
        torch.cuda.synchronize()
        self.alone_ms = gemm_ms(alone)
        self.during = []

    def step(self):
        self.during += gemm_run(self.comp, self.a, self.per_step)

    def result(self):
        # Kernel time of each GEMM alone and while the swaps run (gaps in the
        # compute stream are not counted).
        during_ms = gemm_ms(self.during)
        return {"gemm_ms_alone": round(self.alone_ms, 4),
                "gemm_ms_during_swaps": round(during_ms, 4), "gemm_iters": self.n,
                "slowdown": round(during_ms / self.alone_ms - 1, 4)}


def gemm_ms(evs):
    return sum(x.elapsed_time(y) for x, y in evs) / len(evs)


def run_pair(args, res_common):
    """Steps of (swap-out of the preempted prompts, swap-in into fresh blocks)."""
    import numpy as np
    import torch

    from paper_2407_21255_amd import aqua
    from paper_2407_21255_amd import workload as wl

    case, pinned = _case(args.workload)
    s = case.shape
    pool = torch.empty(s.pool_bytes, dtype=torch.uint8, device="cuda")
    wl.fill_pool(pool, s, case.seed, case.owner)
    payload = case.payload_bytes
    if pinned:
        img = torch.empty(payload, dtype=torch.uint8, pin_memory=True)
    else:
        img = torch.empty(payload, dtype=torch.uint8, device="cuda")
    img.zero_()
    if args.copy_reference and not pinned:
        # A plain device-to-device copy of the payload size, for scaling the
        # HBM traffic counters of the swap kernels.
        img.copy_(pool[:payload])
    torch.cuda.synchronize()

    tab_a = aqua._csr(case.out_tables)
    tab_b = aqua._csr(case.in_tables)
    stream = torch.cuda.Stream()
    kv = aqua.KVPool(s.as_tuple(), pool)
    if args.max_workgroups:
        kv.set_max_workgroups(aqua.AQUA_TARGET_HOST if pinned else aqua.AQUA_TARGET_DEVICE,
                              args.max_workgroups)
    if pinned:
        _configure_host(kv, args.host_path)
    evs = []
    two_step = args.two_step if not pinned else None
    if two_step:
        # The paper's scheme as an ablation: gather into a temporary HBM
        # tensor, then one bulk copy into the offload region, and the reverse
        # on swap-in.  The bulk copy is the runtime's own device-to-device
        # copy, on its blit kernel or (NoCU) on a copy engine.
        temp = torch.empty(payload, dtype=torch.uint8, device="cuda")
        hip = ctypes.CDLL("libamdhip64.so.7")
        hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_int, ctypes.c_void_p]

        def bulk(dst_t, src_t):
            if two_step == "blit":
                with torch.cuda.stream(stream):
                    dst_t.copy_(src_t)
            else:
                assert hip.hipMemcpyAsync(dst_t.data_ptr(), src_t.data_ptr(), payload,
                                          HIP_MEMCPY_D2D_NO_CU, stream.cuda_stream) == 0

    def step(i, timed):
        src, dst = (tab_a, tab_b) if i % 2 == 0 else (tab_b, tab_a)
        if timed:
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            e0.record(stream)
        if two_step:
            kv.swap_out(src, temp, stream=stream)
            bulk(img, temp)
        else:
            kv.swap_out(src, img, stream=stream)
        if timed:
            e1.record(stream)
        if two_step:
            bulk(temp, img)
            kv.swap_in(dst, temp, stream=stream)
        else:
            kv.swap_in(dst, img, stream=stream)
        if timed:
            e2.record(stream)
            evs.append((e0, e1, e2))

    gemm = None
    for i in range(args.warmup):
        if i == 1:
            kv.sync(0)
            tw = time.perf_counter()
        step(i, False)
    kv.sync(0)
    torch.cuda.synchronize()
    step_s = (time.perf_counter() - tw) / (args.warmup - 1) if args.warmup > 1 else 0.0
    # GEMMs enqueued step by step beside the swaps, so that both streams
    # start together.
    comp = GemmCompanion(step_s, args.steps) if args.gemm else None
    with _no_gc():
        t0 = time.perf_counter()
        st0 = kv.stats()
        for i in range(args.steps):
            if comp:
                comp.step()
            step(args.warmup + i, True)
        kv.sync(0)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    st = _since(kv.stats(), st0)
    carrier = ([kv.link_engine(0), kv.link_engine(1)]
               if pinned and args.host_path == "staged" else None)
    kv.close()
    if comp:
        gemm = comp.result()

    out_ms = np.array([a.elapsed_time(b) for a, b, _ in evs])
    in_ms = np.array([b.elapsed_time(c) for _, b, c in evs])
    value = 2 * payload * args.steps / wall / 1e9
    dom, dom_ms = ("gather (swap-out)", out_ms) if out_ms.mean() >= in_ms.mean() else \
        ("scatter (swap-in)", in_ms)
    if pinned:
        bound, peak, alg = "host_link", HOST_LINK_PEAK_GBS, payload
    elif two_step:
        # Gather and bulk copy each read and write the payload once.
        bound, peak, alg = "hbm", HBM_PEAK_GBS, 4 * payload
    else:
        bound, peak, alg = "hbm", HBM_PEAK_GBS, 2 * payload
    achieved = alg / (dom_ms.mean() * 1e-3) / 1e9
    # A call may be carried by several launches of the kernel (whole layers
    # each); the roofline is stated per launch, as a kernel trace lists it.
    calls = max(1, st["calls_out"] + st["calls_in"])
    per_call = st["launches"] / calls
    khash = _kernel_hash(max_workgroups=args.max_workgroups)
    res = dict(res_common)
    res.update({
        "value": round(value, 2),
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "dtype": wl.DTYPE_NAME[s.dtype],
        "config": {
            "workload": WORKLOADS[args.workload],
            "layers": s.num_layers, "kv_heads": s.num_kv_heads, "head_dim": s.head_dim,
            "block_tokens": s.block_tokens, "pool_blocks": s.num_blocks,
            "chunk_bytes": s.chunk_bytes, "swapped_blocks": case.nblocks,
            "payload_bytes_per_direction": payload,
            "offload_target": "pinned_host" if pinned else "hbm",
            "host_path": args.host_path if pinned else None,
            "link_carrier": carrier,
            "two_step": two_step,
            "parallelism": "single_gpu",
        },
        "roofline": {
            "bound": bound, "kernel": dom,
            "achieved": round(achieved, 1), "peak": peak,
            "unit": "GB/s", "frac": round(achieved / peak, 4),
            "traffic": (None if two_step else
                        MEASURED_TRAFFIC.get((args.workload, khash), {}).get(dom)),
            "algorithmic_bytes_per_launch": round(alg / per_call) if per_call else alg,
            "launches_per_call": round(per_call, 3),
            "launch_ms_mean": round(float(dom_ms.mean()) / per_call, 4) if per_call else None,
        },
        "kernel_ms": {"swap_out_mean": round(float(out_ms.mean()), 4),
                      "swap_out_min": round(float(out_ms.min()), 4),
                      "swap_in_mean": round(float(in_ms.mean()), 4),
                      "swap_in_min": round(float(in_ms.min()), 4)},
        "swap_out_GBps": round(payload / (out_ms.mean() * 1e-3) / 1e9, 2),
        "swap_in_GBps": round(payload / (in_ms.mean() * 1e-3) / 1e9, 2),
        "host_us_per_call": round(st["host_ns"] / max(1, st["calls_out"] + st["calls_in"]) / 1e3,
                                  2),
        "host_wait_us_per_call": round(st["wait_ns"] / max(1, st["calls_out"] + st["calls_in"]) /
                                       1e3, 2),
        "kernel_source": khash,
    })
    if gemm:
        res["compute_stream"] = gemm
    if pinned:
        res["link_ceiling"] = link_ceiling()
        res["host_link_frac"] = {
            "swap_out": round(res["swap_out_GBps"] / HOST_LINK_PEAK_GBS, 4),
            "swap_in": round(res["swap_in_GBps"] / HOST_LINK_PEAK_GBS, 4),
            "swap_out_vs_copy_engine": round(res["swap_out_GBps"] / res["link_ceiling"]["d2h"], 4),
            "swap_in_vs_copy_engine": round(res["swap_in_GBps"] / res["link_ceiling"]["h2d"], 4),
        }
    elif not two_step:
        copy_gbs = runtime_copy_rate(img, pool[:payload])
        res["hbm_runtime_copy"] = {
            "GBps_traffic": copy_gbs,
            "swap_out_vs_runtime_copy": round(2 * res["swap_out_GBps"] / copy_gbs, 4),
            "swap_in_vs_runtime_copy": round(2 * res["swap_in_GBps"] / copy_gbs, 4),
        }
        res["hbm_ceiling"] = ceil = hbm_ceiling(img, pool[:payload])
        for ref in ("copy", "serial"):
            for d in ("out", "in"):
                ceil[f"swap_{d}_vs_{ref}"] = round(2 * res[f"swap_{d}_GBps"] /
                                                   ceil[f"{ref}_GBps"], 4)
    return res, s


def hbm_ceiling(dst, src, reps: int = 5) -> dict:
    """Same-run HBM yardsticks of the payload's size with the library's own
    copy loop (aqua_hbm_yardstick): a contiguous copy (GB/s of read + write
    traffic), a pure read and a pure write, each timed with HIP events on
    its launch stream after one untimed pass; each as a share of 8 TB/s.
    ``serial`` is the rate of reading the payload and then writing it, one
    after the other (2 * bytes over the sum of the read and write times):
    the rate of a copy in which the memory serves reads and writes in turn
    and never both at once."""
    import torch

    from paper_2407_21255_amd import aqua
    nbytes = src.numel()
    stream = torch.cuda.Stream()
    out = {"bytes": nbytes}
    for name, kind, traffic in (("copy", aqua.AQUA_YARDSTICK_COPY, 2 * nbytes),
                                ("read", aqua.AQUA_YARDSTICK_READ, nbytes),
                                ("write", aqua.AQUA_YARDSTICK_WRITE, nbytes)):
        aqua.hbm_yardstick(kind, dst, src, stream=stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            aqua.hbm_yardstick(kind, dst, src, stream=stream)
        e1.record(stream)
        stream.synchronize()
        gbs = traffic * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
        out[f"{name}_GBps"] = round(gbs, 1)
        out[f"{name}_frac"] = round(gbs / HBM_PEAK_GBS, 4)
    serial = 2.0 / (1.0 / out["read_GBps"] + 1.0 / out["write_GBps"])
    out["serial_GBps"] = round(serial, 1)
    out["serial_frac"] = round(serial / HBM_PEAK_GBS, 4)
    return out


def runtime_copy_rate(dst, src, reps: int = 5) -> float:
    """HBM traffic rate (read + write, GB/s) of the runtime's own contiguous
    device-to-device copy of the payload size (torch ``copy_``), timed with
    HIP events after one untimed copy: the same-run yardstick for the swap
    kernels' rates."""
    import torch
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        dst.copy_(src)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            dst.copy_(src)
        e1.record(stream)
    stream.synchronize()
    return round(2 * src.numel() * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)


def link_ceiling(nbytes: int = 1 << 30, reps: int = 5):
    """GB/s of the runtime's copies over the host link: plain 1 GiB copies
    between pinned host memory and the device (hipMemcpyAsync), each
    direction alone, then both at once (total)."""
    import torch
    h = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    h.fill_(1)
    d.fill_(2)
    torch.cuda.synchronize()
    out = {}
    for name, dst, src in (("h2d", d, h), ("d2h", h, d)):
        dst.copy_(src, non_blocking=True)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            dst.copy_(src, non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
        out[name] = round(nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9, 2)
    # Both directions at once, on two streams: the link's rate when it is
    # busy both ways.
    h2 = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    d2 = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        with torch.cuda.stream(s1):
            h.copy_(d, non_blocking=True)
        with torch.cuda.stream(s2):
            d2.copy_(h2, non_blocking=True)
    torch.cuda.synchronize()
    out["both_total"] = round(2 * nbytes * reps / (time.perf_counter() - t0) / 1e9, 2)
    out["pcie"] = pcie_link()
    return out


def pcie_link():
    """The trained PCIe link of the (single) AMD GPU, from sysfs, e.g.
    "32.0 GT/s PCIe x16"; None where sysfs does not say."""
    import glob
    for dev in sorted(glob.glob("/sys/class/drm/card*/device")):
        try:
            if open(os.path.join(dev, "vendor")).read().strip() != "0x1002":
                continue
            speed = open(os.path.join(dev, "current_link_speed")).read().strip()
            width = open(os.path.join(dev, "current_link_width")).read().strip()
            return f"{speed} x{width}"
        except OSError:
            continue
    return None


@contextlib.contextmanager
def _no_gc():
    """Python's cyclic collector paused over a timed region, after one
    collection: a full pass over a process that holds torch stalls the host
    for tens of milliseconds, long enough for the GPU to drain its queue and
    idle.  (The collector is Python's, not part of the measured path.)"""
    gc.collect()
    was = gc.isenabled()
    gc.disable()
    try:
        yield
    finally:
        if was:
            gc.enable()


def _since(after: dict, before: dict) -> dict:
    """Pool counters accumulated between two snapshots (the timed steps
    only: the first staged call of a direction also allocates its slots)."""
    return {k: (v - before[k] if k != "hip_error" else v) for k, v in after.items()}


LINK_ENGINE = {"auto": -2, "runtime": -1}
_link_request = "auto"


def _configure_link(kv):
    """Carrier of a pool's link copies (``--link-engine``): staged host swaps
    and migrations between HBM and host memory."""
    e = LINK_ENGINE.get(_link_request)
    e = int(_link_request) if e is None else e
    for direction in (0, 1):
        kv.set_link_engine(direction, e)


def _configure_host(kv, host_path):
    """Host path of a pool and the carrier of its link copies."""
    from paper_2407_21255_amd import aqua
    kv.set_host_path(aqua.AQUA_HOST_STAGED if host_path == "staged"
                     else aqua.AQUA_HOST_ZERO_COPY)
    _configure_link(kv)


def _time_slices(sched, pool, region, ids, warmup, host_path=None, streams=2, legs="both"):
    """Issues slices ``ids`` of a swap schedule (the first ``warmup`` of them
    untimed): out on one stream, in on another, ``aqua_sync`` at the end of
    each, as a scheduler's loop boundary does.  (Issued without it, slices
    stay correct -- the library orders reused blocks and slots -- but
    consecutive slices then contend for HBM.)  ``streams=1`` issues both
    calls on one stream, one after the other; ``legs`` "out" or "in" issues
    only that direction of every slice (a breakdown of the slice's time, not
    the workload itself)."""
    import numpy as np
    import torch

    from paper_2407_21255_amd import aqua
    from paper_2407_21255_amd.cycle import slice_tables

    s = sched.shape
    prepared = {k: slice_tables(sched, k) for k in ids}
    sa = torch.cuda.Stream()
    sb = torch.cuda.Stream() if streams == 2 else sa
    kv = aqua.KVPool(s.as_tuple(), pool)
    if host_path is not None:
        _configure_host(kv, host_path)
    evs = []
    do_out, do_in = legs != "in", legs != "out"

    def one(k, timed):
        out, out_off, inn, in_off = prepared[k]
        ev = [None] * 4
        if timed:
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        if do_out:
            if timed:
                ev[0].record(sa)
            kv.swap_out(out, region, out_off, stream=sa)
            if timed:
                ev[1].record(sa)
        if do_in:
            if timed:
                ev[2].record(sb)
            kv.swap_in(inn, region, in_off, stream=sb)
            if timed:
                ev[3].record(sb)
        if timed:
            evs.append((*ev, len(out[0]) if do_out else 0, len(inn[0]) if do_in else 0))
        kv.sync(0)

    for k in ids[:warmup]:
        one(k, False)
    kv.sync(0)
    torch.cuda.synchronize()
    st0 = kv.stats()
    with _no_gc():
        t0 = time.perf_counter()
        for k in ids[warmup:]:
            one(k, True)
        kv.sync(0)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    st = _since(kv.stats(), st0)
    kv.close()
    unit = s.num_layers * s.chunk_bytes
    out_b = np.array([e[4] for e in evs], dtype=np.float64) * unit
    in_b = np.array([e[5] for e in evs], dtype=np.float64) * unit
    out_ms = np.array([e[0].elapsed_time(e[1]) if do_out else 0.0 for e in evs])
    in_ms = np.array([e[2].elapsed_time(e[3]) if do_in else 0.0 for e in evs])

    def union(e):
        # Union of the issued calls' intervals in a slice, from the first start.
        starts = [x for x, on in ((e[0], do_out), (e[2], do_in)) if on]
        ends = [x for x, on in ((e[1], do_out), (e[3], do_in)) if on]
        ref = starts[0]
        return (max(ref.elapsed_time(x) for x in ends)
                - min([0.0] + [ref.elapsed_time(x) for x in starts[1:]]))

    both_ms = np.array([union(e) for e in evs])
    return wall, st, out_b, in_b, out_ms, in_ms, both_ms


def _slice_kernel(config, host):
    """What the slice roofline covers: the calls issued and their streams."""
    legs = config.get("slice_legs", "both")
    if legs != "both":
        return ("gather" if legs == "out" else "scatter") + " of a slice"
    if config.get("slice_streams", 2) == 1:
        return "gather then scatter of a slice, on one stream"
    return "gather and scatter of a slice, on two streams" + (
        " (one link direction each)" if host else " (sharing HBM)")


def _slice_result(res_common, s, wall, st, out_b, in_b, out_ms, in_ms, both_ms, steps, config,
                  host=False):
    from paper_2407_21255_amd import workload as wl

    moved = float(out_b.sum() + in_b.sum())
    ok = out_b > 0
    # A slice's swap-out and swap-in run on two streams (at once, unless the
    # library orders them) and share the bound: every payload byte is read and
    # written once in HBM, or crosses one direction of the host link once
    # (both directions busy: twice the per-direction peak).  Rate of each slice
    # over the union of the two calls' intervals.
    per = 1 if host else 2
    both = (out_b + in_b) > 0
    achieved = (float((per * (out_b + in_b)[both] / (both_ms[both] * 1e-3)).mean()) / 1e9
                if both.any() else 0.0)
    peak = 2 * HOST_LINK_PEAK_GBS if host else HBM_PEAK_GBS
    res = dict(res_common)
    res.update({
        "value": round(moved / wall / 1e9, 2),
        "ms_per_step": round(wall * 1e3 / max(1, steps), 4),
        "dtype": wl.DTYPE_NAME[s.dtype],
        "config": config,
        "roofline": {
            "bound": "host_link" if host else "hbm",
            "kernel": _slice_kernel(config, host),
            "achieved": round(achieved, 1), "peak": peak, "unit": "GB/s",
            "frac": round(achieved / peak, 4), "traffic": None,
            "algorithmic_bytes_per_launch": round(float(per * (out_b + in_b)[both].mean()))
            if both.any() else 0,
        },
        "kernel_ms": {"swap_out_mean": round(float(out_ms[ok].mean()), 4) if ok.any() else 0,
                      "swap_in_mean": round(float(in_ms[in_b > 0].mean()), 4)
                      if (in_b > 0).any() else 0},
        "slice_hbm_GBps": None if host else round(2 * moved / wall / 1e9, 1),
        "waits_inserted": st["waits_inserted"],
        "host_us_per_call": round(st["host_ns"] / max(1, st["calls_out"] + st["calls_in"]) / 1e3,
                                  2),
        "kernel_source": _kernel_hash(),
    })
    return res


def run_cycle(args, res_common):
    """Slices of the preemption schedule: out on one stream, in on another."""
    import torch

    from paper_2407_21255_amd import workload as wl

    n = args.warmup + args.steps
    sched = wl.preemption_schedule(n_slices=n)
    s = sched.shape
    pool = torch.empty(s.pool_bytes, dtype=torch.uint8, device="cuda")
    wl.fill_pool(pool, s, sched.seed, wl.schedule_owner(sched))
    on_host = args.workload == "cycle_host"
    if on_host:
        # Pinned host swap space; its contents do not change the timing.
        region = torch.empty(sched.region_bytes, dtype=torch.uint8, pin_memory=True)
    else:
        region = torch.empty(sched.region_bytes, dtype=torch.uint8, device="cuda")
        wl.fill_region(region, sched)
    torch.cuda.synchronize()
    timed = _time_slices(sched, pool, region, list(range(n)), args.warmup,
                         host_path=args.host_path if on_host else None,
                         streams=args.slice_streams, legs=args.slice_legs)
    out_b, in_b = timed[2], timed[3]
    config = {
        "workload": WORKLOADS[args.workload], "layers": s.num_layers,
        "kv_heads": s.num_kv_heads, "head_dim": s.head_dim, "block_tokens": s.block_tokens,
        "pool_blocks": s.num_blocks, "chunk_bytes": s.chunk_bytes,
        "prompts": len(sched.nblocks), "swaps_per_slice": 16, "slices_timed": args.steps,
        "host_sync_per_slice": True, "slice_streams": args.slice_streams,
        "slice_legs": args.slice_legs,
        "mean_payload_bytes_per_direction":
            round(float((in_b if args.slice_legs == "in" else out_b).mean())),
        "offload_target": "pinned_host" if on_host else "hbm",
        "host_path": args.host_path if on_host else None, "parallelism": "single_gpu",
    }
    res = _slice_result(res_common, s, *timed, args.steps, config, host=on_host)
    if on_host:
        res["link_ceiling"] = link_ceiling()
    return res, s


def run_elastic(args, res_common):
    """Reclaim and restore of a swap space in the middle of a fair-scheduling
    run: per-phase reschedule times and the link rate of the moves."""
    import numpy as np
    import torch

    from paper_2407_21255_amd import aqua, cfs
    from paper_2407_21255_amd import workload as wl
    from paper_2407_21255_amd.cycle import run_slices_in_space

    cfg = wl.CFS_LLAMA8B
    s = cfg.shape
    tr = cfg.trace()
    log, _ = cfs.run_trace(tr, s.num_blocks, s.block_tokens, cfg.batch_tokens,
                           cfg.decode_slots(tr), cfg.k)
    sched = wl.cfs_swap_schedule(s, cfg.seed, tr, log)
    n1, n2, n3 = 20, 25, 30
    prompts = sorted({p for sl in sched.slices[:n3] for p in sl.out_prompts + sl.in_prompts})
    sizes = {p: s.image_bytes(sched.nblocks[p]) for p in prompts}
    room = sum((b + 255) // 256 * 256 for b in sizes.values())
    pool = torch.empty(s.pool_bytes, dtype=torch.uint8, device="cuda")
    wl.fill_pool(pool, s, cfg.seed)
    torch.cuda.synchronize()
    kv = aqua.KVPool(s.as_tuple(), pool)
    _configure_host(kv, "staged")
    space = aqua.SwapSpace(kv, room, room)
    tensors = {p: space.alloc(sizes[p]) for p in prompts}
    assert space.usage()["host_tensors"] == 0
    sa, sb, sc = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()

    def payload(a, b):
        return sum(s.image_bytes(len(t)) for sl in sched.slices[a:b]
                   for t in sl.out_tables + sl.in_tables)

    def phase(a, b):
        per = []
        for k in range(a, b):
            t0 = time.perf_counter()
            run_slices_in_space(kv, space, tensors, sched, k, 1, sa, sb)
            per.append(time.perf_counter() - t0)
        moved = payload(a, b)
        return {"reschedules": [a, b], "ms_per_reschedule": round(float(np.mean(per)) * 1e3, 3),
                "payload_bytes": moved, "GBps": round(moved / sum(per) / 1e9, 2)}

    def move(fn):
        before = space.usage()
        t0 = time.perf_counter()
        fn(stream=sc)
        kv.sync(0)
        dt = time.perf_counter() - t0
        after = space.usage()
        moved = abs(after["device_free"] - before["device_free"])
        return {"bytes": moved, "ms": round(dt * 1e3, 3), "GBps": round(moved / dt / 1e9, 2),
                "tensors_moved": abs(after["host_tensors"] - before["host_tensors"])}

    with _no_gc():
        wall0 = time.perf_counter()
        ph = [phase(0, n1)]
        rec = move(space.reclaim)
        ph.append(phase(n1, n2))
        res_ = move(space.restore)
        ph.append(phase(n2, n3))
        wall = time.perf_counter() - wall0
    carrier = [kv.link_engine(0), kv.link_engine(1)]
    space.close()
    kv.close()
    moved = sum(p["payload_bytes"] for p in ph) + rec["bytes"] + res_["bytes"]
    res = dict(res_common)
    res.update({
        # a fixed sequence: 30 reschedules, a reclaim and a restore, no warm-up
        "steps": n3, "warmup": 0,
        "value": round(moved / wall / 1e9, 2),
        "ms_per_step": round(wall * 1e3 / n3, 4),
        "dtype": wl.DTYPE_NAME[s.dtype],
        "config": {"workload": WORKLOADS["elastic"], "layers": s.num_layers,
                   "kv_heads": s.num_kv_heads, "head_dim": s.head_dim,
                   "block_tokens": s.block_tokens, "pool_blocks": s.num_blocks,
                   "chunk_bytes": s.chunk_bytes, "prompts": len(prompts),
                   "swap_space_bytes": room, "link_carrier": carrier,
                   "parallelism": "single_gpu"},
        "phases": {"device_region": ph[0], "host_after_reclaim": ph[1],
                   "device_after_restore": ph[2]},
        "reclaim": rec, "restore": res_,
        "roofline": {"bound": "host_link", "kernel": "reclaim (engine copies to host)",
                     "achieved": rec["GBps"], "peak": HOST_LINK_PEAK_GBS, "unit": "GB/s",
                     "frac": round(rec["GBps"] / HOST_LINK_PEAK_GBS, 4), "traffic": None,
                     "algorithmic_bytes_per_launch": rec["bytes"]},
    })
    return res, s


def run_cfs(args, res_common):
    """Fair scheduling of a burst on the 8B-shaped pool: the rescheduler's
    page-outs and page-ins, slice by slice, for the slices that swap."""
    import torch

    from paper_2407_21255_amd import cfs
    from paper_2407_21255_amd import workload as wl

    cfg = wl.CFS_LLAMA8B
    s = cfg.shape
    tr = cfg.trace()
    d = cfg.decode_slots(tr)
    t0 = time.perf_counter()
    log, sch = cfs.run_trace(tr, s.num_blocks, s.block_tokens, cfg.batch_tokens, d, cfg.k)
    sched_s = time.perf_counter() - t0
    sched = wl.cfs_swap_schedule(s, cfg.seed, tr, log)
    ids = [k for k, sl in enumerate(sched.slices) if sl.out_tables or sl.in_tables]
    ids = ids[:args.warmup + args.steps]
    steps = len(ids) - min(args.warmup, len(ids))
    pool = torch.empty(s.pool_bytes, dtype=torch.uint8, device="cuda")
    wl.fill_pool(pool, s, cfg.seed)
    region = torch.empty(sched.region_bytes, dtype=torch.uint8, device="cuda")
    wl.fill_region(region, sched)
    torch.cuda.synchronize()
    timed = _time_slices(sched, pool, region, ids, args.warmup, streams=args.slice_streams,
                         legs=args.slice_legs)
    out_b, in_b = timed[2], timed[3]
    config = {
        "workload": WORKLOADS["cfs"], "layers": s.num_layers, "kv_heads": s.num_kv_heads,
        "head_dim": s.head_dim, "block_tokens": s.block_tokens, "pool_blocks": s.num_blocks,
        "chunk_bytes": s.chunk_bytes, "requests": len(tr), "batch_tokens": cfg.batch_tokens,
        "decode_slots": d, "k": cfg.k, "iterations": len(log), "reschedules": len(sched.slices),
        "swapping_slices": len([1 for sl in sched.slices if sl.out_tables or sl.in_tables]),
        "slices_timed": steps, "host_sync_per_slice": True,
        "slice_streams": args.slice_streams, "slice_legs": args.slice_legs,
        "mean_payload_bytes_per_direction":
            round(float((in_b if args.slice_legs == "in" else out_b).mean())) if len(out_b) else 0,
        "offload_target": "hbm", "parallelism": "single_gpu",
    }
    res = _slice_result(res_common, s, *timed, steps, config)
    res["scheduler"] = {
        "partition_calls": sch.partition_calls,
        "host_us_per_iteration": round(sched_s * 1e6 / len(log), 2),
        "swap_ms_per_swapping_slice": round(float(timed[0] * 1e3 / max(1, steps)), 3),
    }
    return res, s


def run_next(args, res_common):
    """Prefix swap-in, layer-group swap-in, and image migration."""
    import numpy as np
    import torch

    from paper_2407_21255_amd import aqua
    from paper_2407_21255_amd import workload as wl

    w = args.workload
    if w.startswith("prefix"):
        s = wl.YI34B
        n = ceil_div_tokens(100000, s.block_tokens)          # 6250 blocks
        m = n - 256 // s.block_tokens                          # prefix: all but 256 tokens
        perm = wl.permutation(s.num_blocks, 6)
        prompt, fresh = perm[:n], perm[s.num_blocks - m:]
        owner = {b: (0, i) for i, b in enumerate(prompt)}
    else:
        case = wl.llama70b_case()
        s, prompt, fresh, owner = case.shape, case.out_tables[0], case.in_tables[0], case.owner
        n = m = len(prompt)
    pool = torch.empty(s.pool_bytes, dtype=torch.uint8, device="cuda")
    wl.fill_pool(pool, s, 6, owner)
    pinned = w in ("prefix_host", "layered_host")
    nbytes = s.image_bytes(n)
    img = (torch.empty(nbytes, dtype=torch.uint8, pin_memory=True) if pinned
           else torch.empty(nbytes, dtype=torch.uint8, device="cuda"))
    img.zero_()
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    kv = aqua.KVPool(s.as_tuple(), pool)
    if pinned:
        _configure_host(kv, args.host_path)
    else:
        _configure_link(kv)
    kv.swap_out([prompt], img, stream=stream)
    kv.sync(0)
    extra = {}
    tf = aqua._csr([fresh])
    if w == "migrate":
        back = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
        moved = 2 * nbytes
        def step(timed_evs):
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            e0.record(stream)
            kv.migrate(img, back, [0], [0], [nbytes], stream=stream)
            e1.record(stream)
            kv.migrate(back, img, [0], [0], [nbytes], stream=stream)
            e2.record(stream)
            timed_evs.append((e0, e1, e2))
    elif w == "prefix_mixed":
        # Background swaps on blocks the prefix loads do not touch.
        bg_a = [perm[0:448], perm[448:896]]
        bg_b = [perm[896:1344], perm[1344:1792]]
        bg_bytes = s.image_bytes(896)
        img_bg = torch.empty(bg_bytes, dtype=torch.uint8, device="cuda")
        sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
        ta, tb = aqua._csr(bg_a), aqua._csr(bg_b)
        moved = s.image_bytes(m) + 20 * bg_bytes

        def prefix_load():
            e0, e1 = (torch.cuda.Event(enable_timing=True) for _ in range(2))
            e0.record(stream)
            kv.swap_in(tf, img, stream=stream, img_blocks=[n])
            e1.record(stream)
            return e0, e1

        def step(timed_evs):
            p0, p1 = prefix_load()
            b0, b1 = (torch.cuda.Event(enable_timing=True) for _ in range(2))
            b0.record(sa)
            for j in range(10):
                src, dst = (ta, tb) if j % 2 == 0 else (tb, ta)
                kv.swap_out(src, img_bg, stream=sa)
                kv.swap_in(dst, img_bg, stream=sb)
            b1.record(sb)
            timed_evs.append((p0, p1, b0, b1))
    elif w.startswith("layered"):
        groups = [(l0, 8) for l0 in range(0, s.num_layers, 8)]
        moved = nbytes
        def step(timed_evs):
            evs = [torch.cuda.Event(enable_timing=True)]
            evs[0].record(stream)
            for l0, nl in groups:
                kv.swap_in(tf, img, stream=stream, layers=(l0, nl))
                e = torch.cuda.Event(enable_timing=True)
                e.record(stream)
                evs.append(e)
            timed_evs.append(tuple(evs))
    else:
        moved = s.image_bytes(m)
        def step(timed_evs):
            e0, e1 = (torch.cuda.Event(enable_timing=True) for _ in range(2))
            e0.record(stream)
            kv.swap_in(tf, img, stream=stream, img_blocks=[n])
            e1.record(stream)
            timed_evs.append((e0, e1))
    warm = []
    tw = None
    # With GEMMs beside the steps, a warm step after the first sizes the GEMM
    # load.
    for i in range(max(args.warmup, 2) if args.gemm else args.warmup):
        if i == 1:
            kv.sync(0)
            torch.cuda.synchronize()
            tw = time.perf_counter()
        step(warm)
    kv.sync(0)
    torch.cuda.synchronize()
    n_warm = max(args.warmup, 2) if args.gemm else args.warmup
    step_s = (time.perf_counter() - tw) / (n_warm - 1) if tw is not None else 0.0
    if w == "prefix_mixed":
        # The same prefix load with nothing else running, for comparison.
        alone = [prefix_load() for _ in range(3)]
        kv.sync(0)
        torch.cuda.synchronize()
        alone_ms = float(np.mean([a.elapsed_time(b) for a, b in alone]))
    comp = GemmCompanion(step_s, args.steps) if args.gemm else None
    evs = []
    st0 = kv.stats()
    with _no_gc():
        t0 = time.perf_counter()
        for _ in range(args.steps):
            if comp:
                comp.step()
            step(evs)
        kv.sync(0)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    st = _since(kv.stats(), st0)
    carrier = ([kv.link_engine(0), kv.link_engine(1)]
               if (pinned and args.host_path == "staged") or w == "migrate" else None)
    kv.close()
    if w == "migrate":
        d2h = np.mean([a.elapsed_time(b) for a, b, _ in evs])
        h2d = np.mean([b.elapsed_time(c) for _, b, c in evs])
        extra = {"hbm_to_host_ms": round(float(d2h), 3), "host_to_hbm_ms": round(float(h2d), 3),
                 "hbm_to_host_GBps": round(nbytes / d2h / 1e6, 2),
                 "host_to_hbm_GBps": round(nbytes / h2d / 1e6, 2)}
        bound, peak, dom_ms, alg = "host_link", HOST_LINK_PEAK_GBS, max(d2h, h2d), nbytes
    elif w == "prefix_mixed":
        beside = float(np.mean([a.elapsed_time(b) for a, b, _, _ in evs]))
        bg_ms = float(np.mean([c.elapsed_time(d) for _, _, c, d in evs]))
        extra = {"prefix_tokens": m * s.block_tokens, "cached_tokens": 100000,
                 "prefix_alone_ms": round(alone_ms, 3),
                 "prefix_beside_traffic_ms": round(beside, 3),
                 "background_ms_per_10_iterations": round(bg_ms, 3),
                 "background_GBps": round(20 * bg_bytes / bg_ms / 1e6, 1)}
        bound, peak, dom_ms, alg = "hbm", HBM_PEAK_GBS, wall * 1e3 / args.steps, 2 * moved
    elif w.startswith("layered"):
        first = np.mean([e[0].elapsed_time(e[1]) for e in evs])
        total = np.mean([e[0].elapsed_time(e[-1]) for e in evs])
        extra = {"first_group_ms": round(float(first), 3), "all_groups_ms": round(float(total), 3),
                 "groups": 10, "layers_per_group": 8}
        if pinned:
            bound, peak, dom_ms, alg = "host_link", HOST_LINK_PEAK_GBS, total / 10, nbytes / 10
        else:
            bound, peak, dom_ms, alg = "hbm", HBM_PEAK_GBS, total / 10, 2 * nbytes / 10
    else:
        ms = np.mean([a.elapsed_time(b) for a, b in evs])
        extra = {"prefix_tokens": m * s.block_tokens, "cached_tokens": 100000,
                 "load_ms": round(float(ms), 3)}
        if pinned:
            bound, peak, dom_ms, alg = "host_link", HOST_LINK_PEAK_GBS, ms, moved
        else:
            bound, peak, dom_ms, alg = "hbm", HBM_PEAK_GBS, ms, 2 * moved
    achieved = alg / (dom_ms * 1e-3) / 1e9
    res = dict(res_common)
    res.update({
        "value": round(moved * args.steps / wall / 1e9, 2),
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "dtype": wl.DTYPE_NAME[s.dtype],
        "config": {"workload": WORKLOADS[w], "layers": s.num_layers, "kv_heads": s.num_kv_heads,
                   "head_dim": s.head_dim, "block_tokens": s.block_tokens,
                   "pool_blocks": s.num_blocks, "chunk_bytes": s.chunk_bytes,
                   "image_blocks": n, "moved_bytes_per_step": moved,
                   "host_path": args.host_path if pinned else None,
                   "link_carrier": carrier,
                   "parallelism": "single_gpu"},
        "roofline": {"bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": "GB/s",
                     "frac": round(achieved / peak, 4), "traffic": None,
                     "algorithmic_bytes_per_launch": alg},
        "host_us_per_call": round(st["host_ns"] / max(1, st["calls_out"] + st["calls_in"] +
                                                       st["calls_migrate"]) / 1e3, 2),
        "kernel_source": _kernel_hash(),
    })
    if comp:
        res["compute_stream"] = comp.result()
    res.update(extra)
    return res, s


SWEEP_BLOCKS = (2, 8, 32, 128, 512, 2048)   # prompt lengths of the size sweep, in blocks


def _timed_on(stream, reps, fn):
    """Mean HIP-event time (ms) of ``fn()`` over ``reps`` calls on ``stream``,
    after one untimed call, and the host wall time per call (ms)."""
    import torch
    fn()
    stream.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    stream.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / reps
    return e0.elapsed_time(e1) / reps, wall


def _round_trips(kv, stream, a, b, buf, reps):
    """``reps`` round trips (swap-out of one table into ``buf``, swap-in into
    the other, the two tables trading places each time, as in the pair
    workloads) after one untimed round trip: mean HIP-event time of the
    swap-outs and of the swap-ins (ms), and the host wall time per round trip
    (ms, enqueue to completion)."""
    import numpy as np
    import torch
    kv.swap_out(a, buf, stream=stream)
    kv.swap_in(b, buf, stream=stream)
    stream.synchronize()
    evs = []
    t0 = time.perf_counter()
    for i in range(reps):
        src, dst = (a, b) if i % 2 else (b, a)
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record(stream)
        kv.swap_out(src, buf, stream=stream)
        e[1].record(stream)
        kv.swap_in(dst, buf, stream=stream)
        e[2].record(stream)
        evs.append(e)
    stream.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / reps
    out_ms = float(np.mean([x.elapsed_time(y) for x, y, _ in evs]))
    in_ms = float(np.mean([y.elapsed_time(z) for _, y, z in evs]))
    return out_ms, in_ms, wall


def run_sizes(args, res_common):
    """Swap rate against payload size, the measurement behind the paper's case
    for a gather (a copy's rate grows with its size, so one prompt's many small
    chunks move slowly one by one).  For each prompt length: the library's
    gather and scatter to an HBM region and, staged, to pinned host memory;
    one contiguous runtime copy of the same bytes (device to device, and
    device to pinned host); and the runtime's copies of the same chunks one
    chunk at a time (hipMemcpyAsync per (layer, block), as a serving engine
    without a gather kernel would issue them)."""
    import numpy as np
    import torch

    from paper_2407_21255_amd import aqua
    from paper_2407_21255_amd import workload as wl

    s = wl.LLAMA8B
    C, L, N = s.chunk_bytes, s.num_layers, s.num_blocks
    pool = torch.empty(s.pool_bytes, dtype=torch.uint8, device="cuda")
    wl.fill_pool(pool, s, 41)
    perm = wl.permutation(N, 41)
    biggest = s.image_bytes(max(SWEEP_BLOCKS))
    dimg = torch.zeros(biggest, dtype=torch.uint8, device="cuda")
    himg = torch.zeros(biggest, dtype=torch.uint8, pin_memory=True)
    torch.cuda.synchronize()
    hip = ctypes.CDLL("libamdhip64.so.7")
    hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_int, ctypes.c_void_p]
    hip.hipMemcpyAsync.restype = ctypes.c_int
    memcpy = hip.hipMemcpyAsync
    stream = torch.cuda.Stream()
    sh = stream.cuda_stream
    kv = aqua.KVPool(s.as_tuple(), pool)
    _configure_host(kv, "staged")   # host-target calls only; HBM calls are unaffected
    rows = []
    with _no_gc():
        # The swaps to the HBM region first, every size, before any host-target
        # call; then the staged host swaps and the runtime's copies.
        hbm = {}
        for n in SWEEP_BLOCKS:
            payload = s.image_bytes(n)
            a, b = aqua._csr([perm[:n]]), aqua._csr([perm[n:2 * n]])
            reps = max(8, min(50, (1 << 30) // payload))
            hbm[n] = _round_trips(kv, stream, a, b, dimg[:payload], reps)
        for n in SWEEP_BLOCKS:
            payload = s.image_bytes(n)
            a, b = aqua._csr([perm[:n]]), aqua._csr([perm[n:2 * n]])
            d, h = dimg[:payload], himg[:payload]
            out_ms, in_ms, rt_wall = hbm[n]
            reps = max(8, min(50, (1 << 30) // payload))
            hreps = max(2, min(20, (256 << 20) // payload))
            hout_ms, hin_ms, _ = _round_trips(kv, stream, a, b, h, hreps)
            src = pool[:payload]

            def bulk_d2d():
                with torch.cuda.stream(stream):
                    d.copy_(src)

            def bulk_d2h():
                with torch.cuda.stream(stream):
                    h.copy_(src, non_blocking=True)

            d2d_ms, _ = _timed_on(stream, reps, bulk_d2d)
            d2h_ms, _ = _timed_on(stream, hreps, bulk_d2h)
            # One runtime copy per (layer, block) chunk of the same prompt.
            blk = np.asarray(perm[:n], dtype=np.int64)
            lay = np.arange(L, dtype=np.int64)[:, None]
            srcs = (pool.data_ptr() + (lay * N + blk[None, :]) * C).ravel().tolist()
            offs = (np.arange(L * n, dtype=np.int64) * C).tolist()
            dd = [d.data_ptr() + o for o in offs]
            hh = [h.data_ptr() + o for o in offs]

            def chunks(dsts, kind):
                def go():
                    for x, y in zip(dsts, srcs):
                        if memcpy(x, y, C, kind, sh):
                            raise RuntimeError("hipMemcpyAsync failed")
                return go

            preps = max(1, min(10, 4096 // (L * n)))
            pc_d2d_ms, pc_d2d_wall = _timed_on(stream, preps, chunks(dd, 3))
            pc_d2h_ms, pc_d2h_wall = _timed_on(stream, preps, chunks(hh, 2))
            gbs = lambda ms: round(payload / (ms * 1e-3) / 1e9, 2)  # noqa: E731
            rows.append({
                "blocks": n, "payload_bytes": payload, "chunks": L * n,
                "hbm": {"gather_GBps": gbs(out_ms), "scatter_GBps": gbs(in_ms),
                        "gather_ms": round(out_ms, 4), "scatter_ms": round(in_ms, 4),
                        "round_trip_wall_ms": round(rt_wall, 4),
                        "runtime_copy_GBps": gbs(d2d_ms),
                        "per_chunk_copies_GBps": gbs(pc_d2d_ms),
                        "per_chunk_copies_wall_GBps": gbs(pc_d2d_wall)},
                "pinned_host_staged": {"swap_out_GBps": gbs(hout_ms),
                                       "swap_in_GBps": gbs(hin_ms),
                                       "runtime_copy_d2h_GBps": gbs(d2h_ms),
                                       "per_chunk_copies_d2h_GBps": gbs(pc_d2h_ms),
                                       "per_chunk_copies_d2h_wall_GBps": gbs(pc_d2h_wall)},
            })
            row = rows[-1]["hbm"]
            print(f"size sweep: {payload >> 20} MiB gather {row['gather_GBps']} GB/s, "
                  f"per-chunk copies {row['per_chunk_copies_GBps']} GB/s",
                  file=sys.stderr, flush=True)
        # The largest HBM round trip again, after the host-target calls.
        n = SWEEP_BLOCKS[-1]
        again = _round_trips(kv, stream, aqua._csr([perm[:n]]), aqua._csr([perm[n:2 * n]]),
                             dimg[:s.image_bytes(n)], 4)
    kv.close()
    top = rows[-1]
    t_out, t_in = top["hbm"]["gather_ms"], top["hbm"]["scatter_ms"]
    payload = top["payload_bytes"]
    dom_ms = max(t_out, t_in)
    achieved = 2 * payload / (dom_ms * 1e-3) / 1e9
    res = dict(res_common)
    res.update({
        "value": round(2 * payload / ((t_out + t_in) * 1e-3) / 1e9, 2),
        "ms_per_step": round(t_out + t_in, 4),
        "dtype": wl.DTYPE_NAME[s.dtype],
        "config": {
            "workload": WORKLOADS["sizes"],
            "layers": L, "kv_heads": s.num_kv_heads, "head_dim": s.head_dim,
            "block_tokens": s.block_tokens, "pool_blocks": N, "chunk_bytes": C,
            "swapped_blocks": list(SWEEP_BLOCKS),
            "offload_target": "hbm and pinned_host", "parallelism": "single_gpu",
        },
        "roofline": {
            "bound": "hbm", "kernel": "gather (swap-out)" if t_out >= t_in else
            "scatter (swap-in)", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
            "algorithmic_bytes_per_launch": 2 * payload,
        },
        "sweep": rows,
        "largest_hbm_after_host_calls": {
            "gather_GBps": round(payload / (again[0] * 1e-3) / 1e9, 2),
            "scatter_GBps": round(payload / (again[1] * 1e-3) / 1e9, 2)},
        "kernel_source": _kernel_hash(),
    })
    return res, s


def secondary_legs(args, common) -> dict:
    """Two shorter legs reported beside the default line, outside its timed
    region: the same 32768-token prompt swapped out to pinned host memory
    and back on the library's default host path (staged through HBM, link
    copies on a copy engine; 2 timed steps), and the fp8 preemption cycle
    (10 timed slices of 16 out on one stream and 16 in on another)."""
    import torch

    legs = {}
    sub = argparse.Namespace(**vars(args))
    sub.workload, sub.host_path, sub.steps, sub.warmup = "llama70b_host", "staged", 2, 1
    sub.copy_reference = False
    r, _ = run_pair(sub, {})
    legs["llama70b_host_staged"] = {
        "workload": WORKLOADS["llama70b_host"] + " (staged through HBM)",
        "steps": sub.steps, "value": r["value"], "unit": "GB/s",
        "swap_out_GBps": r["swap_out_GBps"], "swap_in_GBps": r["swap_in_GBps"],
        "roofline": {k: r["roofline"][k] for k in ("bound", "achieved", "peak", "frac")},
        "host_link_frac": r["host_link_frac"], "link_ceiling": r["link_ceiling"],
        "link_carrier": r["config"]["link_carrier"]}
    torch.cuda.empty_cache()
    sub = argparse.Namespace(**vars(args))
    sub.workload, sub.steps, sub.warmup = "cycle", 10, 2
    r, _ = run_cycle(sub, {})
    legs["preemption_cycle"] = {
        "workload": WORKLOADS["cycle"], "slices_timed": sub.steps, "value": r["value"],
        "unit": "GB/s", "ms_per_slice": r["ms_per_step"],
        "roofline": {k: r["roofline"][k] for k in ("bound", "achieved", "peak", "frac")},
        "kernel_ms": r["kernel_ms"], "waits_inserted": r["waits_inserted"]}
    torch.cuda.empty_cache()
    return legs


def ceil_div_tokens(tokens, block_tokens):
    return -(-tokens // block_tokens)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama70b_hbm", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gemm", action="store_true",
                    help="run 4096^3 bf16 GEMMs on a compute stream during the swaps")
    ap.add_argument("--max-workgroups", type=int, default=0,
                    help="cap the swap kernels' grid (0: library default)")
    ap.add_argument("--host-path", default="zero_copy", choices=["zero_copy", "staged"],
                    help="pinned-host workloads: the kernels writing host memory over the "
                         "link (the zero-copy target these workloads are defined with), or "
                         "HBM staging plus link copies on a copy engine (the library's "
                         "default, which leaves the compute units to other streams)")
    ap.add_argument("--two-step", choices=["blit", "sdma"], default=None,
                    help="HBM-target pair workloads: the paper's two-step scheme as an ablation "
                         "(gather into a temporary HBM tensor, then one runtime device-to-device "
                         "copy on its blit kernel or on a copy engine)")
    ap.add_argument("--link-engine", default="auto",
                    help="staged path: carrier of the link copies, 'auto', 'runtime' (the HIP "
                         "runtime's copies) or an SDMA engine index 0..15")
    ap.add_argument("--copy-reference", action="store_true",
                    help="one plain device copy of the payload size before timing")
    ap.add_argument("--slice-streams", type=int, default=2, choices=[1, 2],
                    help="cycle, cycle_host, cfs: each slice's swap-out and swap-in on two "
                         "streams (the workload as defined) or on one, one after the other")
    ap.add_argument("--slice-legs", default="both", choices=["both", "out", "in"],
                    help="cycle, cycle_host, cfs: issue only the swap-outs or only the "
                         "swap-ins of every slice (a breakdown of the slice's time)")
    ap.add_argument("--no-secondary", action="store_true",
                    help="default workload: skip the two shorter legs reported beside it (the "
                         "same prompt to pinned host memory, and the preemption cycle)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the swap path runs on a single MI355X "
              "(no sharding, no collectives); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    global _link_request
    if args.link_engine not in LINK_ENGINE and not (args.link_engine.isdigit()
                                                    and int(args.link_engine) <= 15):
        ap.error("--link-engine: 'auto', 'runtime' or 0..15")
    _link_request = args.link_engine

    import torch

    from paper_2407_21255_amd import aqua

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    aqua.load()
    common = {
        "metric": "KV page swap GB/s (out+in) and % of HBM / host-link peak, 1 MI355X",
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "data": "synthetic",
    }
    if args.workload in ("cycle", "cycle_host"):
        res, shape = run_cycle(args, common)
    elif args.workload == "cfs":
        res, shape = run_cfs(args, common)
    elif args.workload == "elastic":
        res, shape = run_elastic(args, common)
    elif args.workload == "sizes":
        res, shape = run_sizes(args, common)
    elif args.workload in ("prefix", "prefix_host", "prefix_mixed", "layered", "layered_host",
                           "migrate"):
        res, shape = run_next(args, common)
    else:
        res, shape = run_pair(args, common)
    if args.workload == "llama70b_hbm" and not (args.no_secondary or args.gemm or
                                                args.two_step or args.max_workgroups):
        res["secondary"] = secondary_legs(args, common)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(shape, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
