// aqua_capi.hip -- the C ABI: pools, tickets, descriptor delivery,
// cross-stream ordering, the staged host path and the launches of the
// gather/scatter kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <map>
#include <mutex>
#include <new>
#include <set>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "aqua.h"
#include "aqua_core.h"
#include "link_engine.h"
#include "swap_kernels.h"

namespace {

using aqua::HazardTracker;
using aqua::RunDesc;

constexpr uint64_t kDefaultRingBytes = 4ull << 20;  // 131072 descriptors
constexpr uint64_t kDefaultUnitBytes = 64ull << 10;
constexpr uint64_t kDefaultSlotBytes = 512ull << 20;  // staged path, per slot
constexpr uint32_t kHostZeroCopyWorkgroups = 16;

// Measurement switches: the defaults are the shipped configuration, the
// macros exist so that sweeps can build variants.
// Smallest workgroup of the swap kernels.  1024 lanes for every chunk size:
// workgroups sized to 32 KiB chunks (512 lanes) measured no faster, and to
// 16 KiB chunks (256 lanes) 4 % slower.
#ifndef AQUA_MIN_THREADS
#define AQUA_MIN_THREADS 1024
#endif
// 1: HBM-target calls read their descriptors from the device ring too.
// Off: reading them in place from the pinned ring measured as fast or faster
// (no upload kernel on the stream).
#ifndef AQUA_DESC_DEVICE
#define AQUA_DESC_DEVICE 0
#endif
// 0: runs stay in table order (see aqua::run_order for the shipped rule).
#ifndef AQUA_SORT_RUNS
#define AQUA_SORT_RUNS 1
#endif

// Names one library call on the host timeline of a profiler that records
// markers (rocprofv3 --marker-trace); with none attached a push and a pop
// cost a function call each.
struct TraceRange {
    explicit TraceRange(const char* name) { roctxRangePushA(name); }
    ~TraceRange() { roctxRangePop(); }
    TraceRange(const TraceRange&) = delete;
    TraceRange& operator=(const TraceRange&) = delete;
};

uint64_t env_u64(const char* name, uint64_t dflt) {
    const char* v = std::getenv(name);
    if (!v || !*v) return dflt;
    char* end = nullptr;
    const unsigned long long x = std::strtoull(v, &end, 0);
    return (end && *end == 0) ? (uint64_t)x : dflt;
}

// Device scratch of the allocation-free swap entry point
// (aqua_swap_noalloc): its run descriptors, copied there from the pool's
// pinned ring on the call's stream.  One array per device for the life of
// the process; host code uses only the device address that
// hipGetSymbolAddress gives for the current device (scratch_address).
constexpr uint64_t kScratchBytes = 2ull << 20;  // 65536 run descriptors
constexpr uint32_t kPoolEvents = 16;             // events made at pool creation
__device__ __align__(256) uint8_t scratch[kScratchBytes];

// Device address of `scratch` on `device`, looked up once per device with
// that device current (the caller has made it current); nullptr on failure.
uint8_t* scratch_address(int device) {
    static std::mutex mu;
    static std::map<int, uint8_t*> addr;
    std::lock_guard<std::mutex> lk(mu);
    auto it = addr.find(device);
    if (it != addr.end()) return it->second;
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
        (void)hipGetLastError();
        return nullptr;
    }
    addr[device] = (uint8_t*)ptr;
    return (uint8_t*)ptr;
}

struct Outstanding {
    uint64_t ticket;
    hipEvent_t ev;                 // recorded on the call's stream, last
    std::vector<hipEvent_t> aux;   // events inside the call (staging slots)
};

struct RingUse {
    uint64_t lo, hi, ticket;
};

// One sequence of a staged call: image offset in the caller's buffer, its
// first entry in the concatenated table, its table length and its image's
// blocks per layer.
struct StagedSeq {
    uint64_t off, first, n, m;
};

}  // namespace

struct aqua_kv_pool {
    aqua::Shape shape;
    int device = 0;
    uint8_t* base = nullptr;
    uint64_t bytes = 0;

    aqua::DupMarks marks;
    HazardTracker tracker;
    std::vector<RunDesc> plan;
    std::vector<uint32_t> sort_counts;  // scratch of aqua::sort_by_block
    std::vector<RunDesc> sort_tmp;
    std::vector<std::pair<uint64_t, uint64_t>> ranges;
    std::vector<HazardTracker::Dep> deps;

    aqua::LaneMap lanes;                                // stream -> lane
    std::vector<std::deque<Outstanding>> outstanding;   // per lane, in order
    std::vector<hipEvent_t> spare_events;

    // Run descriptors reach the kernels through a pinned, coherent host ring:
    // the kernels read them in place (one 32-byte scalar load per workgroup,
    // no copy on the call's stream), except for calls that keep the host
    // link busy with their data (staged host swaps, migrations), whose
    // descriptors are copied to the device ring first.
    uint8_t* ring_host_dev = nullptr;  // device address of ring_host
    uint8_t* ring_host = nullptr;
    uint8_t* ring_dev = nullptr;
    uint64_t ring_bytes = 0;
    uint64_t ring_head = 0;
    std::deque<RingUse> ring_uses;

    // Staged host path, per direction (0: swap-out, device to host; 1:
    // swap-in, host to device): two HBM slots and a carrier for the link
    // copies, so that a swap-out and a swap-in use both directions of the
    // link at once.  The carrier is an SDMA engine driven by a LinkEngine,
    // or the runtime's copies on a copy stream.
    int32_t host_path = AQUA_HOST_STAGED;
    int32_t link_request[2] = {AQUA_LINK_AUTO, AQUA_LINK_AUTO};
    int32_t link_used[2] = {AQUA_LINK_AUTO, AQUA_LINK_AUTO};  // AUTO: not chosen yet
    bool hsa_up = false;
    aqua::LinkAgents agents;
    aqua::LinkEngine link[2];
    hipStream_t copy[2] = {nullptr, nullptr};
    uint8_t* staging[2] = {nullptr, nullptr};
    uint64_t staging_bytes[2] = {0, 0};
    uint64_t slot_target = kDefaultSlotBytes;
    // Launches of the kernel that releases engine jobs, and the one (from 0)
    // to report as failed without making it (AQUA_FAIL_RELEASE_AT: tests of
    // the failure path force it from the host, every kernel still ending).
    uint64_t releases = 0;
    uint64_t fail_release_at = ~0ull;
    std::vector<StagedSeq> sseq;
    std::vector<uint64_t> slot_offsets;  // per sequence, in a slot
    uint64_t call_blocks = 0;            // table entries of the call being enqueued

    uint64_t next_ticket = 1;
    uint64_t unit_bytes = kDefaultUnitBytes;
    uint8_t* scratch = nullptr;  // this device's scratch (aqua_swap_noalloc)
    // Grid caps per target (0: one workgroup per unit).  Zero-copy host
    // swaps are link-bound: 16 workgroups of 1024 lanes saturate the link.
    uint32_t max_wg[2] = {0, kHostZeroCopyWorkgroups};
    aqua_pool_stats stats{};
    hipError_t sticky = hipSuccess;
};

// Swap space: a device region and a host region, each handed out by a range
// allocator, and the tensors placed in them, by handle.
struct aqua_swap_space {
    aqua_kv_pool* pool = nullptr;
    uint8_t* region[2] = {nullptr, nullptr};  // index: AQUA_TARGET_DEVICE / _HOST
    uint64_t region_bytes[2] = {0, 0};
    aqua::RangeAllocator ranges[2];
    struct Tensor {
        uint64_t bytes;
        int32_t target;
        uint64_t off;
    };
    std::map<uint64_t, Tensor> tensors;  // by handle, oldest first
    uint64_t next_handle = 1;
};

namespace {

constexpr uint64_t kSwapAlign = 256;

// Switches to the pool's device for the duration of a call.
struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) {
            ok = false;
            return;
        }
        if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
        if (prev == dev) prev = -1;
    }
    ~DeviceGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

aqua_status latch(aqua_kv_pool* p, hipError_t e) {
    if (e != hipSuccess && p->sticky == hipSuccess) {
        p->sticky = e;
        p->stats.hip_error = (int32_t)e;
    }
    return AQUA_ERR_HIP;
}

// A call that fails after enqueueing work returns once that work has ended
// (or the device has failed), so that nothing it enqueued outlives the error
// it reports.
aqua_status fail_enqueued(hipStream_t stream, aqua_status st) {
    (void)hipStreamSynchronize(stream);
    (void)hipGetLastError();
    return st;
}

// Enqueues the release of up to two engine jobs' ready flags on `stream`.
hipError_t release_flags(aqua_kv_pool* p, int64_t* a, int64_t* b, hipStream_t stream) {
    if (!a) std::swap(a, b);
    if (!a) return hipSuccess;
    if (p->releases++ == p->fail_release_at) return hipErrorLaunchFailure;
    return aqua::launch_release_flags(a, b, stream);
}

// After a failure between submitting engine jobs and enqueueing their
// release: once the stream's earlier work has ended, the held flags are
// released from the host, so that the engine's queue drains, and the call
// returns once those jobs' copies have ended too.
aqua_status fail_held(aqua_kv_pool* p, aqua::LinkEngine& w, hipStream_t stream,
                      int64_t* const* held, int n, hipError_t e) {
    (void)hipStreamSynchronize(stream);
    (void)hipGetLastError();
    uint64_t upto = 0;
    for (int i = 0; i < n; ++i) upto = std::max(upto, w.release_on_host(held[i]));
    w.wait_published(upto);
    return latch(p, e);
}

uint32_t lane_for(aqua_kv_pool* p, hipStream_t s) {
    // A lane is handed to another stream only once the tracker knows every
    // call on it complete, which retire() reports as its queue empties.
    const uint32_t m = p->lanes.lane_for((uintptr_t)s, p->tracker);
    if (m >= p->outstanding.size()) p->outstanding.resize(m + 1);
    return m;
}

hipError_t take_event(aqua_kv_pool* p, hipEvent_t* ev) {
    if (!p->spare_events.empty()) {
        *ev = p->spare_events.back();
        p->spare_events.pop_back();
        return hipSuccess;
    }
    return hipEventCreateWithFlags(ev, hipEventDisableTiming);
}

// Everything on lane m up to `ticket` is known complete: recycle events.
void retire(aqua_kv_pool* p, uint32_t m, uint64_t ticket) {
    auto& q = p->outstanding[m];
    while (!q.empty() && q.front().ticket <= ticket) {
        p->spare_events.push_back(q.front().ev);
        for (hipEvent_t e : q.front().aux) p->spare_events.push_back(e);
        q.pop_front();
    }
    p->tracker.complete(m, ticket);
}

// A failure on a link engine's thread becomes the pool's sticky error.
aqua_status check_links(aqua_kv_pool* p) {
    for (int d = 0; d < 2; ++d) {
        const hipError_t e = p->link[d].error();
        if (e != hipSuccess) return latch(p, e);
    }
    return AQUA_OK;
}

// Non-blocking: retire whatever has finished.
aqua_status poll(aqua_kv_pool* p) {
    if (check_links(p) != AQUA_OK) return AQUA_ERR_HIP;
    for (uint32_t m = 0; m < p->outstanding.size(); ++m) {
        auto& q = p->outstanding[m];
        while (!q.empty()) {
            const hipError_t e = hipEventQuery(q.front().ev);
            if (e == hipErrorNotReady) break;
            if (e != hipSuccess) return latch(p, e);
            retire(p, m, q.front().ticket);
        }
    }
    return AQUA_OK;
}

hipEvent_t event_of(aqua_kv_pool* p, uint64_t ticket) {
    const uint32_t m = p->tracker.lane_of(ticket);
    if (m == HazardTracker::kNoLane) return nullptr;  // complete
    for (const Outstanding& o : p->outstanding[m])
        if (o.ticket == ticket) return o.ev;
    return nullptr;
}

// Blocks until `ticket` has completed.
aqua_status wait_ticket(aqua_kv_pool* p, uint64_t ticket) {
    const uint32_t m = p->tracker.lane_of(ticket);
    if (m == HazardTracker::kNoLane) return AQUA_OK;  // complete
    hipEvent_t ev = event_of(p, ticket);
    if (!ev) return AQUA_OK;  // retired already
    const hipError_t e = hipEventSynchronize(ev);
    if (e != hipSuccess) return latch(p, e);
    retire(p, m, ticket);
    return check_links(p);
}

aqua_status wait_all(aqua_kv_pool* p) {
    for (uint32_t m = 0; m < p->outstanding.size(); ++m) {
        auto& q = p->outstanding[m];
        if (q.empty()) continue;
        const uint64_t last = q.back().ticket;
        const hipError_t e = hipEventSynchronize(q.back().ev);
        if (e != hipSuccess) return latch(p, e);
        retire(p, m, last);
    }
    p->ring_uses.clear();
    return check_links(p);
}

// An event for a call of the allocation-free entry point: a spare one, or,
// while none is spare, the event of the oldest outstanding call once that
// call has completed.  Creates nothing: the pool made kPoolEvents events
// when it was created, and each is either spare or held by a call.
aqua_status take_event_noalloc(aqua_kv_pool* p, hipEvent_t* ev) {
    for (;;) {
        if (!p->spare_events.empty()) {
            *ev = p->spare_events.back();
            p->spare_events.pop_back();
            return AQUA_OK;
        }
        uint32_t oldest = UINT32_MAX;
        for (uint32_t m = 0; m < p->outstanding.size(); ++m)
            if (!p->outstanding[m].empty() &&
                (oldest == UINT32_MAX ||
                 p->outstanding[m].front().ticket < p->outstanding[oldest].front().ticket))
                oldest = m;
        if (oldest == UINT32_MAX) return AQUA_ERR_STATE;  // no event at all
        const aqua_status st = wait_ticket(p, p->outstanding[oldest].front().ticket);
        if (st != AQUA_OK) return st;
    }
}

void free_rings(aqua_kv_pool* p) {
    if (p->ring_dev) (void)hipFree(p->ring_dev);
    if (p->ring_host) (void)hipHostFree(p->ring_host);
    p->ring_dev = nullptr;
    p->ring_host = nullptr;
    p->ring_bytes = 0;
    p->ring_head = 0;
}

aqua_status alloc_rings(aqua_kv_pool* p, uint64_t bytes) {
    // The device ring serves calls that keep the host link busy (staged
    // host swaps, migrations): descriptors fetched over it would stall
    // their kernels.
    hipError_t e = hipMalloc((void**)&p->ring_dev, bytes);
    if (e == hipSuccess)
        e = hipHostMalloc((void**)&p->ring_host, bytes,
                          hipHostMallocMapped | hipHostMallocCoherent);
    if (e == hipSuccess)
        e = hipHostGetDevicePointer((void**)&p->ring_host_dev, p->ring_host, 0);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        free_rings(p);
        return AQUA_ERR_HIP;
    }
    p->ring_bytes = bytes;
    p->ring_head = 0;
    return AQUA_OK;
}

// Reserves `bytes` of the descriptor rings, waiting for the calls that used
// the space last.  Grows the rings when one call needs more than they hold.
aqua_status ring_reserve(aqua_kv_pool* p, uint64_t bytes, uint64_t* off, bool grow = true) {
    bytes = (bytes + 255) & ~255ull;
    if (bytes > p->ring_bytes && !grow) return AQUA_ERR_CAPACITY;
    if (bytes > p->ring_bytes) {
        aqua_status st = wait_all(p);
        if (st != AQUA_OK) return st;
        uint64_t nb = p->ring_bytes ? p->ring_bytes : kDefaultRingBytes;
        while (nb < bytes) nb *= 2;
        free_rings(p);
        st = alloc_rings(p, nb);
        if (st != AQUA_OK) return st;
    }
    // Uses of calls already known complete free their space.  The uses are
    // in allocation order and calls on different streams can complete out
    // of order, so only finished uses at the front are dropped.
    while (!p->ring_uses.empty() && p->tracker.done(p->ring_uses.front().ticket))
        p->ring_uses.pop_front();
    // Start again at the front of the ring when no live call's descriptors
    // are there: the host then writes into lines it wrote a few calls ago,
    // still in its caches.  Walking the whole ring wrote lines evicted long
    // before, and copying a 135 KB plan into them took about 30 us.
    bool front_free = true;
    for (const RingUse& u : p->ring_uses)
        if (u.lo < bytes) {
            front_free = false;
            break;
        }
    uint64_t lo = p->ring_head;
    if (front_free || lo + bytes > p->ring_bytes) lo = 0;
    const uint64_t hi = lo + bytes;
    for (;;) {
        bool overlap = false;
        for (const RingUse& u : p->ring_uses)
            if (u.lo < hi && lo < u.hi) {
                overlap = true;
                break;
            }
        if (!overlap) break;
        const aqua_status st = wait_ticket(p, p->ring_uses.front().ticket);
        if (st != AQUA_OK) return st;
        p->ring_uses.pop_front();
    }
    p->ring_head = hi;
    *off = lo;
    return AQUA_OK;
}

// Makes direction dir's staging buffer hold at least `bytes`, waiting for
// every outstanding call before it is replaced.  A direction without slots
// gets them at the same time, best effort (two slots of the default size,
// or `bytes` if larger), so that its first staged call does not wait for
// this one.
aqua_status ensure_staging(aqua_kv_pool* p, int dir, uint64_t bytes) {
    if (bytes <= p->staging_bytes[dir]) return AQUA_OK;
    aqua_status st = wait_all(p);
    if (st != AQUA_OK) return st;
    auto alloc = [&](int d, uint64_t nb) -> aqua_status {
        if (p->staging[d]) (void)hipFree(p->staging[d]);
        p->staging[d] = nullptr;
        p->staging_bytes[d] = 0;
        if (hipMalloc((void**)&p->staging[d], nb) != hipSuccess) {
            (void)hipGetLastError();
            p->staging[d] = nullptr;
            return AQUA_ERR_HIP;
        }
        p->staging_bytes[d] = nb;
        return AQUA_OK;
    };
    st = alloc(dir, bytes);
    // Best effort: on failure the other direction allocates on its own call.
    if (st == AQUA_OK && !p->staging[1 - dir])
        (void)alloc(1 - dir, std::max<uint64_t>(bytes, 2 * p->slot_target));
    return st;
}

// Copies n 16-byte vectors of run descriptors from the pinned host ring to
// the device ring (see upload_descs).
__global__ __launch_bounds__(256) void upload_descs_kernel(const uint4* __restrict__ src,
                                                           uint4* __restrict__ dst, uint32_t n) {
    for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < n; i += gridDim.x * 256u)
        dst[i] = src[i];
}

// Moves a call's descriptors, [ring_off, ring_off + bytes) of the rings, to
// the device ring on the call's stream: one pass over the link ahead of the
// call's kernels instead of a fetch per workgroup while the link carries
// the call's own data.  A kernel, not a runtime copy: the runtime can hold
// the calling thread on such a small copy until the stream's earlier host
// functions have run.  `bytes` is a multiple of 32 (whole descriptors).
hipError_t upload_to(const uint8_t* src, uint8_t* dst, uint64_t bytes, hipStream_t stream) {
    const uint32_t n = (uint32_t)(bytes / 16);
    if (!n) return hipSuccess;
    const uint32_t grid = std::min<uint32_t>(256u, (n + 255u) / 256u);
    (void)hipGetLastError();
    hipLaunchKernelGGL(upload_descs_kernel, dim3(grid), dim3(256), 0, stream,
                       reinterpret_cast<const uint4*>(src), reinterpret_cast<uint4*>(dst), n);
    return hipGetLastError();
}

hipError_t upload_descs(aqua_kv_pool* p, uint64_t ring_off, uint64_t bytes, hipStream_t stream) {
    return upload_to(p->ring_host_dev + ring_off, p->ring_dev + ring_off, bytes, stream);
}

// Launches one kernel of each of the library's source files once, with
// nothing to copy, on a private stream, so that the runtime loads their
// device code (one code object per source file) when the first pool of a
// process is created rather than at its first swap (the first launch in a
// process took 76 ms, and the first staged call's other kernels 7 ms more).
// The range-copy kernel, which shares its file with the swap kernels, gets
// one range of no bytes and reads only that descriptor; the flag kernel and
// the upload write only the pool's own, still unused, device ring.  The
// swap kernels themselves are not launched, so their dispatches are the
// caller's alone.
hipError_t warm_kernels(aqua_kv_pool* p) {
    static std::mutex mu;
    static std::set<int> warmed;
    std::lock_guard<std::mutex> lk(mu);
    if (warmed.count(p->device)) return hipSuccess;
    std::memset(p->ring_host, 0, 64);  // a zero CopyDesc: a range of no bytes
    hipStream_t s = nullptr;
    hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    if (e != hipSuccess) return e;
    e = aqua::launch_copy(p->base, p->base,
                              reinterpret_cast<const aqua::CopyDesc*>(p->ring_host_dev), 1, 0, s);
    if (e == hipSuccess) e = upload_descs(p, 0, 32, s);
    if (e == hipSuccess)
        e = aqua::launch_release_flags(reinterpret_cast<int64_t*>(p->ring_dev + 64), nullptr, s);
    const hipError_t es = hipStreamSynchronize(s);
    (void)hipStreamDestroy(s);
    if (e == hipSuccess) e = es;
    if (e == hipSuccess) warmed.insert(p->device);
    (void)hipGetLastError();
    return e;
}

// Chooses direction dir's carrier for link copies on its first staged call
// or host-side migration: the requested engine, or for AQUA_LINK_AUTO the
// automatic engine choice, falling back to the runtime's copies when the
// HSA runtime or the engine is unavailable.  An explicitly requested engine
// that cannot start is an error.
aqua_status ensure_link(aqua_kv_pool* p, int dir) {
    if (p->link_used[dir] != AQUA_LINK_AUTO) return AQUA_OK;
    const int32_t req = p->link_request[dir];
    if (req != AQUA_LINK_RUNTIME) {
        if (!p->hsa_up) p->hsa_up = aqua::link_acquire(p->device, &p->agents);
        int32_t eng = req;
        if (p->hsa_up && eng == AQUA_LINK_AUTO) {
            int32_t e2h = -1, h2d = -1;
            aqua::link_auto_engines(p->agents, &e2h, &h2d);
            eng = dir ? h2d : e2h;
        }
        if (p->hsa_up && eng >= 0 &&
            p->link[dir].start(p->device, p->agents, dir, eng) == hipSuccess) {
            p->link_used[dir] = eng;
            return AQUA_OK;
        }
        (void)hipGetLastError();
        if (req >= 0) return AQUA_ERR_HIP;
    }
    if (!p->copy[dir] &&
        hipStreamCreateWithFlags(&p->copy[dir], hipStreamNonBlocking) != hipSuccess) {
        (void)hipGetLastError();
        p->copy[dir] = nullptr;
        return AQUA_ERR_HIP;
    }
    p->link_used[dir] = AQUA_LINK_RUNTIME;
    return AQUA_OK;
}

// Device-accessible address of the buffer, after checking that its memory
// class matches the target and that [ptr, ptr + bytes) lies in one
// allocation.
aqua_status resolve_buffer(aqua_kv_pool* p, const void* ptr, uint64_t bytes,
                           int32_t target, uint8_t** dev) {
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof(attr));
    hipError_t e = hipPointerGetAttributes(&attr, ptr);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return AQUA_ERR_INVALID;
    }
    if (target == AQUA_TARGET_DEVICE) {
        if (attr.type != hipMemoryTypeDevice || attr.device != p->device)
            return AQUA_ERR_INVALID;
        *dev = (uint8_t*)const_cast<void*>(ptr);
    } else {
        if (attr.type != hipMemoryTypeHost || !attr.devicePointer)
            return AQUA_ERR_INVALID;
        *dev = (uint8_t*)attr.devicePointer;
    }
    hipDeviceptr_t rbase = nullptr;
    size_t rsize = 0;
    e = hipMemGetAddressRange(&rbase, &rsize, (hipDeviceptr_t)*dev);
    if (e == hipSuccess && rbase) {
        const uintptr_t b = (uintptr_t)rbase, x = (uintptr_t)*dev;
        if (x < b || x - b > rsize || bytes > rsize - (x - b)) return AQUA_ERR_INVALID;
    } else {
        (void)hipGetLastError();
        if (target == AQUA_TARGET_DEVICE) return AQUA_ERR_INVALID;
    }
    return AQUA_OK;
}

// One launch over layers [l0, l0 + nl) of the call being enqueued.
aqua::SwapLaunch make_launch(aqua_kv_pool* p, bool is_in, uint8_t* img, const RunDesc* descs,
                             uint32_t ndesc, int32_t target, uint32_t l0, uint32_t nl) {
    aqua::SwapLaunch L;
    L.out = !is_in;
    L.pool = p->base;
    L.img = img;
    L.img_l0 = 0;
    L.descs = descs;
    L.ndesc = ndesc;
    L.first_layer = l0;
    L.num_layers = nl;
    L.chunk_bytes = p->shape.C;
    L.pool_lstride = (uint64_t)p->shape.N * p->shape.C;
    L.max_workgroups = p->max_wg[target];
    L.nt_pool_store = aqua::nt_pool_store(p->shape.C, (uint64_t)nl * p->call_blocks * p->shape.C);
    L.threads = aqua::swap_threads(p->shape.C, AQUA_MIN_THREADS);
    L.xcd_order = false;
    return L;
}

// Staged host path.  Layers go through two HBM slots of G layers each
// (per direction: swap-outs and swap-ins have their own slots and link
// carrier, so one of each can run at once on the two directions of the
// link).  A slot holds, sequence after sequence, the sequence's G layers in
// image order ([G][n_s][C] at G * first_s * C), so each sequence's piece of a
// layer group is contiguous both in the slot and in the host image: one
// copy per sequence per group.  Swap-out: the gather fills a slot on the
// call's stream, then the carrier moves the pieces to the host image.
// Swap-in: the carrier fills a slot from the host image, then the scatter
// drains it on the call's stream.  A slot is refilled only after its
// previous user has finished with it.
//
// The copies moving sequence q's layers [l0, l0 + nl) between a slot and the
// host image: one piece when the image holds exactly the table's blocks,
// else one per layer (only the first n of its m blocks).
void stage_pieces(aqua_kv_pool* p, bool to_host, const void* buf, uint8_t* slot, uint32_t G,
                  uint32_t l0, uint32_t nl, std::vector<aqua::LinkPiece>* out) {
    const uint64_t C = p->shape.C;
    out->clear();
    for (const StagedSeq& q : p->sseq) {
        uint8_t* s = slot + G * q.first * C;
        uint8_t* h = (uint8_t*)const_cast<void*>(buf) + q.off;
        const uint32_t pieces = q.m == q.n ? 1 : nl;
        const uint64_t bytes = q.m == q.n ? nl * q.n * C : q.n * C;
        for (uint32_t j = 0; j < pieces; ++j) {
            const uint64_t l = l0 + j;
            uint8_t* hj = h + l * q.m * C;
            uint8_t* sj = s + (uint64_t)j * q.n * C;
            out->push_back(to_host ? aqua::LinkPiece{hj, sj, bytes}
                                   : aqua::LinkPiece{sj, hj, bytes});
        }
    }
}

aqua::SwapLaunch slot_launch(aqua_kv_pool* p, bool is_in, uint8_t* slot, const RunDesc* descs,
                             uint32_t ndesc, uint32_t l0, uint32_t nl) {
    // The kernels only touch HBM here: no host-link grid cap.
    aqua::SwapLaunch L = make_launch(p, is_in, slot, descs, ndesc, AQUA_TARGET_DEVICE, l0, nl);
    L.img_l0 = l0;
    return L;
}

// Link copies by the runtime, on the direction's copy stream.
aqua_status enqueue_staged_runtime(aqua_kv_pool* p, bool is_in, const void* buf,
                                   hipStream_t stream, const RunDesc* descs, uint32_t ndesc,
                                   uint64_t slot, uint32_t G, uint32_t l_begin, uint32_t l_end,
                                   Outstanding* rec) {
    hipError_t e = hipSuccess;
    auto ev = [&](hipEvent_t* x) -> hipError_t {
        hipError_t r = take_event(p, x);
        if (r == hipSuccess) rec->aux.push_back(*x);
        return r;
    };
    auto copies = [&](const std::vector<aqua::LinkPiece>& v) -> hipError_t {
        for (const aqua::LinkPiece& pc : v) {
            const hipError_t r = hipMemcpyAsync(
                pc.dst, pc.src, pc.bytes, is_in ? hipMemcpyHostToDevice : hipMemcpyDeviceToHost,
                p->copy[is_in]);
            if (r != hipSuccess) return r;
        }
        return hipSuccess;
    };
    // The copy stream starts after everything the call's stream must wait
    // for (ordering waits inserted for this call, earlier work).
    hipEvent_t start = nullptr;
    if ((e = ev(&start)) != hipSuccess) return latch(p, e);
    if ((e = hipEventRecord(start, stream)) != hipSuccess) return latch(p, e);
    hipStream_t copy = p->copy[is_in];
    if ((e = hipStreamWaitEvent(copy, start, 0)) != hipSuccess) return latch(p, e);

    std::vector<aqua::LinkPiece> pieces;
    hipEvent_t slot_free[2] = {nullptr, nullptr};
    hipEvent_t last_copy = nullptr;
    for (uint32_t l0 = l_begin, k = 0; l0 < l_end; l0 += G, ++k) {
        const uint32_t nl = std::min<uint32_t>(G, l_end - l0);
        uint8_t* s = p->staging[is_in] + (k % 2) * slot;
        const aqua::SwapLaunch Lk = slot_launch(p, is_in, s, descs, ndesc, l0, nl);
        stage_pieces(p, !is_in, buf, s, G, l0, nl, &pieces);
        hipEvent_t e1 = nullptr, e2 = nullptr;
        if ((e = ev(&e1)) != hipSuccess || (e = ev(&e2)) != hipSuccess) return latch(p, e);
        hipStream_t first = is_in ? copy : stream;   // fills the slot
        hipStream_t second = is_in ? stream : copy;  // drains it
        if (slot_free[k % 2] && (e = hipStreamWaitEvent(first, slot_free[k % 2], 0)))
            return latch(p, e);
        if (is_in) {
            if ((e = copies(pieces)) != hipSuccess) return latch(p, e);
        } else {
            (void)hipGetLastError();
            if ((e = aqua::launch_swap(Lk, stream, &p->stats.launches)) != hipSuccess)
                return latch(p, e);
        }
        if ((e = hipEventRecord(e1, first)) != hipSuccess) return latch(p, e);
        if ((e = hipStreamWaitEvent(second, e1, 0)) != hipSuccess) return latch(p, e);
        if (is_in) {
            (void)hipGetLastError();
            if ((e = aqua::launch_swap(Lk, stream, &p->stats.launches)) != hipSuccess)
                return latch(p, e);
        } else {
            if ((e = copies(pieces)) != hipSuccess) return latch(p, e);
        }
        if ((e = hipEventRecord(e2, second)) != hipSuccess) return latch(p, e);
        slot_free[k % 2] = e2;
        if (!is_in) last_copy = e2;
    }
    // The call completes on its own stream: after the last copy.
    if (last_copy && (e = hipStreamWaitEvent(stream, last_copy, 0)) != hipSuccess)
        return latch(p, e);
    return AQUA_OK;
}

// Link copies on the direction's SDMA engine.  Each layer group is one job
// of the LinkEngine, queued on the engine during this call and released by
// a one-lane kernel on the call's stream; the stream waits on the engine's
// completed-job count where it needs copies done.  Swap-out: group k's job
// is released after its gather; the gather into a slot waits until the job
// that last used the slot (two jobs back) has completed, and the call ends
// after its last job.  Swap-in: the first two jobs are released after the
// call's earlier work, job k + 2 after the scatter of job k, which shares
// its slot; each scatter waits for its own job.
aqua_status enqueue_staged_engine(aqua_kv_pool* p, bool is_in, const void* buf,
                                  hipStream_t stream, const RunDesc* descs, uint32_t ndesc,
                                  uint64_t slot, uint32_t G, uint32_t l_begin, uint32_t l_end) {
    aqua::LinkEngine& w = p->link[is_in];
    const uint32_t K = (l_end - l_begin + G - 1) / G;
    std::vector<aqua::LinkPiece> pieces;
    auto group = [&](uint32_t k, uint32_t* l0, uint32_t* nl) {
        *l0 = l_begin + k * G;
        *nl = std::min<uint32_t>(G, l_end - *l0);
        return p->staging[is_in] + (k % 2) * slot;
    };
    uint64_t submitted = 0;  // completed-job count that covers this call's jobs so far
    auto submit = [&](uint32_t k, int64_t** flag) {
        uint32_t l0, nl;
        uint8_t* s = group(k, &l0, &nl);
        stage_pieces(p, !is_in, buf, s, G, l0, nl, &pieces);
        const uint64_t job = w.submit(pieces, flag);
        submitted = job + 1;
        return job;
    };
    // A later step failed with no flag held: the jobs already released still
    // run, and the call returns once they and the stream's work have ended.
    auto fail = [&](hipError_t e) {
        (void)hipStreamSynchronize(stream);
        (void)hipGetLastError();
        w.wait_published(submitted);
        return latch(p, e);
    };
    auto kernel = [&](uint32_t k) {
        uint32_t l0, nl;
        uint8_t* s = group(k, &l0, &nl);
        (void)hipGetLastError();
        return aqua::launch_swap(slot_launch(p, is_in, s, descs, ndesc, l0, nl), stream,
                                 &p->stats.launches);
    };
    // A flag is held from its job's submission until its release kernel is
    // enqueued; a failure in between hands it to fail_held.
    hipError_t e = hipSuccess;
    if (!is_in) {
        uint64_t first = 0, job = 0;
        for (uint32_t k = 0; k < K; ++k) {
            if (k >= 2 && (e = w.stream_wait(stream, first + k - 1)) != hipSuccess)
                return fail(e);
            if ((e = kernel(k)) != hipSuccess) return fail(e);
            int64_t* flag = nullptr;
            job = submit(k, &flag);
            if (k == 0) first = job;
            if ((e = release_flags(p, flag, nullptr, stream)) != hipSuccess)
                return fail_held(p, w, stream, &flag, 1, e);
        }
        if ((e = w.stream_wait(stream, job + 1)) != hipSuccess) return fail(e);
    } else {
        int64_t* held[2] = {nullptr, nullptr};
        const uint64_t first = submit(0, &held[0]);
        if (K > 1) (void)submit(1, &held[1]);
        if ((e = release_flags(p, held[0], held[1], stream)) != hipSuccess)
            return fail_held(p, w, stream, held, 2, e);
        for (uint32_t k = 0; k < K; ++k) {
            if ((e = w.stream_wait(stream, first + k + 1)) != hipSuccess) return fail(e);
            if ((e = kernel(k)) != hipSuccess) return fail(e);
            if (k + 2 < K) {
                int64_t* flag = nullptr;
                (void)submit(k + 2, &flag);
                if ((e = release_flags(p, flag, nullptr, stream)) != hipSuccess)
                    return fail_held(p, w, stream, &flag, 1, e);
            }
        }
    }
    return AQUA_OK;
}

aqua_status enqueue_staged(aqua_kv_pool* p, bool is_in, const void* buf, hipStream_t stream,
                           const RunDesc* descs, uint32_t ndesc, uint64_t slot, uint32_t G,
                           uint32_t l_begin, uint32_t l_end, Outstanding* rec) {
    if (p->link[is_in].running())
        return enqueue_staged_engine(p, is_in, buf, stream, descs, ndesc, slot, G, l_begin,
                                     l_end);
    return enqueue_staged_runtime(p, is_in, buf, stream, descs, ndesc, slot, G, l_begin, l_end,
                                  rec);
}

aqua_status do_swap(aqua_kv_pool* p, bool is_in, uint32_t num_seqs,
                    const int32_t* ids, const uint64_t* offs, const void* buf,
                    uint64_t buf_bytes, const uint64_t* img_offsets,
                    const aqua_swap_range* range, int32_t target, void* stream_ptr,
                    uint64_t* ticket_out, bool noalloc = false) {
    if (!p) return AQUA_ERR_INVALID;
    if (p->sticky != hipSuccess) return AQUA_ERR_STATE;
    const auto t0 = std::chrono::steady_clock::now();

    aqua::CallArgs a;
    a.num_seqs = num_seqs;
    a.ids = ids;
    a.offs = offs;
    a.img_offsets = img_offsets;
    a.buf = (uintptr_t)buf;
    a.buf_bytes = buf_bytes;
    a.is_in = is_in;
    if (range) {
        a.img_blocks = range->img_blocks;
        a.first_layer = range->first_layer;
        a.num_layers = range->num_layers;
    }
    aqua_status st = (target == AQUA_TARGET_DEVICE || target == AQUA_TARGET_HOST)
                         ? aqua::validate_call(p->shape, a, p->marks)
                         : AQUA_ERR_INVALID;
    if (st == AQUA_ERR_INVALID) return st;
    const uint64_t total = num_seqs ? offs[num_seqs] : 0;
    p->call_blocks = total;

    DeviceGuard dg(p->device);
    if (!dg.ok) {
        (void)hipGetLastError();
        return AQUA_ERR_HIP;  // nothing enqueued: not latched
    }

    uint8_t* dbuf = nullptr;
    if (total) {
        const aqua_status pc = resolve_buffer(p, buf, buf_bytes, target, &dbuf);
        if (pc != AQUA_OK) return pc;
    }
    if (st != AQUA_OK) return st;

    hipStream_t stream = (hipStream_t)stream_ptr;
    st = poll(p);
    if (st != AQUA_OK) return st;

    const uint32_t lane = lane_for(p, stream);
    const uint64_t ticket = p->next_ticket;
    // The allocation-free form moves a host image zero-copy: the staged
    // path needs the library's slots and copy engines.
    const bool staged = target == AQUA_TARGET_HOST && p->host_path == AQUA_HOST_STAGED &&
                        total && !noalloc;
    const uint32_t l_begin = a.first_layer;
    const uint32_t l_count = a.num_layers ? a.num_layers : p->shape.L;

    // Plan.  The staged path plans the concatenated table as one packed
    // sequence (its layout in the HBM slots).
    p->plan.clear();
    uint64_t slot = 0;
    uint32_t G = 0;
    if (staged) {
        const uint64_t per_layer = total * p->shape.C;
        G = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(l_count, p->slot_target / per_layer));
        slot = (uint64_t)G * per_layer;
        // Descriptors for the slot layout: sequence s at G * first_s * C.
        p->sseq.clear();
        p->slot_offsets.assign(num_seqs, 0);
        for (uint32_t k = 0; k < num_seqs; ++k) {
            p->slot_offsets[k] = (uint64_t)G * offs[k] * p->shape.C;
            if (offs[k + 1] > offs[k])
                p->sseq.push_back({aqua::image_offset(p->shape, a, k), offs[k],
                                   offs[k + 1] - offs[k], aqua::image_blocks(a, k)});
        }
        // Slot images are dense: [G][n_s][C].
        aqua::CallArgs c = a;
        c.img_offsets = p->slot_offsets.data();
        c.img_blocks = nullptr;
        aqua::plan_runs(p->shape, c, p->unit_bytes, &p->plan);
        st = ensure_staging(p, is_in, 2 * slot);
        if (st == AQUA_OK) st = ensure_link(p, is_in);
        if (st != AQUA_OK) return st;
    } else {
        aqua::plan_runs(p->shape, a, p->unit_bytes, &p->plan);
    }
    const aqua::RunOrder order =
        AQUA_SORT_RUNS ? aqua::run_order(is_in, p->shape.C, total, p->shape.N, num_seqs)
                       : aqua::RunOrder::kTable;
    if (order == aqua::RunOrder::kSortedDealt)
        aqua::sort_by_block(&p->plan, p->shape.N, &p->sort_counts, &p->sort_tmp);
    const bool dealt = order != aqua::RunOrder::kTable;
    if (dealt) aqua::interleave_runs(&p->plan, aqua::kXcdWays, &p->sort_tmp);
    aqua::image_ranges(p->shape, a, &p->ranges);
    for (auto& r : p->ranges) {  // tracked by the caller's address of the buffer
        r.first += a.buf;
        r.second += a.buf;
    }
    const std::pair<uint64_t, uint64_t> stage_range{
        (uint64_t)(uintptr_t)p->staging[is_in],
        (uint64_t)(uintptr_t)p->staging[is_in] + 2 * slot};

    // Reserve descriptor space before registering the ticket: a reservation
    // may wait on earlier tickets.
    uint64_t ring_off = 0;
    const uint64_t dbytes = p->plan.size() * sizeof(RunDesc);
    uint64_t waited_ns = 0;
    Outstanding rec{ticket, nullptr, {}};
    // The allocation-free form: descriptors beyond the scratch are refused
    // before anything happens, and the call's event is a recycled one.
    const std::pair<uint64_t, uint64_t> scratch_range{
        (uint64_t)(uintptr_t)p->scratch, (uint64_t)(uintptr_t)p->scratch + dbytes};
    if (noalloc) {
        if (dbytes > kScratchBytes) return AQUA_ERR_CAPACITY;
        if (!p->scratch) return AQUA_ERR_HIP;
        const auto w0 = std::chrono::steady_clock::now();
        st = take_event_noalloc(p, &rec.ev);
        waited_ns += (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
                         std::chrono::steady_clock::now() - w0)
                         .count();
        if (st != AQUA_OK) return st;
    }
    auto give_back = [&]() {
        if (rec.ev) p->spare_events.push_back(rec.ev);
        rec.ev = nullptr;
    };
    if (dbytes) {
        const auto w0 = std::chrono::steady_clock::now();
        st = ring_reserve(p, dbytes, &ring_off, !noalloc);
        waited_ns += (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
                         std::chrono::steady_clock::now() - w0)
                         .count();
        if (st != AQUA_OK) {
            give_back();
            return st;
        }
    }

    // Accesses: swap-out reads the table's blocks and writes the images,
    // swap-in reads the images and writes the blocks; the staged path also
    // writes its slots, and the allocation-free form the device scratch (so
    // that two such calls on one pool never overlap).
    HazardTracker::Access acc;
    if (is_in) {
        acc.blocks_written = ids;
        acc.n_blocks_written = (size_t)total;
        acc.ranges_read = p->ranges.data();
        acc.n_ranges_read = p->ranges.size();
        if (staged) {
            acc.ranges_written = &stage_range;
            acc.n_ranges_written = 1;
        } else if (noalloc && dbytes) {
            acc.ranges_written = &scratch_range;
            acc.n_ranges_written = 1;
        }
    } else {
        acc.blocks_read = ids;
        acc.n_blocks_read = (size_t)total;
        if (staged) p->ranges.push_back(stage_range);
        if (noalloc && dbytes) p->ranges.push_back(scratch_range);
        acc.ranges_written = p->ranges.data();
        acc.n_ranges_written = p->ranges.size();
    }
    p->stats.waits_elided += p->tracker.issue(ticket, lane, acc, &p->deps);
    p->next_ticket++;

    for (const HazardTracker::Dep& d : p->deps) {
        hipEvent_t ev = event_of(p, d.ticket);
        if (!ev) continue;
        const hipError_t e = hipStreamWaitEvent(stream, ev, 0);
        if (e != hipSuccess) return fail_enqueued(stream, latch(p, e));
        p->stats.waits_inserted++;
    }

    if (dbytes) {
        std::memcpy(p->ring_host + ring_off, p->plan.data(), dbytes);
        hipError_t e = hipSuccess;
        const uint8_t* descs = p->ring_host_dev + ring_off;
        if (noalloc) {
            descs = p->scratch;
            e = upload_to(p->ring_host_dev + ring_off, p->scratch, dbytes, stream);
        } else if (staged || AQUA_DESC_DEVICE) {
            descs = p->ring_dev + ring_off;
            e = upload_descs(p, ring_off, dbytes, stream);
        }
        if (e != hipSuccess) return fail_enqueued(stream, latch(p, e));
        if (staged) {
            st = enqueue_staged(p, is_in, buf, stream, reinterpret_cast<const RunDesc*>(descs),
                                (uint32_t)p->plan.size(), slot, G, l_begin, l_begin + l_count,
                                &rec);
            if (st != AQUA_OK) {
                // The runtime carrier's copies run on the library's copy stream.
                if (p->copy[is_in]) (void)hipStreamSynchronize(p->copy[is_in]);
                return fail_enqueued(stream, st);
            }
        } else {
            aqua::SwapLaunch L =
                make_launch(p, is_in, dbuf, reinterpret_cast<const RunDesc*>(descs),
                            (uint32_t)p->plan.size(), target, l_begin, l_count);
            L.xcd_order = target == AQUA_TARGET_DEVICE && aqua::xcd_unit_order(p->shape.C, dealt);
            (void)hipGetLastError();
            e = aqua::launch_swap(L, stream, &p->stats.launches);
            if (e != hipSuccess) return fail_enqueued(stream, latch(p, e));
        }
    }

    hipError_t e = rec.ev ? hipSuccess : take_event(p, &rec.ev);
    if (e == hipSuccess) e = hipEventRecord(rec.ev, stream);
    if (e != hipSuccess) return fail_enqueued(stream, latch(p, e));
    p->outstanding[lane].push_back(std::move(rec));
    if (dbytes) p->ring_uses.push_back({ring_off, ring_off + ((dbytes + 255) & ~255ull), ticket});

    const uint64_t moved = (uint64_t)l_count * total * p->shape.C;
    if (is_in) {
        p->stats.calls_in++;
        p->stats.bytes_in += moved;
    } else {
        p->stats.calls_out++;
        p->stats.bytes_out += moved;
    }
    if (target == AQUA_TARGET_HOST) p->stats.bytes_host += moved;
    p->stats.descriptors += p->plan.size();
    const uint64_t total_ns = (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
                                  std::chrono::steady_clock::now() - t0)
                                  .count();
    // Reserving descriptor space blocks only when the ring is full; that
    // back-pressure is reported apart from the call's own host work.
    p->stats.wait_ns += waited_ns;
    p->stats.host_ns += total_ns > waited_ns ? total_ns - waited_ns : 0;
    if (ticket_out) *ticket_out = ticket;
    return AQUA_OK;
}

aqua_status do_migrate(aqua_kv_pool* p, const void* src, uint64_t src_bytes, int32_t src_target,
                       void* dst, uint64_t dst_bytes, int32_t dst_target, uint32_t n,
                       const uint64_t* so, const uint64_t* dof, const uint64_t* len,
                       void* stream_ptr, uint64_t* ticket_out) {
    if (!p) return AQUA_ERR_INVALID;
    if (p->sticky != hipSuccess) return AQUA_ERR_STATE;
    const auto t0 = std::chrono::steady_clock::now();
    auto valid_target = [](int32_t t) {
        return t == AQUA_TARGET_DEVICE || t == AQUA_TARGET_HOST;
    };
    aqua_status st = (valid_target(src_target) && valid_target(dst_target))
                         ? aqua::validate_migrate((uintptr_t)src, src_bytes, (uintptr_t)dst,
                                                  dst_bytes, n, so, dof, len)
                         : AQUA_ERR_INVALID;
    if (st == AQUA_ERR_INVALID) return st;
    uint64_t moved = 0;
    for (uint32_t k = 0; k < n; ++k) moved += len[k];

    DeviceGuard dg(p->device);
    if (!dg.ok) {
        (void)hipGetLastError();
        return AQUA_ERR_HIP;
    }
    uint8_t* dsrc = nullptr;
    uint8_t* ddst = nullptr;
    if (moved) {
        aqua_status pc = resolve_buffer(p, src, src_bytes, src_target, &dsrc);
        if (pc == AQUA_OK) pc = resolve_buffer(p, dst, dst_bytes, dst_target, &ddst);
        if (pc != AQUA_OK) return pc;
    }
    if (st != AQUA_OK) return st;

    hipStream_t stream = (hipStream_t)stream_ptr;
    st = poll(p);
    if (st != AQUA_OK) return st;
    // Between the HBM region and pinned host memory the ranges go to the
    // direction's copy engine when it has one, one engine copy per range;
    // otherwise the range-copy kernel moves them.
    const int link_dir = (src_target == AQUA_TARGET_DEVICE && dst_target == AQUA_TARGET_HOST)   ? 0
                         : (src_target == AQUA_TARGET_HOST && dst_target == AQUA_TARGET_DEVICE) ? 1
                                                                                                : -1;
    if (moved && link_dir >= 0) {
        st = ensure_link(p, link_dir);
        if (st != AQUA_OK) return st;
    }
    const bool engine = moved && link_dir >= 0 && p->link[link_dir].running();
    const uint32_t lane = lane_for(p, stream);
    const uint64_t ticket = p->next_ticket;

    std::vector<aqua::CopyDesc> pieces;
    if (!engine) aqua::plan_copies(n, so, dof, len, kDefaultUnitBytes, &pieces);
    p->ranges.clear();
    std::vector<std::pair<uint64_t, uint64_t>> wr;
    for (uint32_t k = 0; k < n; ++k) {
        if (!len[k]) continue;
        p->ranges.emplace_back((uint64_t)(uintptr_t)src + so[k], (uint64_t)(uintptr_t)src + so[k] + len[k]);
        wr.emplace_back((uint64_t)(uintptr_t)dst + dof[k], (uint64_t)(uintptr_t)dst + dof[k] + len[k]);
    }
    uint64_t ring_off = 0;
    const uint64_t dbytes = pieces.size() * sizeof(aqua::CopyDesc);
    uint64_t waited_ns = 0;
    if (dbytes) {
        const auto w0 = std::chrono::steady_clock::now();
        st = ring_reserve(p, dbytes, &ring_off);
        waited_ns = (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
                        std::chrono::steady_clock::now() - w0)
                        .count();
        if (st != AQUA_OK) return st;
    }
    HazardTracker::Access acc;
    acc.ranges_read = p->ranges.data();
    acc.n_ranges_read = p->ranges.size();
    acc.ranges_written = wr.data();
    acc.n_ranges_written = wr.size();
    p->stats.waits_elided += p->tracker.issue(ticket, lane, acc, &p->deps);
    p->next_ticket++;
    for (const HazardTracker::Dep& d : p->deps) {
        hipEvent_t ev = event_of(p, d.ticket);
        if (!ev) continue;
        const hipError_t e = hipStreamWaitEvent(stream, ev, 0);
        if (e != hipSuccess) return fail_enqueued(stream, latch(p, e));
        p->stats.waits_inserted++;
    }
    Outstanding rec{ticket, nullptr, {}};
    if (engine) {
        std::vector<aqua::LinkPiece> copies;
        for (uint32_t k = 0; k < n; ++k)
            if (len[k])
                copies.push_back({(uint8_t*)dst + dof[k], (const uint8_t*)src + so[k], len[k]});
        aqua::LinkEngine& w = p->link[link_dir];
        int64_t* flag = nullptr;
        const uint64_t job = w.submit(copies, &flag);
        hipError_t e = release_flags(p, flag, nullptr, stream);
        if (e != hipSuccess) return fail_held(p, w, stream, &flag, 1, e);
        if ((e = w.stream_wait(stream, job + 1)) != hipSuccess) {
            const aqua_status st = fail_enqueued(stream, latch(p, e));
            w.wait_published(job + 1);  // the released copies end before the call returns
            return st;
        }
    }
    if (dbytes) {
        // Descriptors go to the device ring: a migration touching host
        // memory keeps the link busy.
        std::memcpy(p->ring_host + ring_off, pieces.data(), dbytes);
        hipError_t e = upload_descs(p, ring_off, dbytes, stream);
        if (e != hipSuccess) return fail_enqueued(stream, latch(p, e));
        const bool host_side = src_target == AQUA_TARGET_HOST || dst_target == AQUA_TARGET_HOST;
        (void)hipGetLastError();
        e = aqua::launch_copy(dsrc, ddst,
                              reinterpret_cast<const aqua::CopyDesc*>(p->ring_dev + ring_off),
                              (uint32_t)pieces.size(),
                              host_side ? p->max_wg[AQUA_TARGET_HOST] : p->max_wg[AQUA_TARGET_DEVICE],
                              stream);
        if (e != hipSuccess) return fail_enqueued(stream, latch(p, e));
    }
    hipError_t e = take_event(p, &rec.ev);
    if (e == hipSuccess) e = hipEventRecord(rec.ev, stream);
    if (e != hipSuccess) return fail_enqueued(stream, latch(p, e));
    p->outstanding[lane].push_back(std::move(rec));
    if (dbytes) p->ring_uses.push_back({ring_off, ring_off + ((dbytes + 255) & ~255ull), ticket});
    p->stats.calls_migrate++;
    p->stats.bytes_migrated += moved;
    if (src_target == AQUA_TARGET_HOST || dst_target == AQUA_TARGET_HOST) p->stats.bytes_host += moved;
    const uint64_t total_ns = (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
                                  std::chrono::steady_clock::now() - t0)
                                  .count();
    p->stats.wait_ns += waited_ns;
    p->stats.host_ns += total_ns > waited_ns ? total_ns - waited_ns : 0;
    if (ticket_out) *ticket_out = ticket;
    return AQUA_OK;
}

// Moves the tensors in `moves` (handle, destination offset) from region
// `from` to the other one as one migration on the pool; on success the
// tensors point at their new ranges and their old ranges are released.
aqua_status swap_move(aqua_swap_space* s, int from,
                      const std::vector<std::pair<uint64_t, uint64_t>>& moves, void* stream,
                      uint64_t* ticket) {
    const int to = 1 - from;
    std::vector<uint64_t> so, dof, len;
    for (const auto& m : moves) {
        const auto& t = s->tensors.at(m.first);
        so.push_back(t.off);
        dof.push_back(m.second);
        len.push_back(t.bytes);
    }
    uint64_t tk = 0;
    const aqua_status st =
        do_migrate(s->pool, s->region[from], s->region_bytes[from], from, s->region[to],
                   s->region_bytes[to], to, (uint32_t)moves.size(), so.data(), dof.data(),
                   len.data(), stream, &tk);
    if (st != AQUA_OK) {
        for (const auto& m : moves) s->ranges[to].free(m.second);
        return st;
    }
    for (const auto& m : moves) {
        auto& t = s->tensors.at(m.first);
        s->ranges[from].free(t.off);
        t.target = to;
        t.off = m.second;
    }
    if (ticket) *ticket = tk;
    return AQUA_OK;
}

}  // namespace


extern "C" {

aqua_status aqua_kv_pool_create(const aqua_kv_desc* desc, void* pool_base,
                                uint64_t pool_bytes, aqua_kv_pool_t* out) {
    TraceRange trace("aqua_kv_pool_create");
    if (!out) return AQUA_ERR_INVALID;
    aqua::Shape s;
    aqua_status st = aqua::make_shape(desc, &s);
    if (st != AQUA_OK) return st;
    if (!pool_base || ((uintptr_t)pool_base % 16)) return AQUA_ERR_INVALID;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return AQUA_ERR_HIP;
    }
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof(attr));
    if (hipPointerGetAttributes(&attr, pool_base) != hipSuccess) {
        (void)hipGetLastError();
        return AQUA_ERR_INVALID;
    }
    if (attr.type != hipMemoryTypeDevice || attr.device != dev) return AQUA_ERR_INVALID;
    hipDeviceptr_t rbase = nullptr;
    size_t rsize = 0;
    if (hipMemGetAddressRange(&rbase, &rsize, (hipDeviceptr_t)pool_base) != hipSuccess) {
        (void)hipGetLastError();
        return AQUA_ERR_INVALID;
    }
    const uintptr_t b = (uintptr_t)rbase, x = (uintptr_t)pool_base;
    if (x < b || pool_bytes > rsize - (x - b)) return AQUA_ERR_INVALID;
    if (pool_bytes < s.pool_bytes) return AQUA_ERR_CAPACITY;

    aqua_kv_pool* p = new (std::nothrow) aqua_kv_pool();
    if (!p) return AQUA_ERR_HIP;
    p->shape = s;
    p->device = dev;
    p->base = (uint8_t*)pool_base;
    p->bytes = pool_bytes;
    p->tracker.reset(s.N);
    // Work per workgroup; capped so that a run's 16-byte vector count fits
    // the kernels' 32-bit counters.
    p->unit_bytes = env_u64("AQUA_UNIT_BYTES", kDefaultUnitBytes);
    if (!p->unit_bytes) p->unit_bytes = kDefaultUnitBytes;
    if (p->unit_bytes > aqua::kMaxChunkBytes) p->unit_bytes = aqua::kMaxChunkBytes;
    p->slot_target = env_u64("AQUA_STAGE_SLOT_BYTES", kDefaultSlotBytes);
    p->fail_release_at = env_u64("AQUA_FAIL_RELEASE_AT", ~0ull);
    st = alloc_rings(p, env_u64("AQUA_RING_BYTES", kDefaultRingBytes));
    if (st == AQUA_OK && warm_kernels(p) != hipSuccess) st = AQUA_ERR_HIP;
    // Set-up of the allocation-free entry point: this device's scratch
    // address, and the events its calls recycle.
    if (st == AQUA_OK && !(p->scratch = scratch_address(dev))) st = AQUA_ERR_HIP;
    for (uint32_t k = 0; st == AQUA_OK && k < kPoolEvents; ++k) {
        hipEvent_t ev = nullptr;
        if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
            (void)hipGetLastError();
            st = AQUA_ERR_HIP;
        } else {
            p->spare_events.push_back(ev);
        }
    }
    if (st != AQUA_OK) {
        for (hipEvent_t ev : p->spare_events) (void)hipEventDestroy(ev);
        free_rings(p);
        delete p;
        return st;
    }
    *out = p;
    return AQUA_OK;
}

aqua_status aqua_kv_pool_destroy(aqua_kv_pool_t p) {
    TraceRange trace("aqua_kv_pool_destroy");
    if (!p) return AQUA_ERR_INVALID;
    aqua_status st = AQUA_OK;
    {
        DeviceGuard dg(p->device);
        if (p->sticky == hipSuccess) st = wait_all(p);
        if (p->sticky != hipSuccess) {
            // Calls issued before the failure may still run: let them end
            // before their slots, rings and events are freed.  (The failed
            // call itself waited for its own work before returning.)
            for (auto& q : p->outstanding)
                for (const Outstanding& o : q) (void)hipEventSynchronize(o.ev);
            (void)hipGetLastError();
        }
        // After a failure a link thread may find a job whose flag is still
        // held; it releases it from the host so that the engine drains.
        for (int dir = 0; dir < 2; ++dir) p->link[dir].stop(p->sticky != hipSuccess);
        if (p->hsa_up) aqua::link_release();
        p->hsa_up = false;
        for (auto& q : p->outstanding)
            for (const Outstanding& o : q) {
                (void)hipEventDestroy(o.ev);
                for (hipEvent_t e : o.aux) (void)hipEventDestroy(e);
            }
        for (hipEvent_t ev : p->spare_events) (void)hipEventDestroy(ev);
        free_rings(p);
        for (int dir = 0; dir < 2; ++dir) {
            if (p->staging[dir]) (void)hipFree(p->staging[dir]);
            if (p->copy[dir]) (void)hipStreamDestroy(p->copy[dir]);
        }
        if (p->sticky != hipSuccess) st = AQUA_ERR_HIP;
    }
    delete p;
    return st;
}

aqua_status aqua_swap_out(aqua_kv_pool_t pool, uint32_t num_seqs, const int32_t* block_ids,
                          const uint64_t* seq_offsets, void* dst, uint64_t dst_bytes,
                          const uint64_t* img_offsets, int32_t target, void* stream,
                          uint64_t* ticket) {
    TraceRange trace("aqua_swap_out");
    return do_swap(pool, false, num_seqs, block_ids, seq_offsets, dst, dst_bytes, img_offsets,
                   nullptr, target, stream, ticket);
}

aqua_status aqua_swap_in(aqua_kv_pool_t pool, uint32_t num_seqs, const int32_t* block_ids,
                         const uint64_t* seq_offsets, const void* src, uint64_t src_bytes,
                         const uint64_t* img_offsets, int32_t target, void* stream,
                         uint64_t* ticket) {
    TraceRange trace("aqua_swap_in");
    return do_swap(pool, true, num_seqs, block_ids, seq_offsets, src, src_bytes, img_offsets,
                   nullptr, target, stream, ticket);
}

aqua_status aqua_swap_out_ex(aqua_kv_pool_t pool, uint32_t num_seqs, const int32_t* block_ids,
                             const uint64_t* seq_offsets, void* dst, uint64_t dst_bytes,
                             const uint64_t* img_offsets, const aqua_swap_range* range,
                             int32_t target, void* stream, uint64_t* ticket) {
    TraceRange trace("aqua_swap_out_ex");
    return do_swap(pool, false, num_seqs, block_ids, seq_offsets, dst, dst_bytes, img_offsets,
                   range, target, stream, ticket);
}

aqua_status aqua_swap_in_ex(aqua_kv_pool_t pool, uint32_t num_seqs, const int32_t* block_ids,
                            const uint64_t* seq_offsets, const void* src, uint64_t src_bytes,
                            const uint64_t* img_offsets, const aqua_swap_range* range,
                            int32_t target, void* stream, uint64_t* ticket) {
    TraceRange trace("aqua_swap_in_ex");
    return do_swap(pool, true, num_seqs, block_ids, seq_offsets, src, src_bytes, img_offsets,
                   range, target, stream, ticket);
}

aqua_status aqua_swap_noalloc(aqua_kv_pool_t pool, int32_t direction, uint32_t num_seqs,
                              const int32_t* block_ids, const uint64_t* seq_offsets, void* buf,
                              uint64_t buf_bytes, const uint64_t* img_offsets, int32_t target,
                              void* stream, uint64_t* ticket) {
    TraceRange trace("aqua_swap_noalloc");
    if (direction != 0 && direction != 1) return AQUA_ERR_INVALID;
    return do_swap(pool, direction == 1, num_seqs, block_ids, seq_offsets, buf, buf_bytes,
                   img_offsets, nullptr, target, stream, ticket, true);
}

aqua_status aqua_migrate(aqua_kv_pool_t pool, const void* src, uint64_t src_bytes,
                         int32_t src_target, void* dst, uint64_t dst_bytes, int32_t dst_target,
                         uint32_t n, const uint64_t* src_offsets, const uint64_t* dst_offsets,
                         const uint64_t* lengths, void* stream, uint64_t* ticket) {
    TraceRange trace("aqua_migrate");
    return do_migrate(pool, src, src_bytes, src_target, dst, dst_bytes, dst_target, n,
                      src_offsets, dst_offsets, lengths, stream, ticket);
}

aqua_status aqua_sync(aqua_kv_pool_t p, uint64_t ticket) {
    TraceRange trace("aqua_sync");
    if (!p) return AQUA_ERR_INVALID;
    if (ticket >= p->next_ticket) return AQUA_ERR_INVALID;
    if (p->sticky != hipSuccess) return AQUA_ERR_HIP;
    DeviceGuard dg(p->device);
    aqua_status st = ticket ? wait_ticket(p, ticket) : wait_all(p);
    if (st == AQUA_OK && p->sticky != hipSuccess) st = AQUA_ERR_HIP;
    return st;
}

aqua_status aqua_stream_wait(aqua_kv_pool_t p, uint64_t ticket, void* stream) {
    TraceRange trace("aqua_stream_wait");
    if (!p) return AQUA_ERR_INVALID;
    if (ticket >= p->next_ticket) return AQUA_ERR_INVALID;
    if (p->sticky != hipSuccess) return AQUA_ERR_STATE;
    DeviceGuard dg(p->device);
    aqua_status st = poll(p);
    if (st != AQUA_OK) return st;
    for (uint32_t m = 0; m < p->outstanding.size(); ++m) {
        const auto& q = p->outstanding[m];
        if (q.empty()) continue;
        hipEvent_t ev = nullptr;
        if (ticket == 0) {
            ev = q.back().ev;
        } else if (p->tracker.lane_of(ticket) == m) {
            ev = event_of(p, ticket);
        }
        if (!ev) continue;
        const hipError_t e = hipStreamWaitEvent((hipStream_t)stream, ev, 0);
        if (e != hipSuccess) return latch(p, e);
    }
    return AQUA_OK;
}

aqua_status aqua_query(aqua_kv_pool_t p, uint64_t ticket) {
    if (!p || ticket == 0 || ticket >= p->next_ticket) return AQUA_ERR_INVALID;
    if (p->sticky != hipSuccess) return AQUA_ERR_STATE;
    DeviceGuard dg(p->device);
    const aqua_status st = poll(p);
    if (st != AQUA_OK) return st;
    return p->tracker.done(ticket) ? 1 : 0;
}

aqua_status aqua_kv_pool_set_max_workgroups(aqua_kv_pool_t p, int32_t target,
                                            uint32_t max_workgroups) {
    if (!p || (target != AQUA_TARGET_DEVICE && target != AQUA_TARGET_HOST))
        return AQUA_ERR_INVALID;
    p->max_wg[target] = max_workgroups;
    return AQUA_OK;
}

aqua_status aqua_kv_pool_set_host_path(aqua_kv_pool_t p, int32_t path) {
    if (!p || (path != AQUA_HOST_ZERO_COPY && path != AQUA_HOST_STAGED)) return AQUA_ERR_INVALID;
    p->host_path = path;
    return AQUA_OK;
}

aqua_status aqua_kv_pool_set_link_engine(aqua_kv_pool_t p, int32_t dir, int32_t engine) {
    if (!p || (dir != 0 && dir != 1) ||
        !(engine == AQUA_LINK_AUTO || engine == AQUA_LINK_RUNTIME || (engine >= 0 && engine <= 15)))
        return AQUA_ERR_INVALID;
    if (p->sticky != hipSuccess) return AQUA_ERR_STATE;
    DeviceGuard dg(p->device);
    const aqua_status st = wait_all(p);
    if (st != AQUA_OK) return st;
    p->link[dir].stop();
    p->link_request[dir] = engine;
    p->link_used[dir] = AQUA_LINK_AUTO;
    return AQUA_OK;
}

aqua_status aqua_kv_pool_get_link_engine(aqua_kv_pool_t p, int32_t dir, int32_t* engine) {
    if (!p || (dir != 0 && dir != 1) || !engine) return AQUA_ERR_INVALID;
    *engine = p->link_used[dir];
    return AQUA_OK;
}

aqua_status aqua_pool_stats_get(aqua_kv_pool_t p, aqua_pool_stats* out) {
    if (!p || !out) return AQUA_ERR_INVALID;
    *out = p->stats;
    return AQUA_OK;
}

aqua_status aqua_swap_space_create(aqua_kv_pool_t pool, uint64_t device_bytes,
                                   uint64_t host_bytes, aqua_swap_space_t* out) {
    TraceRange trace("aqua_swap_space_create");
    if (!pool || !out) return AQUA_ERR_INVALID;
    if (pool->sticky != hipSuccess) return AQUA_ERR_STATE;
    DeviceGuard dg(pool->device);
    if (!dg.ok) {
        (void)hipGetLastError();
        return AQUA_ERR_HIP;
    }
    aqua_swap_space* s = new (std::nothrow) aqua_swap_space();
    if (!s) return AQUA_ERR_HIP;
    s->pool = pool;
    hipError_t e = hipSuccess;
    if (device_bytes) e = hipMalloc((void**)&s->region[AQUA_TARGET_DEVICE], device_bytes);
    if (e == hipSuccess && host_bytes)
        e = hipHostMalloc((void**)&s->region[AQUA_TARGET_HOST], host_bytes, hipHostMallocMapped);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        if (s->region[AQUA_TARGET_DEVICE]) (void)hipFree(s->region[AQUA_TARGET_DEVICE]);
        delete s;
        return AQUA_ERR_HIP;
    }
    s->region_bytes[AQUA_TARGET_DEVICE] = device_bytes;
    s->region_bytes[AQUA_TARGET_HOST] = host_bytes;
    s->ranges[AQUA_TARGET_DEVICE].reset(device_bytes, kSwapAlign);
    s->ranges[AQUA_TARGET_HOST].reset(host_bytes, kSwapAlign);
    *out = s;
    return AQUA_OK;
}

aqua_status aqua_swap_space_destroy(aqua_swap_space_t s) {
    TraceRange trace("aqua_swap_space_destroy");
    if (!s) return AQUA_ERR_INVALID;
    aqua_status st = AQUA_OK;
    {
        DeviceGuard dg(s->pool->device);
        if (s->pool->sticky == hipSuccess) st = wait_all(s->pool);
        if (s->region[AQUA_TARGET_DEVICE]) (void)hipFree(s->region[AQUA_TARGET_DEVICE]);
        if (s->region[AQUA_TARGET_HOST]) (void)hipHostFree(s->region[AQUA_TARGET_HOST]);
    }
    delete s;
    return st;
}

aqua_status aqua_swap_alloc(aqua_swap_space_t s, uint64_t bytes, uint64_t* handle) {
    if (!s || !handle || !bytes || bytes % 16) return AQUA_ERR_INVALID;
    uint64_t off = 0;
    int32_t target = AQUA_TARGET_DEVICE;
    if (!s->ranges[target].alloc(bytes, &off)) {
        target = AQUA_TARGET_HOST;
        if (!s->ranges[target].alloc(bytes, &off)) return AQUA_ERR_CAPACITY;
    }
    const uint64_t h = s->next_handle++;
    s->tensors[h] = {bytes, target, off};
    *handle = h;
    return AQUA_OK;
}

aqua_status aqua_swap_free(aqua_swap_space_t s, uint64_t handle) {
    if (!s) return AQUA_ERR_INVALID;
    auto it = s->tensors.find(handle);
    if (it == s->tensors.end()) return AQUA_ERR_INVALID;
    s->ranges[it->second.target].free(it->second.off);
    s->tensors.erase(it);
    return AQUA_OK;
}

aqua_status aqua_swap_locate(aqua_swap_space_t s, uint64_t handle, void** ptr, uint64_t* bytes,
                             int32_t* target) {
    if (!s) return AQUA_ERR_INVALID;
    auto it = s->tensors.find(handle);
    if (it == s->tensors.end()) return AQUA_ERR_INVALID;
    const auto& t = it->second;
    if (ptr) *ptr = s->region[t.target] + t.off;
    if (bytes) *bytes = t.bytes;
    if (target) *target = t.target;
    return AQUA_OK;
}

aqua_status aqua_swap_reclaim(aqua_swap_space_t s, uint64_t bytes, void* stream,
                              uint64_t* ticket) {
    TraceRange trace("aqua_swap_reclaim");
    if (!s) return AQUA_ERR_INVALID;
    if (ticket) *ticket = 0;
    auto& dev = s->ranges[AQUA_TARGET_DEVICE];
    auto& host = s->ranges[AQUA_TARGET_HOST];
    const bool all = bytes == UINT64_MAX;
    uint64_t freed = dev.free_bytes();
    std::vector<std::pair<uint64_t, uint64_t>> moves;
    for (const auto& kv : s->tensors) {
        if (!all && freed >= bytes) break;
        if (kv.second.target != AQUA_TARGET_DEVICE) continue;
        uint64_t off = 0;
        if (!host.alloc(kv.second.bytes, &off)) {
            for (const auto& m : moves) host.free(m.second);
            return AQUA_ERR_CAPACITY;
        }
        moves.emplace_back(kv.first, off);
        freed += dev.granted(kv.second.off);
    }
    if (moves.empty()) return AQUA_OK;
    return swap_move(s, AQUA_TARGET_DEVICE, moves, stream, ticket);
}

aqua_status aqua_swap_restore(aqua_swap_space_t s, void* stream, uint64_t* ticket) {
    TraceRange trace("aqua_swap_restore");
    if (!s) return AQUA_ERR_INVALID;
    if (ticket) *ticket = 0;
    auto& dev = s->ranges[AQUA_TARGET_DEVICE];
    std::vector<std::pair<uint64_t, uint64_t>> moves;
    for (const auto& kv : s->tensors) {
        if (kv.second.target != AQUA_TARGET_HOST) continue;
        uint64_t off = 0;
        if (dev.alloc(kv.second.bytes, &off)) moves.emplace_back(kv.first, off);
    }
    if (moves.empty()) return AQUA_OK;
    return swap_move(s, AQUA_TARGET_HOST, moves, stream, ticket);
}

aqua_status aqua_swap_usage(aqua_swap_space_t s, uint64_t* device_free, uint64_t* host_free,
                            uint64_t* device_tensors, uint64_t* host_tensors) {
    if (!s) return AQUA_ERR_INVALID;
    uint64_t n[2] = {0, 0};
    for (const auto& kv : s->tensors) n[kv.second.target]++;
    if (device_free) *device_free = s->ranges[AQUA_TARGET_DEVICE].free_bytes();
    if (host_free) *host_free = s->ranges[AQUA_TARGET_HOST].free_bytes();
    if (device_tensors) *device_tensors = n[AQUA_TARGET_DEVICE];
    if (host_tensors) *host_tensors = n[AQUA_TARGET_HOST];
    return AQUA_OK;
}

aqua_status aqua_hbm_yardstick(int32_t kind, void* dst, const void* src, uint64_t bytes,
                               void* stream) {
    TraceRange trace("aqua_hbm_yardstick");
    if (kind != AQUA_YARDSTICK_COPY && kind != AQUA_YARDSTICK_READ &&
        kind != AQUA_YARDSTICK_WRITE)
        return AQUA_ERR_INVALID;
    if (bytes % 16 || (uintptr_t)dst % 16 || (uintptr_t)src % 16) return AQUA_ERR_INVALID;
    if (!bytes) return AQUA_OK;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return AQUA_ERR_HIP;
    }
    // [ptr, ptr + n) in one allocation of the current device.
    auto device_range = [dev](const void* ptr, uint64_t n) {
        if (!ptr) return false;
        hipPointerAttribute_t attr;
        std::memset(&attr, 0, sizeof(attr));
        hipDeviceptr_t rbase = nullptr;
        size_t rsize = 0;
        if (hipPointerGetAttributes(&attr, ptr) != hipSuccess ||
            hipMemGetAddressRange(&rbase, &rsize, (hipDeviceptr_t)ptr) != hipSuccess) {
            (void)hipGetLastError();
            return false;
        }
        const uintptr_t b = (uintptr_t)rbase, x = (uintptr_t)ptr;
        return attr.type == hipMemoryTypeDevice && attr.device == dev && x >= b &&
               x - b <= rsize && n <= rsize - (x - b);
    };
    const bool reads = kind != AQUA_YARDSTICK_WRITE;
    const uint64_t dst_bytes = kind == AQUA_YARDSTICK_READ ? 16 : bytes;
    if (!device_range(dst, dst_bytes) || (reads && !device_range(src, bytes)))
        return AQUA_ERR_INVALID;
    if (kind == AQUA_YARDSTICK_COPY) {
        const uintptr_t d = (uintptr_t)dst, q = (uintptr_t)src;
        if (d < q + bytes && q < d + bytes) return AQUA_ERR_INVALID;
    }
    (void)hipGetLastError();
    const hipError_t e =
        aqua::launch_yardstick(kind, (const uint8_t*)src, (uint8_t*)dst, bytes, 0x9E3779B9u,
                               (hipStream_t)stream);
    return e == hipSuccess ? AQUA_OK : AQUA_ERR_HIP;
}

const char* aqua_status_str(aqua_status s) {
    switch (s) {
        case AQUA_OK: return "ok";
        case AQUA_ERR_INVALID: return "invalid argument";
        case AQUA_ERR_RANGE: return "block id out of range";
        case AQUA_ERR_DUPLICATE: return "duplicate destination";
        case AQUA_ERR_CAPACITY: return "image does not fit the buffer";
        case AQUA_ERR_HIP: return "HIP runtime failure";
        case AQUA_ERR_STATE: return "pool unusable after a HIP failure";
        default: return "unknown status";
    }
}

}  // extern "C"
