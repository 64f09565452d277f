// link_engine.hip -- host-link copies on a chosen SDMA engine, ordered against
// HIP streams through a completed-job count in signal memory.
#include "link_engine.h"

#include "aqua_core.h"

#include <hsa/hsa_ext_amd.h>

#include <chrono>

namespace aqua {

namespace {

struct FindGpu {
    uint32_t domain, bus, dev;
    hsa_agent_t found;
    bool hit;
};

hsa_status_t find_gpu(hsa_agent_t a, void* data) {
    FindGpu* f = static_cast<FindGpu*>(data);
    hsa_device_type_t t;
    if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) != HSA_STATUS_SUCCESS ||
        t != HSA_DEVICE_TYPE_GPU)
        return HSA_STATUS_SUCCESS;
    uint32_t bdf = 0, dom = 0;
    if (hsa_agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_BDFID, &bdf) !=
        HSA_STATUS_SUCCESS)
        return HSA_STATUS_SUCCESS;
    if (hsa_agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_DOMAIN, &dom) !=
        HSA_STATUS_SUCCESS)
        dom = 0;
    if ((bdf >> 8) == f->bus && ((bdf >> 3) & 0x1f) == f->dev && dom == f->domain) {
        f->found = a;
        f->hit = true;
        return HSA_STATUS_INFO_BREAK;
    }
    return HSA_STATUS_SUCCESS;
}

hsa_status_t first_cpu(hsa_agent_t a, void* data) {
    hsa_device_type_t t;
    if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) == HSA_STATUS_SUCCESS &&
        t == HSA_DEVICE_TYPE_CPU) {
        *static_cast<hsa_agent_t*>(data) = a;
        return HSA_STATUS_INFO_BREAK;
    }
    return HSA_STATUS_SUCCESS;
}

// A job's copies take milliseconds once its ready flag is released; a job
// not complete this long after the release is taken as failed.  (Before the
// release the job waits for earlier work on the call's stream, for as long
// as that takes.)
constexpr auto kJobTimeLimit = std::chrono::seconds(60);
// Engines that carry the host link at its rate on MI355X: engines 0-3 move
// 55.6-56.0 GB/s each way in staged swaps; engines 4-15 move 7-13 GB/s device
// to host and 28-50 GB/s host to device.
constexpr uint32_t kHostLinkEngines = 0xF;
// Wait slices, in HSA timestamp ticks (nanoseconds to 10 ns each).
constexpr uint64_t kWaitHint = 10000000ull;
// Start value of an engine's completion signal, which every copy decrements.
constexpr hsa_signal_value_t kDoneBase = (hsa_signal_value_t)1 << 62;

// Releases up to two ready flags (see launch_release_flags).
__global__ __launch_bounds__(64) void release_flags_kernel(int64_t* a, int64_t* b) {
    if (threadIdx.x == 0) {
        __hip_atomic_store(a, 0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
        if (b) __hip_atomic_store(b, 0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

}  // namespace

hipError_t launch_release_flags(int64_t* a, int64_t* b, hipStream_t stream) {
    if (!a) return hipErrorInvalidValue;
    hipLaunchKernelGGL(release_flags_kernel, dim3(1), dim3(64), 0, stream, a, b);
    return hipGetLastError();
}

bool link_acquire(int device, LinkAgents* out) {
    if (hsa_init() != HSA_STATUS_SUCCESS) return false;
    int bus = 0, dev = 0, dom = 0;
    if (hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, device) != hipSuccess ||
        hipDeviceGetAttribute(&dev, hipDeviceAttributePciDeviceId, device) != hipSuccess ||
        hipDeviceGetAttribute(&dom, hipDeviceAttributePciDomainId, device) != hipSuccess) {
        (void)hipGetLastError();
        hsa_shut_down();
        return false;
    }
    FindGpu f{(uint32_t)dom, (uint32_t)bus, (uint32_t)dev, {0}, false};
    (void)hsa_iterate_agents(find_gpu, &f);
    if (!f.hit) {
        hsa_shut_down();
        return false;
    }
    hsa_agent_t cpu{0};
    if (hsa_agent_get_info(f.found, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_NEAREST_CPU, &cpu) !=
            HSA_STATUS_SUCCESS ||
        !cpu.handle) {
        cpu.handle = 0;
        (void)hsa_iterate_agents(first_cpu, &cpu);
    }
    if (!cpu.handle) {
        hsa_shut_down();
        return false;
    }
    out->gpu = f.found;
    out->cpu = cpu;
    return true;
}

void link_release() { hsa_shut_down(); }

void link_auto_engines(const LinkAgents& a, int32_t* d2h, int32_t* h2d) {
    uint32_t av[2] = {0, 0}, pref[2] = {0, 0};
    if (hsa_amd_memory_copy_engine_status(a.cpu, a.gpu, &av[0]) != HSA_STATUS_SUCCESS) av[0] = 0;
    if (hsa_amd_memory_copy_engine_status(a.gpu, a.cpu, &av[1]) != HSA_STATUS_SUCCESS) av[1] = 0;
    if (hsa_amd_memory_get_preferred_copy_engine(a.cpu, a.gpu, &pref[0]) != HSA_STATUS_SUCCESS)
        pref[0] = 0;
    if (hsa_amd_memory_get_preferred_copy_engine(a.gpu, a.cpu, &pref[1]) != HSA_STATUS_SUCCESS)
        pref[1] = 0;
    pick_link_engines(av[0], pref[0], av[1], pref[1], kHostLinkEngines, d2h, h2d);
}

hipError_t LinkEngine::start(int device, const LinkAgents& a, int dir, int32_t engine) {
    if (running() || engine < 0 || engine > 15) return hipErrorInvalidValue;
    device_ = device;
    engine_ = engine;
    dst_agent_ = dir == 0 ? a.cpu : a.gpu;
    src_agent_ = dir == 0 ? a.gpu : a.cpu;
    hipError_t e = hipExtMallocWithFlags(&count_, sizeof(uint64_t), hipMallocSignalMemory);
    hipPointerAttribute_t attr{};
    if (e == hipSuccess) e = hipPointerGetAttributes(&attr, count_);
    if (e != hipSuccess || !attr.hostPointer) {
        (void)hipGetLastError();
        if (count_) (void)hipFree(count_);
        count_ = nullptr;
        return e != hipSuccess ? e : hipErrorInvalidValue;
    }
    count_host_ = static_cast<volatile uint64_t*>(attr.hostPointer);
    __atomic_store_n(count_host_, 0ull, __ATOMIC_RELEASE);
    if (hsa_signal_create(kDoneBase, 0, nullptr, &done_) != HSA_STATUS_SUCCESS) {
        done_.handle = 0;
        (void)hipFree(count_);
        count_ = nullptr;
        count_host_ = nullptr;
        return hipErrorOutOfMemory;
    }
    queued_ = 0;
    issued_ = 0;
    stop_ = false;
    err_.store(0);
    th_ = std::thread([this] { loop(); });
    return hipSuccess;
}

void LinkEngine::stop(bool abandon) {
    if (!th_.joinable()) return;
    abandon_.store(abandon, std::memory_order_release);
    {
        std::lock_guard<std::mutex> lk(mu_);
        stop_ = true;
    }
    stopping_.store(true, std::memory_order_release);
    cv_.notify_all();
    th_.join();
    stopping_.store(false);
    abandon_.store(false);
    if (stuck_) {
        // The engine may still wait on a ready flag or decrement done_, and a
        // stream wait may still read the count: keep them all allocated.
        stuck_ = false;
        all_.clear();
        spare_ready_.clear();
        done_.handle = 0;
        count_ = nullptr;
        count_host_ = nullptr;
        return;
    }
    for (hsa_signal_t sg : all_) hsa_signal_destroy(sg);
    all_.clear();
    spare_ready_.clear();
    if (done_.handle) hsa_signal_destroy(done_);
    done_.handle = 0;
    (void)hipFree(count_);
    count_ = nullptr;
    count_host_ = nullptr;
}

bool LinkEngine::take_ready(hsa_signal_t* ready) {
    std::lock_guard<std::mutex> lk(mu_);
    if (spare_ready_.empty()) {
        // Waited on by the engine only; a kernel stores its value directly.
        hsa_signal_t sg;
        if (hsa_amd_signal_create(1, 0, nullptr, HSA_AMD_SIGNAL_AMD_GPU_ONLY, &sg) !=
            HSA_STATUS_SUCCESS)
            return false;
        all_.push_back(sg);
        spare_ready_.push_back(sg);
    }
    *ready = spare_ready_.back();
    spare_ready_.pop_back();
    return true;
}

uint64_t LinkEngine::submit(const std::vector<LinkPiece>& pieces, int64_t** flag) {
    *flag = nullptr;
    const uint64_t index = issued_++;
    Job job{index, queued_, {0}, nullptr};
    volatile hsa_signal_value_t* value = nullptr;
    if (err_.load(std::memory_order_acquire) == 0) {
        if (!take_ready(&job.ready)) {
            fail(hipErrorOutOfMemory);
        } else if (hsa_amd_signal_value_pointer(job.ready, &value) != HSA_STATUS_SUCCESS) {
            fail(hipErrorInvalidValue);
            std::lock_guard<std::mutex> lk(mu_);
            spare_ready_.push_back(job.ready);
            job.ready.handle = 0;
        }
    }
    if (job.ready.handle) {
        hsa_signal_store_relaxed(job.ready, 1);
        for (const LinkPiece& pc : pieces) {
            if (hsa_amd_memory_async_copy_on_engine(
                    pc.dst, dst_agent_, pc.src, src_agent_, pc.bytes, 1, &job.ready, done_,
                    (hsa_amd_sdma_engine_id_t)(1u << engine_), true) != HSA_STATUS_SUCCESS) {
                fail(hipErrorUnknown);
                break;
            }
            ++queued_;
        }
        job.end = queued_;
        // Copies already queued wait for the flag, so it is handed out even
        // when some failed to queue.
        job.flag = const_cast<int64_t*>(value);
        *flag = job.flag;
    }
    {
        std::lock_guard<std::mutex> lk(mu_);
        q_.push_back(job);
    }
    cv_.notify_one();
    return index;
}

uint64_t LinkEngine::release_on_host(int64_t* flag) {
    if (!flag) return 0;
    // A held job cannot have completed, so it is still queued here.
    std::lock_guard<std::mutex> lk(mu_);
    for (const Job& j : q_)
        if (j.flag == flag) {
            hsa_signal_store_screlease(j.ready, 0);
            return j.index + 1;
        }
    return 0;
}

void LinkEngine::wait_published(uint64_t count) const {
    // The library thread publishes every job, at the latest once the job
    // time limit has passed, so this ends.
    while (count_host_ && __atomic_load_n(count_host_, __ATOMIC_ACQUIRE) < count)
        std::this_thread::sleep_for(std::chrono::microseconds(50));
}

hipError_t LinkEngine::stream_wait(hipStream_t stream, uint64_t count) {
    if (__atomic_load_n(count_host_, __ATOMIC_ACQUIRE) >= count) return hipSuccess;
    return hipStreamWaitValue64(stream, count_, count, hipStreamWaitValueGte, ~0ull);
}

hipError_t LinkEngine::error() const { return (hipError_t)err_.load(std::memory_order_acquire); }

void LinkEngine::fail(hipError_t e) {
    int32_t none = 0;
    (void)err_.compare_exchange_strong(none, (int32_t)e);
}

void LinkEngine::publish(uint64_t completed) {
    __atomic_store_n(count_host_, completed, __ATOMIC_RELEASE);
}

void LinkEngine::loop() {
    for (;;) {
        Job job;
        {
            std::unique_lock<std::mutex> lk(mu_);
            cv_.wait(lk, [&] { return stop_ || !q_.empty(); });
            if (q_.empty()) return;  // stopped, nothing left
            job = q_.front();
        }
        // The engine completes copies in queue order, each decrementing
        // done_ once: the job is complete when done_ has dropped by the
        // number of copies queued up to and including it.
        const hsa_signal_value_t target = kDoneBase - (hsa_signal_value_t)job.end;
        // Behind a job that timed out, the engine completes nothing more:
        // later jobs are published failed at once.
        bool recycle = job.ready.handle != 0 && !stuck_;
        if (recycle) {
            // The time limit runs from the flag's release, or from the stop
            // for a flag still held then; before either, the job waits for
            // earlier work on its call's stream for as long as that takes.
            auto since = std::chrono::steady_clock::now();
            bool released = false, timed = false;
            while (hsa_signal_wait_scacquire(done_, HSA_SIGNAL_CONDITION_LT, target + 1,
                                             kWaitHint, HSA_WAIT_STATE_BLOCKED) > target) {
                const auto now = std::chrono::steady_clock::now();
                if (!released) {
                    released = hsa_signal_load_relaxed(job.ready) == 0;
                    if (!released && stopping_.load(std::memory_order_acquire)) {
                        if (abandon_.load(std::memory_order_acquire)) {
                            // The pool failed: its release kernel may never run.
                            hsa_signal_store_screlease(job.ready, 0);
                            released = true;
                        } else if (!timed) {
                            timed = true;
                            since = now;
                        }
                    }
                    if (released) {
                        since = now;
                        continue;
                    }
                    if (!timed) continue;
                }
                if (now - since > kJobTimeLimit) {
                    fail(hipErrorLaunchTimeOut);
                    stuck_ = true;
                    recycle = false;
                    break;
                }
            }
        } else if (job.ready.handle) {
            fail(hipErrorLaunchTimeOut);
        }
        publish(job.index + 1);
        std::lock_guard<std::mutex> lk(mu_);
        q_.pop_front();
        if (recycle) spare_ready_.push_back(job.ready);
    }
}

}  // namespace aqua
