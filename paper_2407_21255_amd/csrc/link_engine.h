// link_engine.h -- copies over the host link on one chosen SDMA engine.
//
// The staged host path (the paper's temporary-tensor scheme, section 7,
// "Efficient context switching") moves each layer group between an HBM slot
// and pinned host memory.  Left to the runtime, a device-to-host copy may run
// as a blit kernel or on any of the device's copy engines, and not all
// engines reach the link rate.  A LinkEngine carries those copies on one
// engine through the HSA runtime instead.
//
// A job is the set of copies of one layer group.  Its copies enter the
// engine's queue when the job is submitted, during the swap call, each made
// to wait for the job's ready flag; a one-lane kernel on the call's stream
// releases the flag once the slot may be read or overwritten.  A library
// thread waits for the jobs' completions in order and publishes the number
// of completed jobs in signal memory; a stream that needs copies done waits
// on that count (hipStreamWaitValue64).
//
// Why this is deadlock-free: a job's release is enqueued when the job is
// submitted, and a stream wait only ever waits for jobs submitted before it,
// so every wait depends only on work enqueued before it, in any queue.  (A
// host function holding the stream would not do: the runtime runs host
// functions one at a time on one thread, so a held stream could keep another
// stream from reaching the release of a job queued ahead on the engine.)
//
// The runtime holds a stream waiting on memory in the command processor when
// GPU_STREAMOPS_CP_WAIT=1 is set before it starts; otherwise with a one-wave
// kernel, which is correct but keeps a compute unit partly occupied, enough
// to make a kernel that fills every compute unit once (a 256-tile GEMM) run a
// second round of tiles.
//
// The engine runs its queue in order.  Everything in it, this library's
// copies and any other user's, was queued after the work it depends on, so
// the queue always drains: a job is never queued behind a copy that waits
// for that job.
#pragma once

#include <hip/hip_runtime.h>
#include <hsa/hsa.h>

#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <deque>
#include <mutex>
#include <thread>
#include <vector>

namespace aqua {

// The GPU agent of a HIP device and the CPU agent nearest to it.
struct LinkAgents {
    hsa_agent_t gpu{};
    hsa_agent_t cpu{};
};

// Initialises the HSA runtime (reference counted) and finds the agents of
// `device`.  On success the caller owes one link_release().
bool link_acquire(int device, LinkAgents* out);
void link_release();

// Engines for the two directions when the caller names none: the HSA
// runtime's preferred engine for the direction if it names one, else the
// lowest-numbered free engine among those that carry the host link at its
// rate, else one of those shared with its other users; the two directions on
// different engines where possible (pick_link_engines).
void link_auto_engines(const LinkAgents& a, int32_t* d2h, int32_t* h2d);

// Enqueues one lane that stores 0, with system-scope release ordering, to
// each non-null flag (a job's ready flag from LinkEngine::submit): the
// stores are ordered after everything enqueued on `stream` before it.
hipError_t launch_release_flags(int64_t* a, int64_t* b, hipStream_t stream);

struct LinkPiece {
    void* dst;
    const void* src;
    uint64_t bytes;
};

class LinkEngine {
  public:
    LinkEngine() = default;
    LinkEngine(const LinkEngine&) = delete;
    LinkEngine& operator=(const LinkEngine&) = delete;
    ~LinkEngine() { stop(); }

    // dir 0: device memory to pinned host memory; 1: the reverse.
    hipError_t start(int device, const LinkAgents& a, int dir, int32_t engine);
    // Waits for every submitted job, then ends the thread.  With `abandon`
    // (after a failure), a job whose ready flag is still held is released
    // from the host, so that its copies and every copy queued behind them
    // on the engine still run.  If a job stays incomplete past the job time
    // limit, the engine may still wait on or write this object's signals:
    // they stay allocated for the life of the process.
    void stop(bool abandon = false);

    // Queues the copies of the next job on the engine, to run once the
    // job's ready flag is released (launch_release_flags).  Returns the job's
    // index (0, 1, ... in submission order) and the flag's device address.
    // On failure the job still counts as submitted and is published, with
    // the error kept for error().
    uint64_t submit(const std::vector<LinkPiece>& pieces, int64_t** flag);
    // Releases from the host the ready flag of a submitted job whose
    // release kernel was never enqueued (its call failed first), so that the
    // engine's queue, which every later copy on the engine shares, does not
    // hold a copy that waits forever.  The caller first waits for the work
    // that the job's copies were to follow.  Returns the completed-job count
    // that covers the job (0 if no held job has this flag).
    uint64_t release_on_host(int64_t* flag);
    // Blocks the calling thread until `count` jobs are published (complete,
    // or failed after the job time limit).
    void wait_published(uint64_t count) const;
    // Makes `stream` wait until `count` jobs have completed.
    hipError_t stream_wait(hipStream_t stream, uint64_t count);

    // First failure (hipSuccess if none).  A failed job is still published,
    // so that no stream waits forever.
    hipError_t error() const;
    int32_t engine() const { return engine_; }
    bool running() const { return th_.joinable(); }

  private:
    struct Job {
        uint64_t index;
        uint64_t end;        // copies queued on the engine up to and including this job
        hsa_signal_t ready;  // the copies' dependency, released by a kernel
        int64_t* flag;       // the address of ready's value, as handed out
    };
    void loop();
    void fail(hipError_t e);
    void publish(uint64_t completed);
    bool take_ready(hsa_signal_t* ready);

    int device_ = 0;
    int32_t engine_ = -1;
    hsa_agent_t dst_agent_{}, src_agent_{};
    void* count_ = nullptr;  // signal memory: the completed-job count
    volatile uint64_t* count_host_ = nullptr;
    uint64_t issued_ = 0;    // jobs submitted (caller's thread)
    std::mutex mu_;
    std::condition_variable cv_;
    std::deque<Job> q_;      // submitted, not yet published
    hsa_signal_t done_{0};   // decremented by every completed copy, in queue order
    uint64_t queued_ = 0;    // copies queued so far (caller's thread)
    std::vector<hsa_signal_t> spare_ready_, all_;
    bool stop_ = false;
    std::atomic<bool> stopping_{false};
    std::atomic<bool> abandon_{false};
    std::atomic<int32_t> err_{0};
    bool stuck_ = false;     // a job timed out (loop thread; read after join)
    std::thread th_;
};

}  // namespace aqua
