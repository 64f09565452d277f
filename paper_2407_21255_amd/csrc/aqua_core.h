// aqua_core.h -- host-side core of the KV page-swap library: argument
// validation, run planning, cross-stream hazard tracking and the swap
// space's range allocator.  Pure C++17,
// no HIP types, so that it builds and is tested on a machine without a GPU.
#pragma once

#include <cstddef>
#include <cstdint>
#include <map>
#include <unordered_map>
#include <utility>
#include <vector>

#include "aqua.h"

namespace aqua {

// Pool geometry.  One (layer, block) chunk of the pool
// [L][N][2][H][T][D] is C = 2*H*T*D*elem contiguous bytes.
struct Shape {
    uint32_t L = 0, N = 0, H = 0, T = 0, D = 0;
    int32_t dtype = 0;
    uint64_t C = 0;          // chunk bytes
    uint64_t pool_bytes = 0; // L*N*C
};

// Largest chunk (1 GiB) and largest pool or image (2^62 bytes) accepted.
constexpr uint64_t kMaxChunkBytes = 1ull << 30;
constexpr uint64_t kMaxBytes = 1ull << 62;

// Fills *out from a descriptor; AQUA_ERR_INVALID for a zero dimension, an
// unknown dtype, or a chunk that is not a multiple of 16 bytes.
aqua_status make_shape(const aqua_kv_desc* d, Shape* out);

// One swap call as the caller described it.
struct CallArgs {
    uint32_t num_seqs = 0;
    const int32_t* ids = nullptr;
    const uint64_t* offs = nullptr;        // num_seqs+1 CSR offsets
    const uint64_t* img_offsets = nullptr; // nullptr: packed images
    uintptr_t buf = 0;                     // offload buffer address
    uint64_t buf_bytes = 0;
    bool is_in = false;                    // swap-in: destinations are blocks
    // Blocks per layer of each image (>= its table length; the table covers
    // the first blocks of every layer).  nullptr: the table lengths.
    const uint64_t* img_blocks = nullptr;
    // Layers moved: [first_layer, first_layer + num_layers); 0 layers with
    // first_layer 0 means every layer.
    uint32_t first_layer = 0;
    uint32_t num_layers = 0;
};

// Blocks per layer of sequence k's image.
uint64_t image_blocks(const CallArgs& a, uint32_t k);

// One range of a migration: len bytes from src_off to dst_off.
struct CopyRange {
    uint64_t src_off, dst_off, len;
};

// Migration validation: offsets and lengths multiples of 16, ranges inside
// their buffers, destination ranges disjoint from each other and from every
// source range (as addresses).  Same codes and precedence as the oracle.
aqua_status validate_migrate(uintptr_t src, uint64_t src_bytes, uintptr_t dst,
                             uint64_t dst_bytes, uint32_t n, const uint64_t* src_off,
                             const uint64_t* dst_off, const uint64_t* len);

// Work item of the range-copy kernel: at most `unit` bytes each.
struct alignas(16) CopyDesc {
    uint64_t src_off;
    uint64_t dst_off;
    uint64_t len;
    uint64_t reserved;
};
static_assert(sizeof(CopyDesc) == 32, "descriptor layout is shared with the kernels");

// Splits the ranges into pieces of at most `unit` bytes.
size_t plan_copies(uint32_t n, const uint64_t* src_off, const uint64_t* dst_off,
                   const uint64_t* len, uint64_t unit, std::vector<CopyDesc>* out);

// Work item of the copy kernels: a run of `nchunks` consecutive pool blocks
// starting at `block` whose image chunks are also consecutive.  In layer l
// the pool side starts at (l*N + block)*C and the image side at
// img_off + l*img_lstride.  32 bytes so that one scalar load fetches it.
struct alignas(16) RunDesc {
    uint64_t img_off;
    uint64_t img_lstride;
    uint32_t block;
    uint32_t nchunks;
    uint32_t reserved0;
    uint32_t reserved1;
};
static_assert(sizeof(RunDesc) == 32, "descriptor layout is shared with the kernels");

// Launch geometry of the copy kernels.  Every lane moves kUnroll 16-byte
// vectors per pass, so a workgroup of `threads` lanes has threads * 64 bytes
// in flight.  A workgroup is sized to the chunk: 1024 lanes for chunks of
// 64 KiB and more, fewer for smaller chunks (down to min_threads, a power
// of two of at least 64), so that every lane still issues kUnroll loads
// before its first store.
constexpr uint32_t kUnroll = 4;
constexpr uint32_t kMaxThreads = 1024;
uint32_t swap_threads(uint64_t chunk_bytes, uint32_t min_threads);

// Workgroups of one launch over `units` work units: one per unit, at most
// `max_workgroups` when that is non-zero, and never more than kMaxGrid.  A
// dispatch counts its work-items in 32 bits, so 1024-lane workgroups allow
// at most 4 194 303 of them; the kernels loop over units with a grid
// stride, so a capped grid still covers every unit.
constexpr uint32_t kMaxGrid = 1u << 21;
uint32_t launch_grid(uint64_t units, uint32_t max_workgroups);

// The order in which a call's runs go to the kernels (each run is
// independent, so the order changes no byte).  Runs dealt out to the XCDs
// (interleave_runs), swap-ins sorted by pool block first:
//   chunks of 64 KiB or more: every swap-in; a swap-out when it covers at
//     least 40 % of the pool's blocks or its sequences average at least 32
//     blocks (the others keep table order);
//   smaller chunks: a swap-in that covers at least 40 % of the pool; every
//     other call keeps table order.
// Sorted, the pool side of consecutive units moves through the pool in
// address order and the image side jumps; in table order the reverse.
// Measured on MI355X, same box:
//   swap-ins (pool written in order), calls covering half the pool: sorted
//     against table order, 70B scatter 3.3 % shorter, one TP2 rank's 1.6 %,
//     one TP4 rank's 2.8 %; a sixteenth of the pool (8B, fp8 8B): no gain,
//     a quarter (the preemption cycle): 3-7 % longer;
//   swap-outs (image written in order in table order), half the pool: sorted
//     against table order, 64 KiB chunks 4.5 % shorter but 32 KiB chunks
//     1.6 % and 16 KiB chunks 6 % longer; once dealt to the XCDs, the 70B
//     gather in table order took 2.8 % less than sorted (3.53 against
//     3.63 ms, four runs each), the pair +1.4 %.
//   sparse calls of 64 KiB chunks, dealt as above against table order
//     (three runs each): one prompt of 1024 or 2048 blocks +3 to +7.5 %,
//     8 prompts +1.3 to +2.7 %, the 8B pair +1.1 %, prefix loads beside
//     other swaps +3.6 %, 64 prompts of 32 blocks +3 to +4 %; dealing the
//     gather of 64 prompts of 16 blocks too cost it 8 %, hence the 32-block
//     mean.  Sorting or dealing sparse calls of smaller chunks lost 2.6 %
//     (the fp8 8B pair, whose scatter then leaves the XCD unit order).
enum class RunOrder { kTable, kSortedDealt, kTableDealt };
constexpr uint64_t kDenseMinPermille = 400;     // share of the pool's blocks
constexpr uint64_t kDealMinChunk = 64ull << 10;
constexpr uint64_t kDealOutMinMeanBlocks = 32;  // sparse swap-outs: blocks per sequence
RunOrder run_order(bool is_in, uint64_t chunk_bytes, uint64_t blocks, uint32_t num_blocks,
                   uint32_t num_seqs);

// Puts the runs in ascending order of their first block, keeping the table
// order of runs that start at the same block (a swap-out may name a block
// twice).  A counting sort over the pool's blocks, O(runs + num_blocks), when
// the runs number at least a sixteenth of the blocks; a stable comparison
// sort, O(runs log runs), below that, so that a small call does not pay for
// the whole pool.  `counts` and `tmp` are reusable scratch.
constexpr uint64_t kSortCountingMinRatio = 16;
void sort_by_block(std::vector<RunDesc>* runs, uint32_t num_blocks,
                   std::vector<uint32_t>* counts, std::vector<RunDesc>* tmp);

// XCD-aware order of a dense call's runs.  A launch's workgroups go to
// MI355X's 8 XCDs (each with its own L2) in turn, and the kernels take one
// unit per workgroup, layer by layer.  Dealing a layer's runs out 8 ways (run
// j of the result is run j / 8 of the (j % 8)-th contiguous eighth of the
// input; the first n % 8 eighths hold one run more) gives each XCD one
// contiguous eighth of the runs in every layer:
// of the pool range when they are sorted, of the image when they are in
// table order, instead of every XCD taking every eighth run of one shared
// range.  Measured on MI355X against sorted order, same box, 3 to 6 runs
// each: 70B pair +1.4 to +3.3 % (four comparisons), one TP4 rank +2.7 to
// +3.3 %, the Yi-34B prefix load +2.1 to +3.6 %, one TP2 rank +1.0 %; the
// fair-scheduling reschedules -0.4 to -1.7 % (within their run-to-run
// spread).  2 ways gained about half as much, 16 or 32 ways lost 1-4 %
// against 8.  Which calls are dealt is run_order's rule.  A launch may start
// its turn at another XCD than the first (where the previous launch left
// off); that only changes which XCD takes which eighth.  Runs only ever
// change order, so no byte changes.  `tmp` is reusable scratch.
constexpr uint32_t kXcdWays = 8;
void interleave_runs(std::vector<RunDesc>* runs, uint32_t ways, std::vector<RunDesc>* tmp);

// XCD-aware unit order inside the kernels, for calls whose runs are not
// dealt out.  On a launch of one workgroup per unit, workgroup b (sent to XCD
// (b + c) % 8, c fixed for the launch) takes unit xcd_unit(b, units), so that
// each XCD copies one contiguous eighth of the launch's units in order (the
// (b % 8)-th eighth; the first units % 8 eighths hold one unit more).  A
// bijection on [0, units).  Used for undealt calls of chunks between 16 and 64 KiB
// (exclusive) to an HBM buffer, where it measured, against plain order on
// the same box (3 to 4 runs each, with launches of at most 512 MiB then):
// the fp8 preemption cycle +4.2 %, one TP2 rank +0.5 %, the fp8 8B pair
// +0.5 %; on the fp8 8B pool, one prompt of
// 1024 or 2048 blocks +3 to +8 %, 64 short prompts +1 to +16 %, the gather of
// 8 prompts -0.4 to -1.9 %.  With 64 KiB chunks it slowed 64 short prompts by
// 6 %, with 16 KiB chunks a TP4 rank by 1.2 %, so those keep plain order.
constexpr uint32_t xcd_unit(uint32_t block, uint32_t units) {
    const uint32_t x = block % kXcdWays, q = units / kXcdWays, r = units % kXcdWays;
    return x * q + (x < r ? x : r) + block / kXcdWays;
}
constexpr uint64_t kXcdUnitMinChunk = 16ull << 10;  // exclusive
constexpr uint64_t kXcdUnitMaxChunk = 64ull << 10;  // exclusive
bool xcd_unit_order(uint64_t chunk_bytes, bool dealt);

// Layers per launch of a call with `ndesc` runs per layer: whole layers and
// fewer than 2^31 units per launch, so that almost every call is one launch.
// Launches of at most 512 MiB had made calls of 32 KiB chunks 3-5 % shorter
// in plain unit order; with the XCD unit order, which gives each XCD an
// eighth of a whole launch, one launch per call measured faster again (one
// TP2 rank +2.4 %, the fp8 preemption cycle and 8B pair +0.4 %, four runs
// each), and splitting 16 or 64 KiB calls lost 2-4 %.
uint32_t layers_per_launch(uint32_t ndesc);

// Reusable scratch for duplicate detection (epoch-stamped marks, O(n)).
struct DupMarks {
    std::vector<uint32_t> mark;
    uint32_t epoch = 0;
};

// Validation in the library's precedence: invalid -> range -> duplicate ->
// capacity.  Pointer classes are checked by the caller (they need HIP).
aqua_status validate_call(const Shape& s, const CallArgs& a, DupMarks& marks);

// Byte offset of sequence k's image inside the buffer.
uint64_t image_offset(const Shape& s, const CallArgs& a, uint32_t k);

// Coalesces each table into runs bt[i+1] == bt[i] + 1, split so that a run
// covers at most max(1, max_unit_bytes / C) chunks.  Appends to *out and
// returns the number of descriptors appended.
size_t plan_runs(const Shape& s, const CallArgs& a, uint64_t max_unit_bytes,
                 std::vector<RunDesc>* out);

// Half-open byte ranges [lo, hi) of the buffer that the call touches (one
// per non-empty sequence).
void image_ranges(const Shape& s, const CallArgs& a,
                  std::vector<std::pair<uint64_t, uint64_t>>* out);

// ---------------------------------------------------------------------------
// Hazard tracker.
//
// Every call gets a ticket (1, 2, 3, ...) and runs on a "lane" (one lane
// per distinct stream).  Work on one lane completes in issue order, so a
// dependency on ticket t of lane m is satisfied by waiting on the newest
// conflicting ticket of m.  Per pool block the tracker keeps the last
// writing ticket and, per lane, the newest ticket reading it since that
// write; per offload byte range it keeps the in-flight readers and writers.
// Tickets known complete (per-lane watermark) are never waited on.
//
// Memory stays bounded however many calls are issued: the lane of a ticket
// is kept only from the oldest ticket not yet known complete onwards (every
// older ticket is complete, whatever its lane), and a lane whose tickets
// have all completed can be handed to another stream (LaneMap).
class HazardTracker {
public:
    struct Dep {
        uint32_t lane;
        uint64_t ticket;
    };

    explicit HazardTracker(uint32_t num_blocks = 0) { reset(num_blocks); }
    void reset(uint32_t num_blocks);

    // What one call touches: pool blocks it reads or writes, and byte
    // ranges [lo, hi) of offload buffers (by address) it reads or writes.
    struct Access {
        const int32_t* blocks_read = nullptr;
        size_t n_blocks_read = 0;
        const int32_t* blocks_written = nullptr;
        size_t n_blocks_written = 0;
        const std::pair<uint64_t, uint64_t>* ranges_read = nullptr;
        size_t n_ranges_read = 0;
        const std::pair<uint64_t, uint64_t>* ranges_written = nullptr;
        size_t n_ranges_written = 0;
    };

    // Registers call `ticket` (must exceed every earlier ticket) on `lane`.
    // Writes into *deps, per other lane, the newest earlier ticket the call
    // must wait for.  Returns the number of conflicts that were skipped
    // because already complete.  Blocks written by one call must be
    // distinct; a range both read and written is listed as written.
    uint64_t issue(uint64_t ticket, uint32_t lane, const Access& a,
                   std::vector<Dep>* deps);

    // Everything on `lane` up to and including `ticket` has completed.
    void complete(uint32_t lane, uint64_t ticket);
    uint64_t completed(uint32_t lane) const;
    // Lane of an issued ticket that is not yet known complete; kNoLane for a
    // ticket already known complete (or never issued).
    static constexpr uint32_t kNoLane = UINT32_MAX;
    uint32_t lane_of(uint64_t ticket) const;
    // Known complete: below the oldest outstanding ticket, or at or below
    // its lane's watermark.
    bool done(uint64_t ticket) const;
    // Every ticket issued on `lane` is known complete.
    bool idle(uint32_t lane) const;
    size_t live_ranges() const { return ranges_.size(); }
    uint64_t last_ticket() const { return last_ticket_; }
    // Tickets whose lane is still kept (from the oldest one not known
    // complete to the newest) and lanes known to the tracker.
    size_t tickets_kept() const { return ticket_lane_.size() - head_; }
    size_t lanes() const { return done_.size(); }

private:
    struct Reader {
        uint32_t lane;
        uint64_t ticket;
    };
    // One pool block: its last writer and its readers since then, at most
    // one per lane.  The first reader is kept in the record, so that a call
    // touches one 24-byte record per block; readers on further lanes at
    // once (several streams reading one block) go to more_.
    struct BlockRec {
        uint64_t writer = 0;       // ticket of the last writer, 0: none
        uint64_t reader = 0;       // ticket of the kept reader, 0: none
        uint32_t reader_lane = 0;
        uint32_t more = 0;         // 1: more_ holds further readers of the block
    };
    struct RangeRec {
        uint64_t lo, hi, ticket;
        uint32_t lane;
        bool write;
    };
    // What issue() found for one earlier ticket (see need()).
    enum class Need : uint8_t { kNone, kComplete, kSameLane, kWait };
    void ensure_lane(uint32_t lane);
    void prune();
    Need need(uint64_t ticket, uint32_t lane);

    std::vector<BlockRec> blocks_;
    std::unordered_map<uint32_t, std::vector<Reader>> more_;
    std::vector<RangeRec> ranges_;
    std::vector<uint64_t> done_;         // per lane watermark
    std::vector<uint64_t> last_;         // per lane, newest ticket issued on it
    std::vector<uint64_t> dep_;          // per lane, scratch of one issue()
    std::vector<uint32_t> ticket_lane_;  // from head_: lanes of tickets base_, base_ + 1, ...
    size_t head_ = 0;
    uint64_t base_ = 1;                  // every ticket below is complete
    uint64_t last_ticket_ = 0;
};

// Stream -> lane map of one pool.  A stream seen before keeps its lane; a
// new stream takes over the lowest lane that is idle in the tracker (every
// ticket issued on it complete), else a new lane, so the lane count is at
// most the number of streams with calls in flight at once, plus one.
class LaneMap {
public:
    uint32_t lane_for(uintptr_t stream, const HazardTracker& t);
    size_t size() const { return stream_.size(); }
    uintptr_t stream_of(uint32_t lane) const { return stream_[lane]; }

private:
    std::vector<uintptr_t> stream_;
};

// First-fit allocator of byte ranges inside one arena [0, size) (the swap
// space's device region and its host region).  Every range starts on an
// `align` boundary and is a multiple of it; freeing coalesces neighbours.
// Host bookkeeping only: whoever reuses a freed range orders the reuse.
// Copy engines for the two link directions from the runtime's masks (bit e:
// engine e).  Per direction the candidates are the runtime's preferred
// engines that are available; else the `fast` engines (those that carry the
// host link at its rate) that are available; else the `fast` engines, shared
// with their other users, rather than a slower free one.  The lowest-numbered
// candidate is taken, the host-to-device direction on a different engine from
// the device-to-host one where its candidates allow.  With `fast` empty the
// available engines stand in for it.  -1 for a direction with no candidate.
void pick_link_engines(uint32_t d2h_avail, uint32_t d2h_pref, uint32_t h2d_avail,
                       uint32_t h2d_pref, uint32_t fast, int32_t* d2h, int32_t* h2d);

class RangeAllocator {
public:
    void reset(uint64_t size, uint64_t align);
    bool alloc(uint64_t bytes, uint64_t* off);  // false: no free range fits
    bool free(uint64_t off);                     // false: off is not allocated
    uint64_t size() const { return size_; }
    uint64_t free_bytes() const { return free_total_; }
    uint64_t largest_free() const;
    uint64_t granted(uint64_t off) const;        // bytes of the range at off (0: none)

private:
    uint64_t size_ = 0, align_ = 1, free_total_ = 0;
    std::map<uint64_t, uint64_t> free_;   // offset -> length
    std::map<uint64_t, uint64_t> used_;   // offset -> length
};

}  // namespace aqua
