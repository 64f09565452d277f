// core_testapi.cpp -- C entry points into the host core for CPU tests.
// Built into a separate library (libaqua_core.so) with the system C++
// compiler; the GPU library does not contain these symbols.
#include <algorithm>
#include <cstring>
#include <vector>

#include "aqua.h"
#include "aqua_core.h"

extern "C" {

aqua_status aqua_core_validate(const aqua_kv_desc* desc, uint32_t num_seqs,
                               const int32_t* ids, const uint64_t* offs,
                               uint64_t buf_addr, uint64_t buf_bytes,
                               const uint64_t* img_offsets, int32_t is_in) {
    aqua::Shape s;
    aqua_status st = aqua::make_shape(desc, &s);
    if (st != AQUA_OK) return st;
    aqua::CallArgs a;
    a.num_seqs = num_seqs;
    a.ids = ids;
    a.offs = offs;
    a.img_offsets = img_offsets;
    a.buf = (uintptr_t)buf_addr;
    a.buf_bytes = buf_bytes;
    a.is_in = is_in != 0;
    aqua::DupMarks marks;
    return aqua::validate_call(s, a, marks);
}

aqua_status aqua_core_validate_ex(const aqua_kv_desc* desc, uint32_t num_seqs,
                                  const int32_t* ids, const uint64_t* offs,
                                  uint64_t buf_addr, uint64_t buf_bytes,
                                  const uint64_t* img_offsets, const uint64_t* img_blocks,
                                  uint32_t first_layer, uint32_t num_layers, int32_t is_in) {
    aqua::Shape s;
    aqua_status st = aqua::make_shape(desc, &s);
    if (st != AQUA_OK) return st;
    aqua::CallArgs a;
    a.num_seqs = num_seqs;
    a.ids = ids;
    a.offs = offs;
    a.img_offsets = img_offsets;
    a.img_blocks = img_blocks;
    a.first_layer = first_layer;
    a.num_layers = num_layers;
    a.buf = (uintptr_t)buf_addr;
    a.buf_bytes = buf_bytes;
    a.is_in = is_in != 0;
    aqua::DupMarks marks;
    return aqua::validate_call(s, a, marks);
}

aqua_status aqua_core_validate_migrate(uint64_t src, uint64_t src_bytes, uint64_t dst,
                                       uint64_t dst_bytes, uint32_t n, const uint64_t* so,
                                       const uint64_t* dof, const uint64_t* len) {
    return aqua::validate_migrate((uintptr_t)src, src_bytes, (uintptr_t)dst, dst_bytes, n, so,
                                  dof, len);
}

// Writes up to max_out descriptors (32 bytes each) and returns how many the
// plan has; negative status for an invalid shape.
int64_t aqua_core_plan_ex(const aqua_kv_desc* desc, uint32_t num_seqs,
                          const int32_t* ids, const uint64_t* offs,
                          const uint64_t* img_offsets, const uint64_t* img_blocks,
                          uint64_t unit_bytes, void* out, uint64_t max_out) {
    aqua::Shape s;
    aqua_status st = aqua::make_shape(desc, &s);
    if (st != AQUA_OK) return st;
    aqua::CallArgs a;
    a.num_seqs = num_seqs;
    a.ids = ids;
    a.offs = offs;
    a.img_offsets = img_offsets;
    a.img_blocks = img_blocks;
    std::vector<aqua::RunDesc> plan;
    aqua::plan_runs(s, a, unit_bytes, &plan);
    const uint64_t n = plan.size() < max_out ? plan.size() : max_out;
    if (n) std::memcpy(out, plan.data(), n * sizeof(aqua::RunDesc));
    return (int64_t)plan.size();
}

int64_t aqua_core_plan(const aqua_kv_desc* desc, uint32_t num_seqs,
                       const int32_t* ids, const uint64_t* offs,
                       const uint64_t* img_offsets, uint64_t unit_bytes,
                       void* out, uint64_t max_out) {
    aqua::Shape s;
    aqua_status st = aqua::make_shape(desc, &s);
    if (st != AQUA_OK) return st;
    aqua::CallArgs a;
    a.num_seqs = num_seqs;
    a.ids = ids;
    a.offs = offs;
    a.img_offsets = img_offsets;
    std::vector<aqua::RunDesc> plan;
    aqua::plan_runs(s, a, unit_bytes, &plan);
    const uint64_t n = plan.size() < max_out ? plan.size() : max_out;
    if (n) std::memcpy(out, plan.data(), n * sizeof(aqua::RunDesc));
    return (int64_t)plan.size();
}

void* aqua_core_tracker_new(uint32_t num_blocks) {
    return new aqua::HazardTracker(num_blocks);
}

void aqua_core_tracker_free(void* t) { delete static_cast<aqua::HazardTracker*>(t); }

// ranges: nranges pairs (lo, hi).  A swap-out (is_in 0) reads `blocks`
// and writes the ranges; a swap-in reads the ranges and writes `blocks`.
// Returns the number of dependencies and writes them to dep_lanes /
// dep_tickets (at most max_deps).
int64_t aqua_core_tracker_issue(void* t, uint64_t ticket, uint32_t lane,
                                int32_t is_in, const int32_t* blocks,
                                uint64_t nblocks, const uint64_t* ranges,
                                uint64_t nranges, uint32_t* dep_lanes,
                                uint64_t* dep_tickets, uint64_t max_deps) {
    auto* tr = static_cast<aqua::HazardTracker*>(t);
    std::vector<std::pair<uint64_t, uint64_t>> r(nranges);
    for (uint64_t k = 0; k < nranges; ++k) r[k] = {ranges[2 * k], ranges[2 * k + 1]};
    aqua::HazardTracker::Access acc;
    if (is_in) {
        acc.blocks_written = blocks;
        acc.n_blocks_written = nblocks;
        acc.ranges_read = r.data();
        acc.n_ranges_read = r.size();
    } else {
        acc.blocks_read = blocks;
        acc.n_blocks_read = nblocks;
        acc.ranges_written = r.data();
        acc.n_ranges_written = r.size();
    }
    std::vector<aqua::HazardTracker::Dep> deps;
    tr->issue(ticket, lane, acc, &deps);
    for (uint64_t k = 0; k < deps.size() && k < max_deps; ++k) {
        dep_lanes[k] = deps[k].lane;
        dep_tickets[k] = deps[k].ticket;
    }
    return (int64_t)deps.size();
}

// General form: separate read and write sets (ranges as (lo, hi) pairs).
int64_t aqua_core_tracker_issue_rw(void* t, uint64_t ticket, uint32_t lane,
                                   const int32_t* blocks_r, uint64_t nbr,
                                   const int32_t* blocks_w, uint64_t nbw,
                                   const uint64_t* ranges_r, uint64_t nrr,
                                   const uint64_t* ranges_w, uint64_t nrw,
                                   uint32_t* dep_lanes, uint64_t* dep_tickets,
                                   uint64_t max_deps) {
    auto* tr = static_cast<aqua::HazardTracker*>(t);
    std::vector<std::pair<uint64_t, uint64_t>> rr(nrr), rw(nrw);
    for (uint64_t k = 0; k < nrr; ++k) rr[k] = {ranges_r[2 * k], ranges_r[2 * k + 1]};
    for (uint64_t k = 0; k < nrw; ++k) rw[k] = {ranges_w[2 * k], ranges_w[2 * k + 1]};
    aqua::HazardTracker::Access acc;
    acc.blocks_read = blocks_r;
    acc.n_blocks_read = nbr;
    acc.blocks_written = blocks_w;
    acc.n_blocks_written = nbw;
    acc.ranges_read = rr.data();
    acc.n_ranges_read = rr.size();
    acc.ranges_written = rw.data();
    acc.n_ranges_written = rw.size();
    std::vector<aqua::HazardTracker::Dep> deps;
    tr->issue(ticket, lane, acc, &deps);
    for (uint64_t k = 0; k < deps.size() && k < max_deps; ++k) {
        dep_lanes[k] = deps[k].lane;
        dep_tickets[k] = deps[k].ticket;
    }
    return (int64_t)deps.size();
}

void aqua_core_tracker_complete(void* t, uint32_t lane, uint64_t ticket) {
    static_cast<aqua::HazardTracker*>(t)->complete(lane, ticket);
}

uint64_t aqua_core_tracker_live_ranges(void* t) {
    return static_cast<aqua::HazardTracker*>(t)->live_ranges();
}

uint64_t aqua_core_tracker_tickets_kept(void* t) {
    return static_cast<aqua::HazardTracker*>(t)->tickets_kept();
}

uint64_t aqua_core_tracker_lanes(void* t) {
    return static_cast<aqua::HazardTracker*>(t)->lanes();
}

int aqua_core_tracker_done(void* t, uint64_t ticket) {
    return static_cast<aqua::HazardTracker*>(t)->done(ticket) ? 1 : 0;
}

void* aqua_core_lanes_new() { return new aqua::LaneMap(); }
void aqua_core_lanes_free(void* m) { delete static_cast<aqua::LaneMap*>(m); }
uint32_t aqua_core_lanes_lane_for(void* m, uint64_t stream, void* t) {
    return static_cast<aqua::LaneMap*>(m)->lane_for(
        (uintptr_t)stream, *static_cast<aqua::HazardTracker*>(t));
}
uint64_t aqua_core_lanes_size(void* m) { return static_cast<aqua::LaneMap*>(m)->size(); }

// A serving loop in miniature, for the memory bound of the tracker: n_calls
// swaps (alternately out and in, 8 blocks each, of a num_blocks pool) on
// streams drawn round-robin from a set of `streams` handles that is replaced
// by new handles every `rotate` calls; at most `depth` calls are in flight
// (the oldest completes first).  Writes the largest number of tickets whose
// lane the tracker kept, and of lanes, seen after any call.
void aqua_core_tracker_soak(uint64_t n_calls, uint32_t num_blocks, uint32_t streams,
                            uint64_t rotate, uint32_t depth, uint64_t* max_kept,
                            uint64_t* max_lanes) {
    aqua::HazardTracker tr(num_blocks);
    aqua::LaneMap lanes;
    std::vector<std::pair<uint32_t, uint64_t>> fifo;  // (lane, ticket), oldest first
    size_t head = 0;
    std::vector<aqua::HazardTracker::Dep> deps;
    std::vector<int32_t> blocks(8);
    const std::pair<uint64_t, uint64_t> range{0, 4096};
    *max_kept = *max_lanes = 0;
    for (uint64_t i = 0; i < n_calls; ++i) {
        const uint64_t ticket = i + 1;
        const uintptr_t stream = 0x1000 + (i / rotate) * streams + i % streams;
        const uint32_t lane = lanes.lane_for(stream, tr);
        for (uint32_t j = 0; j < 8; ++j)
            blocks[j] = (int32_t)((i * 8 + j) * 2654435761ull % num_blocks);
        aqua::HazardTracker::Access acc;
        std::pair<uint64_t, uint64_t> r = range;
        r.first += (i % 64) * 4096;
        r.second += (i % 64) * 4096;
        if (i % 2) {
            acc.blocks_written = blocks.data();  // distinct: 8 consecutive multiples
            acc.n_blocks_written = 8;
            acc.ranges_read = &r;
            acc.n_ranges_read = 1;
        } else {
            acc.blocks_read = blocks.data();
            acc.n_blocks_read = 8;
            acc.ranges_written = &r;
            acc.n_ranges_written = 1;
        }
        tr.issue(ticket, lane, acc, &deps);
        fifo.emplace_back(lane, ticket);
        while (fifo.size() - head > depth) {
            tr.complete(fifo[head].first, fifo[head].second);
            ++head;
        }
        if (head > 4096) {
            fifo.erase(fifo.begin(), fifo.begin() + head);
            head = 0;
        }
        *max_kept = std::max<uint64_t>(*max_kept, tr.tickets_kept());
        *max_lanes = std::max<uint64_t>(*max_lanes, std::max(tr.lanes(), lanes.size()));
    }
}

uint32_t aqua_core_swap_threads(uint64_t chunk_bytes, uint32_t min_threads) {
    return aqua::swap_threads(chunk_bytes, min_threads);
}

// Sorts n descriptors (32 bytes each) in place by block with sort_by_block.
void aqua_core_sort_by_block(void* descs, uint64_t n, uint32_t num_blocks) {
    std::vector<aqua::RunDesc> v(n), tmp;
    std::vector<uint32_t> counts;
    if (n) std::memcpy(v.data(), descs, n * sizeof(aqua::RunDesc));
    aqua::sort_by_block(&v, num_blocks, &counts, &tmp);
    if (n) std::memcpy(descs, v.data(), n * sizeof(aqua::RunDesc));
}

// Reorders n descriptors (32 bytes each) in place with interleave_runs.
void aqua_core_interleave_runs(void* descs, uint64_t n, uint32_t ways) {
    std::vector<aqua::RunDesc> v(n), tmp;
    if (n) std::memcpy(v.data(), descs, n * sizeof(aqua::RunDesc));
    aqua::interleave_runs(&v, ways, &tmp);
    if (n) std::memcpy(descs, v.data(), n * sizeof(aqua::RunDesc));
}

uint32_t aqua_core_xcd_ways() { return aqua::kXcdWays; }

uint32_t aqua_core_xcd_unit(uint32_t block, uint32_t units) { return aqua::xcd_unit(block, units); }

int aqua_core_xcd_unit_order(uint64_t chunk_bytes, int dealt) {
    return aqua::xcd_unit_order(chunk_bytes, dealt != 0) ? 1 : 0;
}

// 0: table order, 1: sorted and dealt out, 2: table order dealt out.
int aqua_core_run_order(int is_in, uint64_t chunk_bytes, uint64_t blocks, uint32_t num_blocks,
                        uint32_t num_seqs) {
    return (int)aqua::run_order(is_in != 0, chunk_bytes, blocks, num_blocks, num_seqs);
}

uint32_t aqua_core_layers_per_launch(uint32_t ndesc) { return aqua::layers_per_launch(ndesc); }

uint32_t aqua_core_launch_grid(uint64_t units, uint32_t max_workgroups) {
    return aqua::launch_grid(units, max_workgroups);
}

void aqua_core_pick_link_engines(uint32_t d2h_avail, uint32_t d2h_pref, uint32_t h2d_avail,
                                 uint32_t h2d_pref, uint32_t fast, int32_t* d2h, int32_t* h2d) {
    aqua::pick_link_engines(d2h_avail, d2h_pref, h2d_avail, h2d_pref, fast, d2h, h2d);
}

void* aqua_core_ranges_new(uint64_t size, uint64_t align) {
    auto* r = new aqua::RangeAllocator();
    r->reset(size, align);
    return r;
}
void aqua_core_ranges_free_all(void* r) { delete static_cast<aqua::RangeAllocator*>(r); }
int aqua_core_ranges_alloc(void* r, uint64_t bytes, uint64_t* off) {
    return static_cast<aqua::RangeAllocator*>(r)->alloc(bytes, off) ? 1 : 0;
}
int aqua_core_ranges_release(void* r, uint64_t off) {
    return static_cast<aqua::RangeAllocator*>(r)->free(off) ? 1 : 0;
}
uint64_t aqua_core_ranges_free_bytes(void* r) {
    return static_cast<aqua::RangeAllocator*>(r)->free_bytes();
}
uint64_t aqua_core_ranges_largest_free(void* r) {
    return static_cast<aqua::RangeAllocator*>(r)->largest_free();
}

}  // extern "C"
