// aqua_core.cpp -- validation, run planning and hazard tracking (host only).
#include "aqua_core.h"

#include <algorithm>

namespace aqua {

namespace {

uint64_t elem_bytes(int32_t dtype) {
    switch (dtype) {
        case AQUA_F16:
        case AQUA_BF16:
            return 2;
        case AQUA_FP8_E4M3:
            return 1;
        default:
            return 0;
    }
}

}  // namespace

aqua_status make_shape(const aqua_kv_desc* d, Shape* out) {
    if (!d || !out) return AQUA_ERR_INVALID;
    const uint64_t e = elem_bytes(d->dtype);
    if (!d->num_layers || !d->num_blocks || !d->num_kv_heads ||
        !d->block_tokens || !d->head_dim || !e)
        return AQUA_ERR_INVALID;
    if (d->num_blocks > 0x7fffffffu) return AQUA_ERR_INVALID;  // int32 ids
    // Bounds that keep every byte offset, and every kernel's 16-byte vector
    // count per run, far from overflow.
    if (d->num_kv_heads > 65536 || d->block_tokens > 65536 || d->head_dim > 65536)
        return AQUA_ERR_INVALID;
    const unsigned __int128 C = (unsigned __int128)2 * d->num_kv_heads *
                                d->block_tokens * d->head_dim * e;
    if (C > kMaxChunkBytes) return AQUA_ERR_INVALID;
    if ((unsigned __int128)d->num_layers * d->num_blocks * C > kMaxBytes)
        return AQUA_ERR_INVALID;
    Shape s;
    s.L = d->num_layers;
    s.N = d->num_blocks;
    s.H = d->num_kv_heads;
    s.T = d->block_tokens;
    s.D = d->head_dim;
    s.dtype = d->dtype;
    s.C = 2ull * s.H * s.T * s.D * e;
    if (s.C % 16) return AQUA_ERR_INVALID;
    s.pool_bytes = (uint64_t)s.L * s.N * s.C;
    *out = s;
    return AQUA_OK;
}

uint64_t image_blocks(const CallArgs& a, uint32_t k) {
    return a.img_blocks ? a.img_blocks[k] : a.offs[k + 1] - a.offs[k];
}

uint64_t image_offset(const Shape& s, const CallArgs& a, uint32_t k) {
    if (a.img_offsets) return a.img_offsets[k];
    // Packed: images one after another in sequence order.
    if (!a.img_blocks) return (uint64_t)s.L * a.offs[k] * s.C;
    uint64_t off = 0;
    for (uint32_t q = 0; q < k; ++q) off += (uint64_t)s.L * a.img_blocks[q] * s.C;
    return off;
}

aqua_status validate_call(const Shape& s, const CallArgs& a, DupMarks& marks) {
    // -- invalid
    if (a.num_seqs && !a.offs) return AQUA_ERR_INVALID;
    const uint64_t total = a.num_seqs ? a.offs[a.num_seqs] : 0;
    if (a.num_seqs) {
        if (a.offs[0] != 0) return AQUA_ERR_INVALID;
        for (uint32_t k = 0; k < a.num_seqs; ++k)
            if (a.offs[k + 1] < a.offs[k]) return AQUA_ERR_INVALID;
    }
    if (total && (!a.ids || !a.buf)) return AQUA_ERR_INVALID;
    if (a.buf % 16) return AQUA_ERR_INVALID;
    if (a.img_offsets)
        for (uint32_t k = 0; k < a.num_seqs; ++k)
            if (a.img_offsets[k] % 16) return AQUA_ERR_INVALID;
    if (a.img_blocks)
        for (uint32_t k = 0; k < a.num_seqs; ++k)
            if (a.img_blocks[k] < a.offs[k + 1] - a.offs[k]) return AQUA_ERR_INVALID;
    if (a.num_layers == 0 ? a.first_layer != 0
                          : (uint64_t)a.first_layer + a.num_layers > s.L)
        return AQUA_ERR_INVALID;

    // -- range
    for (uint64_t j = 0; j < total; ++j)
        if (a.ids[j] < 0 || (uint32_t)a.ids[j] >= s.N) return AQUA_ERR_RANGE;

    // -- duplicate
    if (a.is_in) {
        if (marks.mark.size() < s.N) {
            marks.mark.assign(s.N, 0);
            marks.epoch = 0;
        }
        if (++marks.epoch == 0) {  // wrapped: clear and restart
            std::fill(marks.mark.begin(), marks.mark.end(), 0);
            marks.epoch = 1;
        }
        for (uint64_t j = 0; j < total; ++j) {
            uint32_t& m = marks.mark[(uint32_t)a.ids[j]];
            if (m == marks.epoch) return AQUA_ERR_DUPLICATE;
            m = marks.epoch;
        }
    } else if (a.img_offsets) {
        // Packed images never overlap; placed ones must not either.
        std::vector<std::pair<uint64_t, uint64_t>> r;
        image_ranges(s, a, &r);
        std::sort(r.begin(), r.end());
        for (size_t k = 1; k < r.size(); ++k)
            if (r[k].first < r[k - 1].second) return AQUA_ERR_DUPLICATE;
    }

    // -- capacity (128-bit so that absurd tables cannot wrap around)
    unsigned __int128 packed = 0;
    for (uint32_t k = 0; k < a.num_seqs; ++k) {
        const uint64_t m = image_blocks(a, k);
        const unsigned __int128 len = (unsigned __int128)s.L * m * s.C;
        const unsigned __int128 off =
            a.img_offsets ? (unsigned __int128)a.img_offsets[k] : packed;
        packed += len;
        if (a.offs[k + 1] == a.offs[k]) continue;
        if (off + len > a.buf_bytes) return AQUA_ERR_CAPACITY;
    }
    return AQUA_OK;
}

void image_ranges(const Shape& s, const CallArgs& a,
                  std::vector<std::pair<uint64_t, uint64_t>>* out) {
    out->clear();
    for (uint32_t k = 0; k < a.num_seqs; ++k) {
        if (a.offs[k + 1] == a.offs[k]) continue;
        const uint64_t lo = image_offset(s, a, k);
        out->emplace_back(lo, lo + (uint64_t)s.L * image_blocks(a, k) * s.C);
    }
}

size_t plan_runs(const Shape& s, const CallArgs& a, uint64_t max_unit_bytes,
                 std::vector<RunDesc>* out) {
    const size_t before = out->size();
    const uint64_t max_run = std::max<uint64_t>(1, max_unit_bytes / s.C);
    // At most one run per block: size once, fill through a pointer (a
    // push_back per run measured several times slower), then trim.
    out->resize(before + (size_t)(a.num_seqs ? a.offs[a.num_seqs] : 0));
    RunDesc* o = out->data() + before;
    for (uint32_t k = 0; k < a.num_seqs; ++k) {
        const uint64_t first = a.offs[k], n = a.offs[k + 1] - first;
        if (!n) continue;
        const int32_t* bt = a.ids + first;
        const uint64_t base = image_offset(s, a, k);
        const uint64_t lstride = image_blocks(a, k) * s.C;
        uint64_t i = 0;
        while (i < n) {
            uint64_t len = 1;
            while (i + len < n && len < max_run &&
                   bt[i + len] == bt[i + len - 1] + 1)
                ++len;
            o->img_off = base + i * s.C;
            o->img_lstride = lstride;
            o->block = (uint32_t)bt[i];
            o->nchunks = (uint32_t)len;
            o->reserved0 = o->reserved1 = 0;
            ++o;
            i += len;
        }
    }
    out->resize((size_t)(o - out->data()));
    return out->size() - before;
}

uint32_t swap_threads(uint64_t chunk_bytes, uint32_t min_threads) {
    uint32_t lo = 64;
    while (lo < min_threads && lo < kMaxThreads) lo *= 2;
    uint32_t t = lo;
    const uint64_t want = chunk_bytes / (16ull * kUnroll);  // lanes for one pass
    while (t < kMaxThreads && t < want) t *= 2;
    return t;
}

RunOrder run_order(bool is_in, uint64_t chunk_bytes, uint64_t blocks, uint32_t num_blocks,
                   uint32_t num_seqs) {
    // Fewer blocks than two per XCD: nothing to deal out.
    if (!num_blocks || blocks < 2 * kXcdWays) return RunOrder::kTable;
    const bool dense = blocks * 1000 >= kDenseMinPermille * num_blocks;
    if (chunk_bytes >= kDealMinChunk) {
        if (is_in) return RunOrder::kSortedDealt;
        const bool long_seqs = blocks >= kDealOutMinMeanBlocks * std::max<uint64_t>(1, num_seqs);
        return dense || long_seqs ? RunOrder::kTableDealt : RunOrder::kTable;
    }
    return dense && is_in ? RunOrder::kSortedDealt : RunOrder::kTable;
}

void sort_by_block(std::vector<RunDesc>* runs, uint32_t num_blocks,
                   std::vector<uint32_t>* counts, std::vector<RunDesc>* tmp) {
    if ((uint64_t)runs->size() * kSortCountingMinRatio < num_blocks) {
        std::stable_sort(runs->begin(), runs->end(),
                         [](const RunDesc& a, const RunDesc& b) { return a.block < b.block; });
        return;
    }
    counts->assign((size_t)num_blocks + 1, 0);
    for (const RunDesc& r : *runs) ++(*counts)[r.block + 1];
    for (uint32_t b = 0; b < num_blocks; ++b) (*counts)[b + 1] += (*counts)[b];
    tmp->resize(runs->size());
    for (const RunDesc& r : *runs) (*tmp)[(*counts)[r.block]++] = r;
    runs->swap(*tmp);
}

void interleave_runs(std::vector<RunDesc>* runs, uint32_t ways, std::vector<RunDesc>* tmp) {
    const size_t n = runs->size();
    if (ways < 2 || n < 2 * (size_t)ways) return;
    // Segment s holds q + 1 runs for s < r and q runs after that, so that
    // every row of the result holds one run of each segment in turn (the
    // last row, of r runs, one of each of the first r segments).
    const size_t q = n / ways, r = n % ways;
    tmp->clear();
    tmp->reserve(n);
    for (size_t i = 0; i <= q; ++i)
        for (size_t s = 0; s < (i < q ? (size_t)ways : r); ++s)
            tmp->push_back((*runs)[s * q + std::min(s, r) + i]);
    runs->swap(*tmp);
}

bool xcd_unit_order(uint64_t chunk_bytes, bool dealt) {
    return !dealt && chunk_bytes > kXcdUnitMinChunk && chunk_bytes < kXcdUnitMaxChunk;
}

uint32_t layers_per_launch(uint32_t ndesc) {
    const uint64_t per = std::max<uint64_t>(1, (1ull << 31) / std::max<uint32_t>(1, ndesc));
    return (uint32_t)std::min<uint64_t>(per, UINT32_MAX);
}

uint32_t launch_grid(uint64_t units, uint32_t max_workgroups) {
    uint64_t g = units;
    if (max_workgroups && g > max_workgroups) g = max_workgroups;
    if (g > kMaxGrid) g = kMaxGrid;
    return (uint32_t)g;
}

aqua_status validate_migrate(uintptr_t src, uint64_t src_bytes, uintptr_t dst,
                             uint64_t dst_bytes, uint32_t n, const uint64_t* src_off,
                             const uint64_t* dst_off, const uint64_t* len) {
    if (n && (!src || !dst || !src_off || !dst_off || !len)) return AQUA_ERR_INVALID;
    if (src % 16 || dst % 16) return AQUA_ERR_INVALID;
    for (uint32_t k = 0; k < n; ++k)
        if (src_off[k] % 16 || dst_off[k] % 16 || len[k] % 16) return AQUA_ERR_INVALID;
    // Overlaps, as address intervals (sorted sweep would do; n is small).
    for (uint32_t k = 0; k < n; ++k) {
        if (!len[k]) continue;
        const unsigned __int128 d0 = (unsigned __int128)dst + dst_off[k], d1 = d0 + len[k];
        for (uint32_t q = 0; q < n; ++q) {
            if (!len[q]) continue;
            const unsigned __int128 s0 = (unsigned __int128)src + src_off[q], s1 = s0 + len[q];
            if (d0 < s1 && s0 < d1) return AQUA_ERR_DUPLICATE;
            if (q > k) {
                const unsigned __int128 e0 = (unsigned __int128)dst + dst_off[q],
                                        e1 = e0 + len[q];
                if (d0 < e1 && e0 < d1) return AQUA_ERR_DUPLICATE;
            }
        }
    }
    for (uint32_t k = 0; k < n; ++k) {
        if ((unsigned __int128)src_off[k] + len[k] > src_bytes) return AQUA_ERR_CAPACITY;
        if ((unsigned __int128)dst_off[k] + len[k] > dst_bytes) return AQUA_ERR_CAPACITY;
    }
    return AQUA_OK;
}

size_t plan_copies(uint32_t n, const uint64_t* src_off, const uint64_t* dst_off,
                   const uint64_t* len, uint64_t unit, std::vector<CopyDesc>* out) {
    const size_t before = out->size();
    unit = std::max<uint64_t>(16, unit & ~15ull);
    for (uint32_t k = 0; k < n; ++k)
        for (uint64_t o = 0; o < len[k]; o += unit) {
            CopyDesc d;
            d.src_off = src_off[k] + o;
            d.dst_off = dst_off[k] + o;
            d.len = std::min<uint64_t>(unit, len[k] - o);
            d.reserved = 0;
            out->push_back(d);
        }
    return out->size() - before;
}

// ---------------------------------------------------------------------------

void HazardTracker::reset(uint32_t num_blocks) {
    blocks_.assign(num_blocks, BlockRec{});
    more_.clear();
    ranges_.clear();
    done_.clear();
    last_.clear();
    dep_.clear();
    ticket_lane_.clear();
    head_ = 0;
    base_ = 1;
    last_ticket_ = 0;
}

void HazardTracker::ensure_lane(uint32_t lane) {
    if (lane >= done_.size()) {
        done_.resize(lane + 1, 0);
        last_.resize(lane + 1, 0);
        dep_.resize(lane + 1, 0);
    }
}

// Drops the lanes of the oldest tickets while they are complete.
void HazardTracker::prune() {
    while (head_ < ticket_lane_.size()) {
        const uint32_t m = ticket_lane_[head_];
        if (m != kNoLane && base_ > done_[m]) break;
        ++head_;
        ++base_;
    }
    // Drop the dropped entries once they are most of the vector.
    if (head_ >= 1024 && head_ * 2 >= ticket_lane_.size()) {
        ticket_lane_.erase(ticket_lane_.begin(), ticket_lane_.begin() + (ptrdiff_t)head_);
        head_ = 0;
    }
}

bool HazardTracker::idle(uint32_t lane) const {
    return lane >= done_.size() || done_[lane] >= last_[lane];
}

uint32_t LaneMap::lane_for(uintptr_t stream, const HazardTracker& t) {
    for (uint32_t m = 0; m < stream_.size(); ++m)
        if (stream_[m] == stream) return m;
    for (uint32_t m = 0; m < stream_.size(); ++m)
        if (t.idle(m)) {
            stream_[m] = stream;
            return m;
        }
    stream_.push_back(stream);
    return (uint32_t)(stream_.size() - 1);
}

uint32_t HazardTracker::lane_of(uint64_t ticket) const {
    if (ticket < base_ || ticket - base_ >= ticket_lane_.size() - head_) return kNoLane;
    const uint32_t m = ticket_lane_[head_ + (ticket - base_)];
    return (m != kNoLane && ticket > done_[m]) ? m : kNoLane;
}

bool HazardTracker::done(uint64_t ticket) const {
    return lane_of(ticket) == kNoLane;
}

uint64_t HazardTracker::completed(uint32_t lane) const {
    return lane < done_.size() ? done_[lane] : 0;
}

void HazardTracker::complete(uint32_t lane, uint64_t ticket) {
    ensure_lane(lane);
    if (ticket > done_[lane]) done_[lane] = ticket;
    prune();
}

HazardTracker::Need HazardTracker::need(uint64_t ticket, uint32_t lane) {
    if (!ticket) return Need::kNone;
    const uint32_t m = lane_of(ticket);
    if (m == kNoLane) return Need::kComplete;   // known complete: no wait
    if (m == lane) return Need::kSameLane;      // ordered by the stream itself
    if (ticket > dep_[m]) dep_[m] = ticket;
    return Need::kWait;
}

uint64_t HazardTracker::issue(uint64_t ticket, uint32_t lane, const Access& a,
                              std::vector<Dep>* deps) {
    ensure_lane(lane);
    deps->clear();
    std::fill(dep_.begin(), dep_.end(), 0);
    // Tickets skipped since the last issue were never issued: complete.
    while (base_ + (ticket_lane_.size() - head_) < ticket) ticket_lane_.push_back(kNoLane);
    ticket_lane_.push_back(lane);
    last_[lane] = ticket;
    last_ticket_ = ticket;
    uint64_t elided = 0;
    // The blocks of one call mostly name the same few earlier tickets (a
    // block's last writer and its last reader), and nothing need() reads
    // changes during the call: the answers for the last two tickets are
    // kept.  Each conflict with a complete ticket still counts.
    uint64_t memo_t[2] = {0, 0};
    Need memo[2] = {Need::kNone, Need::kNone};
    auto after = [&](uint64_t t) {
        if (!t) return;
        Need n;
        if (t == memo_t[0]) {
            n = memo[0];
        } else if (t == memo_t[1]) {
            n = memo[1];
        } else {
            n = need(t, lane);
            memo_t[1] = memo_t[0];
            memo[1] = memo[0];
            memo_t[0] = t;
            memo[0] = n;
        }
        if (n == Need::kComplete) ++elided;
    };

    // Offload ranges: drop finished records, then look for overlaps.  A
    // read conflicts with earlier writes; a write with every earlier access.
    size_t w = 0;
    for (size_t k = 0; k < ranges_.size(); ++k)
        if (!done(ranges_[k].ticket)) ranges_[w++] = ranges_[k];
    ranges_.resize(w);
    const size_t old = ranges_.size();
    for (size_t r = 0; r < a.n_ranges_read; ++r) {
        const uint64_t lo = a.ranges_read[r].first, hi = a.ranges_read[r].second;
        for (size_t k = 0; k < old; ++k) {
            const RangeRec& q = ranges_[k];
            if (q.write && q.lo < hi && lo < q.hi) after(q.ticket);
        }
    }
    for (size_t r = 0; r < a.n_ranges_written; ++r) {
        const uint64_t lo = a.ranges_written[r].first, hi = a.ranges_written[r].second;
        for (size_t k = 0; k < old; ++k) {
            const RangeRec& q = ranges_[k];
            if (q.lo < hi && lo < q.hi) after(q.ticket);
        }
    }
    if (a.n_ranges_written) {
        // A write that covers an earlier record is ordered after it, and
        // every later access that conflicts with the record conflicts with
        // the write too: the record can go.
        size_t k = 0;
        for (size_t i = 0; i < old; ++i) {
            bool covered = false;
            for (size_t r = 0; r < a.n_ranges_written && !covered; ++r)
                covered = a.ranges_written[r].first <= ranges_[i].lo &&
                          ranges_[i].hi <= a.ranges_written[r].second;
            if (!covered) ranges_[k++] = ranges_[i];
        }
        ranges_.resize(k);
    }
    for (size_t r = 0; r < a.n_ranges_read; ++r)
        ranges_.push_back({a.ranges_read[r].first, a.ranges_read[r].second, ticket, lane, false});
    for (size_t r = 0; r < a.n_ranges_written; ++r)
        ranges_.push_back(
            {a.ranges_written[r].first, a.ranges_written[r].second, ticket, lane, true});

    // Pool blocks read: after their last writer; join the readers (one
    // entry per lane, finished readers forgotten when another lane joins).
    for (size_t j = 0; j < a.n_blocks_read; ++j) {
        const uint32_t b = (uint32_t)a.blocks_read[j];
        BlockRec& r = blocks_[b];
        after(r.writer);
        if (r.reader && r.reader_lane == lane) {
            r.reader = ticket;
            continue;
        }
        if (!r.more) {
            if (!r.reader || done(r.reader)) {
                r.reader = ticket;
                r.reader_lane = lane;
            } else {
                more_[b].assign(1, Reader{lane, ticket});
                r.more = 1;
            }
            continue;
        }
        std::vector<Reader>& rd = more_[b];
        bool found = false;
        for (Reader& q : rd)
            if (q.lane == lane) {
                q.ticket = ticket;
                found = true;
            }
        if (found) continue;
        size_t k = 0;
        for (size_t i = 0; i < rd.size(); ++i)
            if (!done(rd[i].ticket)) rd[k++] = rd[i];
        rd.resize(k);
        if (!r.reader || done(r.reader)) {
            r.reader = ticket;
            r.reader_lane = lane;
        } else {
            rd.push_back({lane, ticket});
        }
        if (rd.empty()) {
            more_.erase(b);
            r.more = 0;
        }
    }
    // Pool blocks written: after their last writer and every reader since.
    for (size_t j = 0; j < a.n_blocks_written; ++j) {
        const uint32_t b = (uint32_t)a.blocks_written[j];
        BlockRec& r = blocks_[b];
        after(r.writer);
        if (r.reader && r.reader != ticket) after(r.reader);
        if (r.more) {
            const auto it = more_.find(b);
            for (const Reader& q : it->second)
                if (q.ticket != ticket) after(q.ticket);
            more_.erase(it);
            r.more = 0;
        }
        r.reader = 0;
        r.reader_lane = 0;
        r.writer = ticket;
    }

    for (uint32_t m = 0; m < dep_.size(); ++m)
        if (dep_[m]) deps->push_back({m, dep_[m]});
    return elided;
}

// ---------------------------------------------------------------------------
// RangeAllocator

void RangeAllocator::reset(uint64_t size, uint64_t align) {
    align_ = align ? align : 1;
    size_ = size - size % align_;
    free_.clear();
    used_.clear();
    if (size_) free_[0] = size_;
    free_total_ = size_;
}

bool RangeAllocator::alloc(uint64_t bytes, uint64_t* off) {
    if (!bytes) return false;
    if (bytes > UINT64_MAX - align_) return false;
    const uint64_t need = (bytes + align_ - 1) / align_ * align_;
    for (auto it = free_.begin(); it != free_.end(); ++it) {
        if (it->second < need) continue;
        const uint64_t o = it->first, len = it->second;
        free_.erase(it);
        if (len > need) free_[o + need] = len - need;
        used_[o] = need;
        free_total_ -= need;
        *off = o;
        return true;
    }
    return false;
}

bool RangeAllocator::free(uint64_t off) {
    auto u = used_.find(off);
    if (u == used_.end()) return false;
    uint64_t lo = off, len = u->second;
    used_.erase(u);
    free_total_ += len;
    auto next = free_.lower_bound(lo);
    if (next != free_.end() && next->first == lo + len) {  // merge the right neighbour
        len += next->second;
        next = free_.erase(next);
    }
    if (next != free_.begin()) {                            // merge the left neighbour
        auto prev = std::prev(next);
        if (prev->first + prev->second == lo) {
            lo = prev->first;
            len += prev->second;
            free_.erase(prev);
        }
    }
    free_[lo] = len;
    return true;
}

uint64_t RangeAllocator::largest_free() const {
    uint64_t m = 0;
    for (const auto& f : free_) m = std::max(m, f.second);
    return m;
}

uint64_t RangeAllocator::granted(uint64_t off) const {
    auto u = used_.find(off);
    return u == used_.end() ? 0 : u->second;
}

void pick_link_engines(uint32_t d2h_avail, uint32_t d2h_pref, uint32_t h2d_avail,
                       uint32_t h2d_pref, uint32_t fast, int32_t* d2h, int32_t* h2d) {
    auto lowest = [](uint32_t m) { return m ? (int32_t)__builtin_ctz(m) : -1; };
    auto candidates = [&](uint32_t avail, uint32_t pref) -> uint32_t {
        if (pref & avail) return pref & avail;
        const uint32_t f = fast ? fast : avail;
        return (f & avail) ? (f & avail) : f;
    };
    *d2h = lowest(candidates(d2h_avail, d2h_pref));
    const uint32_t m1 = candidates(h2d_avail, h2d_pref);
    const uint32_t m1x = *d2h >= 0 ? (m1 & ~(1u << *d2h)) : m1;
    *h2d = lowest(m1x ? m1x : m1);
}

}  // namespace aqua
