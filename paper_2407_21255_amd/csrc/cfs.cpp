// Fair batch partitioning for a time-sliced, paging scheduler (Aqua,
// section 7, "Aqua's batch partitioning algorithm").  Host code only.
//
// One iteration computes at most b tokens.  The decode share d is the number
// of prompts that fit in GPU memory (capped at b), the prefill share b - d.
// Prefill chunks go to the prompts with the fewest prompt tokens computed,
// decode tokens (one per prompt) to those with the fewest tokens generated,
// and decode slots nobody uses go back to prefill in the same order.  The
// batch is closed at the first prompt whose KV blocks do not fit.
//
// Service order is a sort of packed 64-bit keys, (service << 32) | index, so
// equal service falls back to the request index with no comparator logic.
#include <algorithm>
#include <cstdint>
#include <vector>

#include "aqua.h"

namespace {

inline uint64_t blocks_for(uint64_t tokens, uint64_t T) { return (tokens + T - 1) / T; }

struct Builder {
    const aqua_cfs_request* r;
    uint64_t T;
    uint64_t mem;                    // free blocks left for the batch
    bool closed = false;             // a prompt did not fit: batch is final
    uint32_t* idx;
    uint32_t* tok;
    uint32_t len = 0;

    // Blocks request i takes if it computes x tokens this iteration.
    uint64_t cost(uint32_t i, uint64_t x) const {
        const uint64_t need = blocks_for(uint64_t(r[i].prefill_done) + r[i].generated + x, T);
        return need > r[i].held_blocks ? need - r[i].held_blocks : 0;
    }

    // Admit request i with x tokens (or grow its entry at slot `at` to x).
    bool admit(uint32_t i, uint64_t x, int64_t at) {
        const uint64_t before = at < 0 ? 0 : cost(i, tok[at]);
        const uint64_t extra = cost(i, x) - before;
        if (extra > mem) {
            closed = true;
            return false;
        }
        mem -= extra;
        if (at < 0) {
            idx[len] = i;
            tok[len] = uint32_t(x);
            ++len;
        } else {
            tok[at] = uint32_t(x);
        }
        return true;
    }
};

// Chunked prefill over `order` from position *pos with `budget` tokens;
// *open_slot is the batch slot of a prompt whose chunk was cut short (or -1).
uint64_t fill_prefill(Builder& b, const std::vector<uint64_t>& order, size_t* pos,
                      int64_t* open_slot, uint64_t budget) {
    while (budget > 0 && *pos < order.size() && !b.closed) {
        const uint32_t i = uint32_t(order[*pos]);
        const uint64_t have = *open_slot >= 0 ? b.tok[*open_slot] : 0;
        const uint64_t left = uint64_t(b.r[i].prompt_tokens) - b.r[i].prefill_done - have;
        const uint64_t x = std::min(left, budget);
        const int64_t slot = *open_slot >= 0 ? *open_slot : int64_t(b.len);
        if (!b.admit(i, have + x, *open_slot))
            break;
        budget -= x;
        if (x == left) {
            ++*pos;
            *open_slot = -1;
        } else {
            *open_slot = slot;
        }
    }
    return budget;
}

}  // namespace

extern "C" AQUA_API aqua_status aqua_cfs_partition(const aqua_cfs_request* requests,
                                                  uint32_t num_requests,
                                                  const aqua_cfs_params* params,
                                                  uint32_t* batch_index, uint32_t* batch_tokens,
                                                  uint32_t* batch_size, uint64_t* blocks_taken) {
    if (!params || !batch_size || (num_requests && (!requests || !batch_index || !batch_tokens)))
        return AQUA_ERR_INVALID;
    const aqua_cfs_params& p = *params;
    if (p.batch_tokens == 0 || p.decode_slots == 0 || p.block_tokens == 0 || p.reserved != 0)
        return AQUA_ERR_INVALID;
    std::vector<uint64_t> prefill, decode;
    for (uint32_t i = 0; i < num_requests; ++i) {
        const aqua_cfs_request& q = requests[i];
        if (q.prompt_tokens == 0 || q.prefill_done > q.prompt_tokens ||
            (q.generated > 0 && q.prefill_done < q.prompt_tokens))
            return AQUA_ERR_INVALID;
        if (q.prefill_done < q.prompt_tokens)
            prefill.push_back(uint64_t(q.prefill_done) << 32 | i);
        else
            decode.push_back(uint64_t(q.generated) << 32 | i);
    }
    std::sort(prefill.begin(), prefill.end());
    std::sort(decode.begin(), decode.end());

    Builder b{requests, p.block_tokens, p.capacity_blocks, false, batch_index, batch_tokens};
    const uint64_t d = std::min<uint64_t>(p.decode_slots, p.batch_tokens);
    size_t pos = 0;
    int64_t open_slot = -1;
    // Prefill share.
    const uint64_t p_left = fill_prefill(b, prefill, &pos, &open_slot, p.batch_tokens - d);
    // Decode share: one token for each of the d least-generated that fit.
    uint64_t used = 0;
    for (size_t j = 0; j < decode.size() && used < d && !b.closed; ++j)
        if (b.admit(uint32_t(decode[j]), 1, -1))
            ++used;
    // Unused decode slots continue the prefill order.
    if (!b.closed)
        fill_prefill(b, prefill, &pos, &open_slot, p_left + (d - used));

    *batch_size = b.len;
    if (blocks_taken)
        *blocks_taken = p.capacity_blocks - b.mem;
    return AQUA_OK;
}
