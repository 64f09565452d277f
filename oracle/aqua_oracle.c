/*
 * aqua_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU reference for the two operations on
 * the KV page-swap path of Aqua (Vuppalapati et al., ASPLOS '25):
 *
 *   swap-out  gather a preempted prompt's KV blocks, which live scattered
 *             across one pool tensor per layer, into one contiguous offload
 *             image (paper section 7, "Efficient context switching": the
 *             small per-layer pieces are gathered into a single tensor
 *             before the bulk copy to the offload location);
 *   swap-in   scatter such an image back into pool blocks (same paragraph:
 *             the offloaded data is brought back and scattered to the small
 *             per-layer tensors).
 *
 * The "_ex" forms move a subset of layers (a layer-by-layer offload as in
 * FlexGen, section 9.1) or only the first blocks of a longer image (a cached
 * prefix, sections 8 and 9.3); migrate moves an image between buffers.
 *
 * The paper stores one KV tensor per layer holding every prompt (section 7,
 * same paragraph) on top of vLLM's paged attention (section 10).  The pool
 * here is therefore [layers][blocks][K|V][kv_heads][block_tokens][head_dim]
 * and one (layer, block) "chunk" of C = 2*H*T*D*e bytes is contiguous.
 * The image of one sequence is layer-major, [layers][n_s][C], so that
 * image(l, i) holds pool chunk (l, bt[i]).  The paper never fixes the image
 * layout; this reading keeps every layer's segment contiguous.
 *
 * Only tests, the smoke check and the bench's CPU-baseline leg may call
 * this file.  It shares no code, header or constant with the GPU library.
 *
 * Status codes (identical numbers on both sides so that error parity can be
 * tested; the values are restated here, not included):
 *    0 ok, -1 invalid argument, -2 block id out of range,
 *   -3 duplicate destination, -4 capacity (image does not fit the buffer).
 * Validation precedence is invalid -> range -> duplicate -> capacity, and a
 * failing call changes no byte.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    uint32_t num_layers;
    uint32_t num_blocks;
    uint32_t num_kv_heads;
    uint32_t block_tokens;
    uint32_t head_dim;
    int32_t dtype; /* 1 fp16, 2 bf16, 3 fp8 e4m3 */
} oracle_kv_desc;

enum {
    ORACLE_OK = 0,
    ORACLE_ERR_INVALID = -1,
    ORACLE_ERR_RANGE = -2,
    ORACLE_ERR_DUPLICATE = -3,
    ORACLE_ERR_CAPACITY = -4
};

/* Bytes of one element: fp16 and bf16 are two bytes, fp8 e4m3 one. */
static uint64_t elem_bytes(int32_t dtype)
{
    if (dtype == 1 || dtype == 2) return 2;
    if (dtype == 3) return 1;
    return 0;
}

/* C = 2 (K and V) * kv_heads * block_tokens * head_dim * element bytes. */
uint64_t oracle_chunk_bytes(const oracle_kv_desc* d)
{
    if (!d) return 0;
    return 2ull * d->num_kv_heads * d->block_tokens * d->head_dim *
           elem_bytes(d->dtype);
}

/* Bytes of KV state per token: every layer stores one K and one V vector
 * per KV head. */
uint64_t oracle_bytes_per_token(const oracle_kv_desc* d)
{
    if (!d) return 0;
    return (uint64_t)d->num_layers * 2ull * d->num_kv_heads * d->head_dim *
           elem_bytes(d->dtype);
}

static int desc_ok(const oracle_kv_desc* d)
{
    if (!d) return 0;
    if (d->num_layers == 0 || d->num_blocks == 0 || d->num_kv_heads == 0 ||
        d->block_tokens == 0 || d->head_dim == 0)
        return 0;
    if (elem_bytes(d->dtype) == 0) return 0;
    if (oracle_chunk_bytes(d) % 16 != 0) return 0;
    return 1;
}

/* Pool creation check: the same shape and size rules the library applies. */
int oracle_pool_check(const oracle_kv_desc* d, const void* pool,
                      uint64_t pool_bytes)
{
    if (!desc_ok(d) || !pool || ((uintptr_t)pool % 16) != 0)
        return ORACLE_ERR_INVALID;
    uint64_t need = (uint64_t)d->num_layers * d->num_blocks *
                    oracle_chunk_bytes(d);
    if (pool_bytes < need) return ORACLE_ERR_CAPACITY;
    return ORACLE_OK;
}

/* Blocks per layer in sequence s's image: the caller's figure, or its table
 * length. */
static uint64_t image_blocks(uint32_t s, const uint64_t* seq_offsets,
                             const uint64_t* img_blocks)
{
    return img_blocks ? img_blocks[s] : seq_offsets[s + 1] - seq_offsets[s];
}

/* Byte offset of sequence s's image inside the offload buffer: the caller's
 * offset, or the packed offset sum_{q<s} L*m_q*C. */
static uint64_t image_offset(const oracle_kv_desc* d, uint32_t s,
                             const uint64_t* seq_offsets,
                             const uint64_t* img_offsets,
                             const uint64_t* img_blocks)
{
    if (img_offsets) return img_offsets[s];
    uint64_t off = 0;
    for (uint32_t q = 0; q < s; q++)
        off += (uint64_t)d->num_layers * image_blocks(q, seq_offsets, img_blocks) *
               oracle_chunk_bytes(d);
    return off;
}

/* Common validation of one swap call.  is_in selects the swap-in rules
 * (destination blocks must be distinct); for swap-out the destinations are
 * the image ranges, which must not overlap each other.  img_blocks (may be
 * NULL) gives each image's blocks per layer, at least its table length;
 * layers [l0, l0 + nl) are moved, nl == 0 meaning every layer. */
static int validate(const oracle_kv_desc* d, const void* pool,
                    uint64_t pool_bytes, uint32_t num_seqs,
                    const int32_t* block_ids, const uint64_t* seq_offsets,
                    const void* buf, uint64_t buf_bytes,
                    const uint64_t* img_offsets, const uint64_t* img_blocks,
                    uint32_t l0, uint32_t nl, int is_in)
{
    int st = oracle_pool_check(d, pool, pool_bytes);
    if (st != ORACLE_OK) return st;
    if (num_seqs > 0 && !seq_offsets) return ORACLE_ERR_INVALID;
    uint64_t total = num_seqs ? seq_offsets[num_seqs] : 0;
    if (num_seqs > 0) {
        if (seq_offsets[0] != 0) return ORACLE_ERR_INVALID;
        for (uint32_t s = 0; s < num_seqs; s++)
            if (seq_offsets[s + 1] < seq_offsets[s]) return ORACLE_ERR_INVALID;
    }
    if (total > 0 && (!block_ids || !buf)) return ORACLE_ERR_INVALID;
    if (((uintptr_t)buf % 16) != 0) return ORACLE_ERR_INVALID;
    if (img_offsets)
        for (uint32_t s = 0; s < num_seqs; s++)
            if (img_offsets[s] % 16 != 0) return ORACLE_ERR_INVALID;
    if (img_blocks)
        for (uint32_t s = 0; s < num_seqs; s++)
            if (img_blocks[s] < seq_offsets[s + 1] - seq_offsets[s])
                return ORACLE_ERR_INVALID;
    if (nl == 0 ? l0 != 0 : ((uint64_t)l0 + nl > d->num_layers))
        return ORACLE_ERR_INVALID;

    for (uint64_t j = 0; j < total; j++)
        if (block_ids[j] < 0 || (uint64_t)block_ids[j] >= d->num_blocks)
            return ORACLE_ERR_RANGE;

    uint64_t C = oracle_chunk_bytes(d);
    if (is_in) {
        /* Two writes to one pool block in a single call: rejected. */
        for (uint64_t j = 0; j < total; j++)
            for (uint64_t k = j + 1; k < total; k++)
                if (block_ids[j] == block_ids[k]) return ORACLE_ERR_DUPLICATE;
    } else {
        /* Two non-empty image ranges of one swap-out that overlap would be
         * written twice: rejected the same way. */
        for (uint32_t s = 0; s < num_seqs; s++) {
            uint64_t ns = image_blocks(s, seq_offsets, img_blocks);
            if (seq_offsets[s + 1] == seq_offsets[s]) continue;
            uint64_t a0 = image_offset(d, s, seq_offsets, img_offsets, img_blocks);
            uint64_t a1 = a0 + (uint64_t)d->num_layers * ns * C;
            for (uint32_t q = s + 1; q < num_seqs; q++) {
                uint64_t nq = image_blocks(q, seq_offsets, img_blocks);
                if (seq_offsets[q + 1] == seq_offsets[q]) continue;
                uint64_t b0 = image_offset(d, q, seq_offsets, img_offsets, img_blocks);
                uint64_t b1 = b0 + (uint64_t)d->num_layers * nq * C;
                if (a0 < b1 && b0 < a1) return ORACLE_ERR_DUPLICATE;
            }
        }
    }

    for (uint32_t s = 0; s < num_seqs; s++) {
        if (seq_offsets[s + 1] == seq_offsets[s]) continue;
        uint64_t ms = image_blocks(s, seq_offsets, img_blocks);
        uint64_t off = image_offset(d, s, seq_offsets, img_offsets, img_blocks);
        uint64_t len = (uint64_t)d->num_layers * ms * C;
        if (off > buf_bytes || len > buf_bytes - off) return ORACLE_ERR_CAPACITY;
    }
    return ORACLE_OK;
}

/* Swap-out: for every sequence s, layer l and table position i, copy pool
 * chunk (l, bt_s[i]) to image chunk (l, i) of s, which sits at
 * off_s + (l * m_s + i) * C with m_s the image's blocks per layer.  Only
 * layers [l0, l0 + nl) move (all when nl == 0).  Pool is read only. */
int oracle_swap_out_ex(const oracle_kv_desc* d, const void* pool,
                       uint64_t pool_bytes, uint32_t num_seqs,
                       const int32_t* block_ids, const uint64_t* seq_offsets,
                       void* dst, uint64_t dst_bytes,
                       const uint64_t* img_offsets, const uint64_t* img_blocks,
                       uint32_t l0, uint32_t nl)
{
    int st = validate(d, pool, pool_bytes, num_seqs, block_ids, seq_offsets,
                      dst, dst_bytes, img_offsets, img_blocks, l0, nl, 0);
    if (st != ORACLE_OK) return st;
    const uint64_t C = oracle_chunk_bytes(d);
    const uint64_t N = d->num_blocks;
    const uint64_t l1 = nl ? (uint64_t)l0 + nl : d->num_layers;
    const unsigned char* p = (const unsigned char*)pool;
    unsigned char* img = (unsigned char*)dst;
    for (uint32_t s = 0; s < num_seqs; s++) {
        const int32_t* bt = block_ids + seq_offsets[s];
        uint64_t ns = seq_offsets[s + 1] - seq_offsets[s];
        uint64_t ms = image_blocks(s, seq_offsets, img_blocks);
        uint64_t off = image_offset(d, s, seq_offsets, img_offsets, img_blocks);
        for (uint64_t l = l0; l < l1; l++)
            for (uint64_t i = 0; i < ns; i++)
                memcpy(img + off + (l * ms + i) * C,
                       p + (l * N + (uint64_t)bt[i]) * C, C);
    }
    return ORACLE_OK;
}

/* Swap-in: for every sequence s, layer l in [l0, l0 + nl) and table
 * position i, copy image chunk (l, i) of s into pool chunk (l, bt_s[i]).
 * The image is read only. */
int oracle_swap_in_ex(const oracle_kv_desc* d, void* pool, uint64_t pool_bytes,
                      uint32_t num_seqs, const int32_t* block_ids,
                      const uint64_t* seq_offsets, const void* src,
                      uint64_t src_bytes, const uint64_t* img_offsets,
                      const uint64_t* img_blocks, uint32_t l0, uint32_t nl)
{
    int st = validate(d, pool, pool_bytes, num_seqs, block_ids, seq_offsets,
                      src, src_bytes, img_offsets, img_blocks, l0, nl, 1);
    if (st != ORACLE_OK) return st;
    const uint64_t C = oracle_chunk_bytes(d);
    const uint64_t N = d->num_blocks;
    const uint64_t l1 = nl ? (uint64_t)l0 + nl : d->num_layers;
    unsigned char* p = (unsigned char*)pool;
    const unsigned char* img = (const unsigned char*)src;
    for (uint32_t s = 0; s < num_seqs; s++) {
        const int32_t* bt = block_ids + seq_offsets[s];
        uint64_t ns = seq_offsets[s + 1] - seq_offsets[s];
        uint64_t ms = image_blocks(s, seq_offsets, img_blocks);
        uint64_t off = image_offset(d, s, seq_offsets, img_offsets, img_blocks);
        for (uint64_t l = l0; l < l1; l++)
            for (uint64_t i = 0; i < ns; i++)
                memcpy(p + (l * N + (uint64_t)bt[i]) * C,
                       img + off + (l * ms + i) * C, C);
    }
    return ORACLE_OK;
}

int oracle_swap_out(const oracle_kv_desc* d, const void* pool,
                    uint64_t pool_bytes, uint32_t num_seqs,
                    const int32_t* block_ids, const uint64_t* seq_offsets,
                    void* dst, uint64_t dst_bytes, const uint64_t* img_offsets)
{
    return oracle_swap_out_ex(d, pool, pool_bytes, num_seqs, block_ids,
                              seq_offsets, dst, dst_bytes, img_offsets, NULL, 0, 0);
}

int oracle_swap_in(const oracle_kv_desc* d, void* pool, uint64_t pool_bytes,
                   uint32_t num_seqs, const int32_t* block_ids,
                   const uint64_t* seq_offsets, const void* src,
                   uint64_t src_bytes, const uint64_t* img_offsets)
{
    return oracle_swap_in_ex(d, pool, pool_bytes, num_seqs, block_ids,
                             seq_offsets, src, src_bytes, img_offsets, NULL, 0, 0);
}

/* Image migration (an offloaded image moving when its holder reclaims the
 * memory, section 6 "Reclaiming Aqua Tensors"): copy n byte ranges,
 * range k from src + src_off[k] to dst + dst_off[k], lengths len[k].
 * Offsets and lengths are multiples of 16 and inside their buffers;
 * destination ranges must not overlap each other or any source range
 * (compared as addresses).  Copies run in order. */
int oracle_migrate(const void* src, uint64_t src_bytes, void* dst,
                   uint64_t dst_bytes, uint32_t n, const uint64_t* src_off,
                   const uint64_t* dst_off, const uint64_t* len)
{
    if (n > 0 && (!src || !dst || !src_off || !dst_off || !len))
        return ORACLE_ERR_INVALID;
    if (((uintptr_t)src % 16) != 0 || ((uintptr_t)dst % 16) != 0)
        return ORACLE_ERR_INVALID;
    for (uint32_t k = 0; k < n; k++)
        if (src_off[k] % 16 || dst_off[k] % 16 || len[k] % 16)
            return ORACLE_ERR_INVALID;
    for (uint32_t k = 0; k < n; k++) {
        if (!len[k]) continue;
        uintptr_t d0 = (uintptr_t)dst + dst_off[k], d1 = d0 + len[k];
        for (uint32_t q = 0; q < n; q++) {
            if (!len[q]) continue;
            uintptr_t s0 = (uintptr_t)src + src_off[q], s1 = s0 + len[q];
            if (d0 < s1 && s0 < d1) return ORACLE_ERR_DUPLICATE;
            if (q > k) {
                uintptr_t e0 = (uintptr_t)dst + dst_off[q], e1 = e0 + len[q];
                if (d0 < e1 && e0 < d1) return ORACLE_ERR_DUPLICATE;
            }
        }
    }
    for (uint32_t k = 0; k < n; k++) {
        if (src_off[k] > src_bytes || len[k] > src_bytes - src_off[k])
            return ORACLE_ERR_CAPACITY;
        if (dst_off[k] > dst_bytes || len[k] > dst_bytes - dst_off[k])
            return ORACLE_ERR_CAPACITY;
    }
    for (uint32_t k = 0; k < n; k++)
        memcpy((unsigned char*)dst + dst_off[k],
               (const unsigned char*)src + src_off[k], len[k]);
    return ORACLE_OK;
}
