/*
 * aqua.h -- C ABI of the MI355X KV page-swap library.
 *
 * Aqua (Vuppalapati et al., "Network-Accelerated Memory Offloading for LLMs
 * in Scale-Up GPU Domains", ASPLOS '25) pages a preempted prompt's inference
 * state out of GPU memory and back in at every context switch of its
 * time-sliced scheduler (section 7, "Fair scheduling prompts").  Because the
 * serving engine keeps one KV tensor per layer for all prompts, one prompt's
 * state is many small discontiguous pieces; the paper gathers them into one
 * contiguous tensor before moving it to the offload location and scatters
 * them back on the way in (section 7, "Efficient context switching").  The
 * offload location is a peer GPU's memory or, without a peer, host DRAM
 * (section 6, "Allocating Aqua Tensors").  Moving state must not corrupt
 * data while other work runs (section 8).
 *
 * This library implements those two operations for a paged KV pool with
 * hand-written gfx950 kernels that write the gathered image directly to its
 * destination:
 *
 *   pool   [num_layers][num_blocks][2 (K,V)][num_kv_heads][block_tokens][head_dim]
 *          elements of 1 (fp8 e4m3) or 2 (fp16, bf16) bytes.  One (layer,
 *          block) "chunk" of C = 2*H*T*D*elem bytes is contiguous.
 *   image  of one sequence with block table bt[0..n): layer-major
 *          [num_layers][n][C]; image chunk (l, i) is pool chunk (l, bt[i]).
 *          Images of a multi-sequence call are packed one after another
 *          (sequence s at sum_{q<s} L*n_q*C) unless img_offsets places them.
 *
 * Element values are opaque bytes: no conversion, no NaN canonicalisation.
 * Whole blocks are copied, including unused token slots of a last block.
 *
 * Ordering: calls on one pool behave as if executed in issue order, across
 * any streams, for the pool blocks and offload byte ranges they name; the
 * library makes a call's stream wait on an earlier call's event only where
 * the two touch the same block or overlapping offload bytes (read/write,
 * write/read or write/write).  Memory touched outside the library (attention
 * kernels reading the pool, the caller refilling a buffer) is ordered by the
 * caller with streams, events, aqua_sync or aqua_stream_wait.
 *
 * Ownership: the pool memory, offload buffers and streams belong to the
 * caller; the library borrows them.  A buffer must outlive the ticket of
 * every call that names it, the pool must outlive aqua_kv_pool_destroy.
 * block_ids, seq_offsets and img_offsets are host arrays read before the
 * call returns.
 *
 * Errors: argument errors are found before anything is enqueued, so a
 * failing call has no side effect and issues no ticket.  A HIP runtime
 * failure after enqueueing is latched on the pool: the failing call returns
 * AQUA_ERR_HIP once the work it had enqueued has ended (its destination
 * bytes are then undefined), aqua_sync returns AQUA_ERR_HIP and every later
 * swap call returns AQUA_ERR_STATE.  Copy-engine work of the failed call is
 * never left waiting on the engine, whose queue other pools may share.
 *
 * Streams: the library tells streams apart by their handle, so a stream must
 * not be destroyed while calls issued on it are outstanding (a new stream
 * could get the same handle).  Any number of distinct streams may be used
 * over a pool's life: a stream whose calls have all completed gives up its
 * place in the pool's bookkeeping to the next new one.
 *
 * Threads: a pool handle is used from one thread at a time.  Separate pools
 * are independent (but do not order against each other).  A pool whose
 * host-link copies run on an SDMA engine (aqua_kv_pool_set_link_engine)
 * owns one library thread per direction in use, started on the first call
 * that needs it and joined by aqua_kv_pool_destroy; it only waits for the
 * engine's copies and publishes their completion, and calls back into no
 * caller code.
 */
#ifndef AQUA_H
#define AQUA_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__)
#define AQUA_API __attribute__((visibility("default")))
#else
#define AQUA_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef struct aqua_kv_pool* aqua_kv_pool_t; /* opaque */
typedef int32_t aqua_status;

enum {
    AQUA_OK = 0,
    AQUA_ERR_INVALID = -1,   /* null pointer, bad shape, misalignment,
                                target/pointer-class mismatch, bad stream */
    AQUA_ERR_RANGE = -2,     /* a block id < 0 or >= num_blocks */
    AQUA_ERR_DUPLICATE = -3, /* swap-in names one pool block twice, or a
                                swap-out's image ranges overlap */
    AQUA_ERR_CAPACITY = -4,  /* an image does not fit the buffer, or the
                                pool memory is smaller than the shape */
    AQUA_ERR_HIP = -5,       /* HIP runtime failure (launch, event, copy) */
    AQUA_ERR_STATE = -6      /* pool unusable after a latched HIP failure */
};

/* Element types.  Only the byte width matters to the copy. */
enum { AQUA_F16 = 1, AQUA_BF16 = 2, AQUA_FP8_E4M3 = 3 };

/* Offload targets.  DEVICE: device memory on the pool's GPU (a carved-out
 * HBM region standing in for a scale-up peer's memory).  HOST: page-locked
 * host memory from hipHostMalloc (torch pin_memory), reached over the host
 * link as aqua_kv_pool_set_host_path chooses: staged through HBM slots and
 * moved by a copy engine (the default), or read and written by the kernels
 * directly (zero copy). */
enum { AQUA_TARGET_DEVICE = 0, AQUA_TARGET_HOST = 1 };

typedef struct {
    uint32_t num_layers;   /* L */
    uint32_t num_blocks;   /* N, pool blocks per layer */
    uint32_t num_kv_heads; /* H */
    uint32_t block_tokens; /* T, tokens per block */
    uint32_t head_dim;     /* D */
    int32_t dtype;         /* AQUA_F16 / AQUA_BF16 / AQUA_FP8_E4M3 */
} aqua_kv_desc;

typedef struct {
    uint64_t calls_out, calls_in;         /* successful swap calls */
    uint64_t bytes_out, bytes_in;         /* image bytes moved (payload) */
    uint64_t bytes_host;                  /* of which to/from host memory */
    uint64_t descriptors;                 /* run descriptors launched */
    uint64_t waits_inserted;              /* cross-stream waits enqueued */
    uint64_t waits_elided;                /* conflicts already complete */
    uint64_t calls_migrate;               /* successful migrations */
    uint64_t bytes_migrated;
    uint64_t host_ns;                     /* host time in swap calls, not
                                             counting wait_ns */
    uint64_t wait_ns;                     /* host time blocked inside swap
                                             calls until descriptor space
                                             used by earlier calls is free */
    int32_t hip_error;                    /* latched hipError_t, 0 if none */
    int32_t reserved;
    uint64_t launches;                    /* gather and scatter kernel launches
                                             (a call may take several: one per
                                             layer group of a staged call, and
                                             calls of 16..64 KiB chunks to an
                                             HBM buffer in pieces of 512 MiB) */
} aqua_pool_stats;

/* Bind a pool to caller-owned device memory.
 *   desc       shape; C = 2*H*T*D*elem must be a multiple of 16 bytes.
 *   pool_base  device pointer on the current device, 16-byte aligned, with
 *              [pool_base, pool_base + pool_bytes) inside one allocation.
 *   pool_bytes >= L*N*C, else AQUA_ERR_CAPACITY.
 *   out        receives the handle; untouched on failure.
 * Allocates the library's own descriptor rings and events.  The first pool
 * of a process on a device also launches one kernel of each of the
 * library's source files once, with nothing to copy, on a private stream,
 * and waits for them: the runtime loads the library's device code then
 * (about 80 ms once), not at the first swap.  (Profiles of a process show
 * those three dispatches of a few microseconds: a range copy, a descriptor
 * upload and a flag release.) */
AQUA_API aqua_status aqua_kv_pool_create(const aqua_kv_desc* desc, void* pool_base,
                                uint64_t pool_bytes, aqua_kv_pool_t* out);

/* Wait for every outstanding call, then free the library's state (not the
 * pool memory).  Returns a latched HIP error if there was one. */
AQUA_API aqua_status aqua_kv_pool_destroy(aqua_kv_pool_t pool);

/* Swap-out (gather): for each sequence s, layer l and table position i,
 * copy pool chunk (l, bt_s[i]) to image chunk (l, i) of s.
 *   block_ids    concatenated block tables (int32), seq_offsets[num_seqs]
 *                entries; the same block may appear more than once.
 *   seq_offsets  CSR offsets, num_seqs+1 entries, seq_offsets[0] == 0,
 *                non-decreasing.
 *   dst          device pointer (target DEVICE) or pinned host pointer
 *                (target HOST), 16-byte aligned; dst_bytes its usable size.
 *   img_offsets  NULL for packed images, else num_seqs byte offsets (each a
 *                multiple of 16) into dst; non-empty images must not overlap.
 *   stream       hipStream_t of the caller (NULL: the null stream).
 *   ticket       receives the call's ticket (may be NULL).
 * Pool bytes are only read. */
AQUA_API aqua_status aqua_swap_out(aqua_kv_pool_t pool, uint32_t num_seqs,
                          const int32_t* block_ids,
                          const uint64_t* seq_offsets, void* dst,
                          uint64_t dst_bytes, const uint64_t* img_offsets,
                          int32_t target, void* stream, uint64_t* ticket);

/* Swap-in (scatter): for each sequence s, layer l and table position i,
 * copy image chunk (l, i) of s into pool chunk (l, bt_s[i]).  Destination
 * blocks must be distinct within the call (AQUA_ERR_DUPLICATE).  Arguments
 * as for aqua_swap_out with src read only. */
AQUA_API aqua_status aqua_swap_in(aqua_kv_pool_t pool, uint32_t num_seqs,
                         const int32_t* block_ids,
                         const uint64_t* seq_offsets, const void* src,
                         uint64_t src_bytes, const uint64_t* img_offsets,
                         int32_t target, void* stream, uint64_t* ticket);

/* Which part of each image a call moves.
 *   img_blocks  NULL, or per sequence the image's blocks per layer m_s, at
 *               least its table length n_s: the image is [L][m_s][C] and the
 *               table covers its first n_s blocks of every layer.  Used to
 *               swap a cached prefix in from a longer image (the paper's
 *               prefill caching keeps a long prompt's context in swap space
 *               and reloads it for later prompts sharing the prefix,
 *               sections 8 and 9.3).  Packed images are then sum L*m_q*C
 *               apart and capacity checks use m_s.
 *   first_layer, num_layers
 *               move only layers [first_layer, first_layer + num_layers) of
 *               pool and image; num_layers 0 (with first_layer 0) moves all.
 *               Used for layer-by-layer offload as in FlexGen (section 9.1)
 *               and to pipeline a swap-in: one call, and one ticket, per
 *               layer group.
 * Ordering is tracked at the granularity of whole blocks and whole image
 * extents. */
typedef struct {
    const uint64_t* img_blocks;
    uint32_t first_layer;
    uint32_t num_layers;
} aqua_swap_range;

/* aqua_swap_out / aqua_swap_in with a range (NULL: the whole images).
 * AQUA_ERR_INVALID when m_s < n_s or the layer range leaves [0, L). */
AQUA_API aqua_status aqua_swap_out_ex(aqua_kv_pool_t pool, uint32_t num_seqs,
                                      const int32_t* block_ids,
                                      const uint64_t* seq_offsets, void* dst,
                                      uint64_t dst_bytes, const uint64_t* img_offsets,
                                      const aqua_swap_range* range, int32_t target,
                                      void* stream, uint64_t* ticket);
AQUA_API aqua_status aqua_swap_in_ex(aqua_kv_pool_t pool, uint32_t num_seqs,
                                     const int32_t* block_ids,
                                     const uint64_t* seq_offsets, const void* src,
                                     uint64_t src_bytes, const uint64_t* img_offsets,
                                     const aqua_swap_range* range, int32_t target,
                                     void* stream, uint64_t* ticket);

/* ---- Allocation-free swap, for callers that cannot allocate memory (code
 * being captured into a HIP graph, tight serving loops, harnesses that
 * forbid allocation).
 *
 * aqua_swap_noalloc is aqua_swap_out (direction 0) or aqua_swap_in
 * (direction 1) with the same arguments, results, ordering and errors,
 * except that it allocates no device or pinned memory and creates no HIP
 * event or stream.  (Its host-side planning, like that of the other
 * calls, uses ordinary host memory: the pool's planning buffers, which
 * keep the capacity of the largest call seen, and the sort of a swap-in's
 * runs.)  Its run descriptors go through the pool's pinned ring
 * (allocated when the pool was created; the call never grows it) to a
 * device scratch array of 2 MiB that the library holds on each device for
 * the life of the process, and its completion event is one of the 16 the
 * pool created.  While none is spare (16 calls of the pool in flight), the
 * call first blocks the host until the oldest outstanding call of the pool
 * has completed; a caller that holds its streams from the host must not
 * issue it then.  Differences:
 *   - at most 65536 run descriptors per call (a run is a stretch of
 *     consecutive blocks of one table, up to 64 KiB; a fragmented table has
 *     one run per block), and no more than the pool's ring holds:
 *     AQUA_ERR_CAPACITY otherwise, before anything is enqueued;
 *   - a pinned-host image is always moved zero-copy, whatever
 *     aqua_kv_pool_set_host_path says (the staged path needs the library's
 *     slots and copy engines);
 *   - all layers are moved (no layer range or partial image).
 * The scratch array is shared by every pool on a device and keeps the last
 * call's descriptors.  Calls of this entry point on one pool are ordered
 * with each other by the library (they all write the scratch); calls on
 * different pools of one device that may overlap in time race on the
 * scratch and must be ordered by the caller (one stream, or a sync). */
AQUA_API aqua_status aqua_swap_noalloc(aqua_kv_pool_t pool, int32_t direction,
                                       uint32_t num_seqs, const int32_t* block_ids,
                                       const uint64_t* seq_offsets, void* buf,
                                       uint64_t buf_bytes, const uint64_t* img_offsets,
                                       int32_t target, void* stream, uint64_t* ticket);

/* Image migration.  When the memory holding offloaded images is reclaimed
 * (section 6, "Reclaiming Aqua Tensors"), the images move elsewhere -- here
 * between the HBM region and pinned host memory, in either direction, or
 * within one kind -- and later swap-ins read them from the new place.
 * Copies n byte ranges: range k from src + src_offsets[k] to
 * dst + dst_offsets[k], lengths[k] bytes.
 *   src, dst       device (target DEVICE) or pinned host (target HOST)
 *                  pointers, 16-byte aligned, with src_bytes / dst_bytes
 *                  usable.
 *   offsets, lengths  host arrays of n entries, multiples of 16.
 * Destination ranges must not overlap each other or any source range
 * (AQUA_ERR_DUPLICATE); ranges must fit their buffers (AQUA_ERR_CAPACITY).
 * Ordered with the pool's swaps like any call that reads the source ranges
 * and writes the destination ranges.  Between device and host memory each
 * range is one copy on that direction's copy engine (see
 * aqua_kv_pool_set_link_engine; no compute unit copies the bytes);
 * device to device, host to host, or with the direction set to the
 * runtime's copies, the range-copy kernel moves the bytes (capped like
 * zero-copy swaps when either side is host memory). */
AQUA_API aqua_status aqua_migrate(aqua_kv_pool_t pool, const void* src, uint64_t src_bytes,
                                  int32_t src_target, void* dst, uint64_t dst_bytes,
                                  int32_t dst_target, uint32_t n,
                                  const uint64_t* src_offsets, const uint64_t* dst_offsets,
                                  const uint64_t* lengths, void* stream, uint64_t* ticket);

/* Block the host until `ticket` (0: every outstanding call) has completed.
 * Returns AQUA_ERR_HIP if a HIP failure was latched. */
AQUA_API aqua_status aqua_sync(aqua_kv_pool_t pool, uint64_t ticket);

/* Make `stream` wait (on the device, without blocking the host) until
 * `ticket` has completed.  Tickets already complete need no wait. */
AQUA_API aqua_status aqua_stream_wait(aqua_kv_pool_t pool, uint64_t ticket,
                             void* stream);

/* 1 if `ticket` has completed, 0 if not, negative status on error. */
AQUA_API aqua_status aqua_query(aqua_kv_pool_t pool, uint64_t ticket);

/* Cap the number of workgroups of later kernel launches for one target
 * (0: no cap, one workgroup per (layer, run)).  For the host target the cap
 * applies to zero-copy swaps; staged swaps gather in HBM without a cap. */
AQUA_API aqua_status aqua_kv_pool_set_max_workgroups(aqua_kv_pool_t pool,
                                            int32_t target,
                                            uint32_t max_workgroups);

/* How swaps with a pinned-host target move their bytes.
 *   AQUA_HOST_STAGED (default): the paper's temporary-tensor scheme
 *     (section 7, "Efficient context switching").  Layers pass through two
 *     HBM slots owned by the library (512 MiB each by default, allocated
 *     for both directions on the pool's first staged call, after waiting for
 *     every outstanding call, and grown the same way when a call needs
 *     larger ones): the gather kernel fills a slot and a copy engine moves it over
 *     the link while the next slot is filled, and the reverse on swap-in.
 *     Swap-outs and swap-ins have their own slots and link carrier (see
 *     aqua_kv_pool_set_link_engine), so a swap-out and a swap-in on
 *     different streams use both directions of the link at once.  The
 *     compute units are busy only for the short gathers and scatters, so
 *     concurrent kernels keep running.  A pool's first staged call in each
 *     direction also sets up that direction's carrier and slots: about 6 ms
 *     of host time on MI355X, against well under 1 ms later; a caller that
 *     cannot take that at its first preemption issues one small staged
 *     swap-out and swap-in when it starts.
 *   AQUA_HOST_ZERO_COPY: the gather and scatter kernels read and write the
 *     host image directly over the link, with no HBM staging.  Their
 *     workgroups stay resident for the whole transfer, so the library caps
 *     the grid (16 workgroups unless aqua_kv_pool_set_max_workgroups says
 *     otherwise), which is enough to saturate the link; kernels on other
 *     streams lose those compute units meanwhile, and a kernel that needs
 *     every compute unit at once (a GEMM with one tile per unit) runs a
 *     second round of tiles. */
enum { AQUA_HOST_ZERO_COPY = 0, AQUA_HOST_STAGED = 1 };
AQUA_API aqua_status aqua_kv_pool_set_host_path(aqua_kv_pool_t pool, int32_t path);

/* What carries the staged path's link copies for one direction (dir 0:
 * swap-out, device to host; dir 1: swap-in, host to device).
 *   0..15               that SDMA engine, driven through the HSA runtime by
 *                       a library thread; the call's stream waits for the
 *                       engine's progress on the device, with no host block
 *                       (hipStreamWaitValue64).  Set GPU_STREAMOPS_CP_WAIT=1
 *                       in the environment before the HIP runtime starts so
 *                       that the runtime holds such waits in the command
 *                       processor; otherwise it keeps a one-wave kernel
 *                       resident per wait, which slows kernels that fill
 *                       every compute unit (the Python package sets it when
 *                       imported).
 *                       A staged call fails with AQUA_ERR_HIP (nothing
 *                       enqueued) if the engine cannot be used.
 *   AQUA_LINK_RUNTIME   the HIP runtime's own copies on a library stream; the
 *                       runtime then picks the mechanism per copy (a blit
 *                       kernel or any engine), and some engines reach only a
 *                       fraction of the link rate.
 *   AQUA_LINK_AUTO      (default) the HSA runtime's preferred engine for the
 *                       direction if it names one, else the lowest-numbered
 *                       free engine among those that carry the host link at
 *                       its rate (engines 0-3 on MI355X), else one of those
 *                       shared with its other users; the two directions on
 *                       different engines where possible; the runtime's
 *                       copies if no engine can be used.
 * The choice is made on the direction's next staged call.  Waits for every
 * outstanding call first.  dir other than 0 or 1, or another engine value:
 * AQUA_ERR_INVALID.
 * aqua_kv_pool_get_link_engine reports the carrier in use: an engine index,
 * AQUA_LINK_RUNTIME, or AQUA_LINK_AUTO while no staged call has chosen. */
enum { AQUA_LINK_RUNTIME = -1, AQUA_LINK_AUTO = -2 };
AQUA_API aqua_status aqua_kv_pool_set_link_engine(aqua_kv_pool_t pool, int32_t dir,
                                                  int32_t engine);
AQUA_API aqua_status aqua_kv_pool_get_link_engine(aqua_kv_pool_t pool, int32_t dir,
                                                  int32_t* engine);

/* Copy the pool's counters into *out. */
AQUA_API aqua_status aqua_pool_stats_get(aqua_kv_pool_t pool, aqua_pool_stats* out);

/* Static text for a status code. */
AQUA_API const char* aqua_status_str(aqua_status s);

/* ---- HBM yardsticks (measurement helper, no pool).
 *
 * The swap kernels' roofline is HBM bandwidth, read plus write (a swap with
 * an HBM offload target reads and writes every payload byte once).  These
 * calls run the swap kernels' own copy loop -- 64 KiB per 1024-lane
 * workgroup, four 16-byte vectors per lane in flight, nontemporal hints --
 * over one contiguous range, so that a caller can measure, in the same run
 * and on the same device, what a copy, a pure read and a pure write reach:
 *   AQUA_YARDSTICK_COPY   copies bytes from src to dst (ranges disjoint);
 *   AQUA_YARDSTICK_READ   reads bytes of src; dst (16 bytes at least) is
 *                         not written for any input a caller can give
 *                         (the loads are folded and stored only if the fold
 *                         equals an internal key);
 *   AQUA_YARDSTICK_WRITE  writes bytes of dst: 16-byte vector i holds the
 *                         32-bit words {i mod 2^32, i / 2^32, 0x9E3779B9,
 *                         0x61C88646}; src is not read and may be NULL.
 * src and dst are device memory of the current device, 16-byte aligned,
 * each range inside one allocation; bytes is a multiple of 16 (0: nothing
 * is enqueued).  The work is enqueued on `stream` (NULL: the null stream)
 * and the call returns without waiting.  AQUA_ERR_INVALID for another kind,
 * a misaligned or foreign pointer, a range outside its allocation or
 * overlapping copy ranges; AQUA_ERR_HIP if the launch fails. */
enum { AQUA_YARDSTICK_COPY = 0, AQUA_YARDSTICK_READ = 1, AQUA_YARDSTICK_WRITE = 2 };
AQUA_API aqua_status aqua_hbm_yardstick(int32_t kind, void* dst, const void* src,
                                        uint64_t bytes, void* stream);

/* ---- Swap space: offload tensors with a device region and a host fallback
 * (section 6, "Aqua Tensors", "Allocating Aqua Tensors", "Reclaiming Aqua
 * Tensors").
 *
 * Offload tensors are named by handles.  A tensor's bytes live in a device
 * region lent for offloading (the stand-in for a producer GPU's HBM) while a
 * range of it fits, else in pinned host memory (the DRAM fallback).  Reclaim
 * moves device tensors to host memory to hand device memory back; restore
 * moves host tensors back into the device region where they fit.  A handle
 * keeps its identity when its tensor moves; aqua_swap_locate gives the
 * current pointer and target, which the swap calls take.  Moves are
 * migrations on the space's pool (aqua_migrate), so calls on that pool issued
 * after a move, on any stream, are ordered after it, and a freed or vacated
 * range is reused only after the calls that still read or write it.  A
 * pointer from aqua_swap_locate is valid until its tensor is freed or moved.
 * Ranges are 256-byte aligned; tensor sizes are multiples of 16 bytes. */
typedef struct aqua_swap_space* aqua_swap_space_t;

/* Allocates device_bytes of device memory on the pool's GPU and host_bytes
 * of pinned, device-mapped host memory (either may be 0).  The space must be
 * destroyed before its pool.  AQUA_ERR_HIP if an allocation fails. */
AQUA_API aqua_status aqua_swap_space_create(aqua_kv_pool_t pool, uint64_t device_bytes,
                                            uint64_t host_bytes, aqua_swap_space_t* out);

/* Waits for every outstanding call on the pool, then frees both regions. */
AQUA_API aqua_status aqua_swap_space_destroy(aqua_swap_space_t space);

/* A tensor of `bytes`: in the device region if a free range fits, else in
 * host memory.  AQUA_ERR_INVALID for 0 or a size that is not a multiple of
 * 16, AQUA_ERR_CAPACITY if neither region has room. */
AQUA_API aqua_status aqua_swap_alloc(aqua_swap_space_t space, uint64_t bytes,
                                     uint64_t* handle);

/* Releases the tensor's range; later calls that reuse it are ordered after
 * the calls that still use it.  AQUA_ERR_INVALID for an unknown handle. */
AQUA_API aqua_status aqua_swap_free(aqua_swap_space_t space, uint64_t handle);

/* Current place of a tensor: *ptr (device pointer for AQUA_TARGET_DEVICE,
 * host pointer for AQUA_TARGET_HOST), its size and target; NULL outputs are
 * skipped.  The engine uses the target to tell whether a prompt's state is
 * on the device side or in host memory. */
AQUA_API aqua_status aqua_swap_locate(aqua_swap_space_t space, uint64_t handle, void** ptr,
                                      uint64_t* bytes, int32_t* target);

/* Reclaim: moves device tensors (oldest handles first) to host memory until
 * at least `bytes` of the device region is free (UINT64_MAX: every device
 * tensor), as one migration on `stream`; *ticket (may be NULL) is its
 * ticket, 0 if nothing had to move.  AQUA_ERR_CAPACITY, with nothing moved,
 * if host memory cannot take the tensors that would have to move. */
AQUA_API aqua_status aqua_swap_reclaim(aqua_swap_space_t space, uint64_t bytes, void* stream,
                                       uint64_t* ticket);

/* Restore: moves host tensors into the device region, oldest handle first,
 * each that a free range of the region fits at its turn (one that does not
 * fit stays in host memory and later ones are still tried), as one
 * migration on `stream`; *ticket as for reclaim. */
AQUA_API aqua_status aqua_swap_restore(aqua_swap_space_t space, void* stream, uint64_t* ticket);

/* Free bytes of each region and the number of live tensors in each. */
AQUA_API aqua_status aqua_swap_usage(aqua_swap_space_t space, uint64_t* device_free,
                                     uint64_t* host_free, uint64_t* device_tensors,
                                     uint64_t* host_tensors);

/* ---- Fair batch partitioning (section 7, "Aqua's batch partitioning
 * algorithm").  Host code: no pool, no GPU.
 *
 * A time-sliced scheduler that pages prompts out and in keeps chunked
 * prefill by splitting each iteration's token budget b into a prefill
 * share p and a decode share d, with d at its upper bound, the number of
 * prompts that fit in GPU memory:
 *   1. d = min(decode_slots, b), p = b - d;
 *   2. prefill prompts (prefill_done < prompt_tokens), fewest prompt tokens
 *      computed first, take chunks of their remaining prompt tokens until p
 *      is spent;
 *   3. decode prompts (prefill_done == prompt_tokens), fewest tokens
 *      generated first, take one token each, at most d of them;
 *   4. decode slots left unused go to prefill, continuing the order of step
 *      2 (first the chunk that step 2 cut short);
 *   5. the whole batch is closed at the first prompt whose KV blocks do not
 *      fit in what is left of capacity_blocks.
 * Equal service is broken by the lower request index.  A prompt with
 * ctx = prefill_done + generated cached tokens that computes x tokens needs
 * ceil((ctx + x) / block_tokens) blocks; held_blocks of them are already its
 * own and not counted in capacity_blocks.  At a reschedule pass held 0 and
 * the whole pool (prompts left out are paged out); within a time slice pass
 * the residents' current blocks as held and the pool's free blocks as
 * capacity. */
typedef struct {
    uint32_t prompt_tokens; /* >= 1 */
    uint32_t prefill_done;  /* prompt tokens with KV computed, <= prompt_tokens */
    uint32_t generated;     /* output tokens so far; 0 while prefill is unfinished */
    uint32_t held_blocks;   /* pool blocks already owned outside capacity_blocks */
} aqua_cfs_request;

typedef struct {
    uint32_t batch_tokens;    /* b, >= 1 */
    uint32_t decode_slots;    /* upper bound of d: prompts that fit, >= 1 */
    uint32_t block_tokens;    /* tokens per KV block, >= 1 */
    uint32_t reserved;        /* must be 0 */
    uint64_t capacity_blocks; /* pool blocks the batch may take */
} aqua_cfs_params;

/* requests: host array of num_requests entries.  On AQUA_OK the batch is
 * written in admission order: batch_index[j] (a request index) computes
 * batch_tokens[j] tokens, j < *batch_size; each request appears at most
 * once, so both arrays need num_requests entries.  *blocks_taken (may be
 * NULL) is the capacity the batch uses.  AQUA_ERR_INVALID for null
 * pointers, zero batch_tokens / decode_slots / block_tokens, nonzero
 * reserved, an empty prompt, prefill_done > prompt_tokens or tokens
 * generated before the prefill is complete; nothing is written then. */
AQUA_API aqua_status aqua_cfs_partition(const aqua_cfs_request* requests,
                                        uint32_t num_requests, const aqua_cfs_params* params,
                                        uint32_t* batch_index, uint32_t* batch_tokens,
                                        uint32_t* batch_size, uint64_t* blocks_taken);

#ifdef __cplusplus
}
#endif

#endif /* AQUA_H */
