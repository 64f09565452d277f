// swap_kernels.h -- launch interface of the gather/scatter kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "aqua_core.h"

namespace aqua {

struct SwapLaunch {
    bool out;                 // true: pool -> image, false: image -> pool
    uint8_t* pool;            // device pointer of the pool base
    uint8_t* img;             // device-accessible pointer of the buffer base
    uint32_t img_l0;          // layer l's image data starts at img_off + (l - img_l0) * lstride
    const RunDesc* descs;     // device copy of the run descriptors
    uint32_t ndesc;
    uint32_t first_layer;     // layers [first_layer, first_layer + num_layers)
    uint32_t num_layers;
    uint64_t chunk_bytes;     // C
    uint64_t pool_lstride;    // N * C
    uint32_t max_workgroups;  // 0: one workgroup per (layer, run)
    bool nt_pool_store;       // scatter: nontemporal stores into the pool
    uint32_t threads;         // lanes per workgroup: 64, 128, 256, 512 or 1024
    bool xcd_order;           // one-pass launches: each XCD takes a contiguous eighth of units
};

// Scatter store hint, measured on MI355X.  Nontemporal pool stores pay for
// large chunks and for calls that write much more than the 256 MB last-level
// cache holds.  A smaller call of smaller chunks ends sooner with ordinary
// stores, which L2 and that cache partly absorb:
//   64 KiB chunks: 0-7 % shorter with nontemporal stores, 2 to 10 GiB calls;
//   32 KiB chunks: 10 % longer at 1 GiB per call, 0.5-2 % shorter at 4.4-5 GiB;
//   16 KiB chunks: 20 % longer at 512 MiB per call, 7 % shorter at 2.5 GiB.
// The bytes are the whole call's, also when several launches carry it: ordinary
// stores chosen for each 512 MiB launch of a larger call made its scatter
// 2-15 % longer.
constexpr uint64_t kNtPoolStoreMinChunk = 64ull << 10;
constexpr uint64_t kNtPoolStoreMinBytes = 2ull << 30;
inline bool nt_pool_store(uint64_t chunk_bytes, uint64_t call_bytes) {
    return chunk_bytes >= kNtPoolStoreMinChunk || call_bytes >= kNtPoolStoreMinBytes;
}

// Enqueues the copy on `stream`; returns the first launch error.  Adds the
// number of kernel launches it made to *launches when that is given.
hipError_t launch_swap(const SwapLaunch& a, hipStream_t stream, uint64_t* launches = nullptr);

// Enqueues one HBM yardstick over `bytes` (a multiple of 16) of device
// memory with the swap kernels' copy loop: mode 0 copies src to dst, mode 1
// reads src only, mode 2 writes dst only (see aqua_hbm_yardstick).
hipError_t launch_yardstick(int mode, const uint8_t* src, uint8_t* dst, uint64_t bytes,
                            uint32_t key, hipStream_t stream);

// Enqueues the range copy of `n` pieces (each at most 64 KiB, 16-byte
// multiples) from `src` to `dst`, both device-accessible addresses.
hipError_t launch_copy(const uint8_t* src, uint8_t* dst, const CopyDesc* descs, uint32_t n,
                       uint32_t max_workgroups, hipStream_t stream);

}  // namespace aqua
