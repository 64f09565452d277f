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
};

// Scatter store hint, measured on MI355X.  Nontemporal pool stores pay for
// large chunks and for launches that write much more than the 256 MB
// last-level cache holds.  A smaller launch of smaller chunks ends sooner with
// ordinary stores, which L2 and that cache partly absorb:
//   64 KiB chunks: 0-7 % shorter with nontemporal stores, 2 to 10 GiB launches;
//   32 KiB chunks: 10 % longer at 1 GiB per launch, 0.5-2 % shorter at 4.4-5 GiB;
//   16 KiB chunks: 20 % longer at 512 MiB per launch, 7 % shorter at 2.5 GiB.
constexpr uint64_t kNtPoolStoreMinChunk = 64ull << 10;
constexpr uint64_t kNtPoolStoreMinBytes = 2ull << 30;
inline bool nt_pool_store(uint64_t chunk_bytes, uint64_t launch_bytes) {
    return chunk_bytes >= kNtPoolStoreMinChunk || launch_bytes >= kNtPoolStoreMinBytes;
}

// Enqueues the copy on `stream`; returns the first launch error.
hipError_t launch_swap(const SwapLaunch& a, hipStream_t stream);

// Enqueues the range copy of `n` pieces (each at most 64 KiB, 16-byte
// multiples) from `src` to `dst`, both device-accessible addresses.
hipError_t launch_copy(const uint8_t* src, uint8_t* dst, const CopyDesc* descs, uint32_t n,
                       uint32_t max_workgroups, hipStream_t stream);

}  // namespace aqua
