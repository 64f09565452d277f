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

// Scatter store hint for a pool of chunk_bytes-sized chunks: measured on
// MI355X, nontemporal pool stores shorten the scatter by up to 5 % for 64 KiB
// chunks and lengthen it by 10 % for the 32 KiB chunks of an fp8 pool.
constexpr uint64_t kNtPoolStoreMinChunk = 64ull << 10;

// Enqueues the copy on `stream`; returns the first launch error.
hipError_t launch_swap(const SwapLaunch& a, hipStream_t stream);

// Enqueues the range copy of `n` pieces (each at most 64 KiB, 16-byte
// multiples) from `src` to `dst`, both device-accessible addresses.
hipError_t launch_copy(const uint8_t* src, uint8_t* dst, const CopyDesc* descs, uint32_t n,
                       uint32_t max_workgroups, hipStream_t stream);

}  // namespace aqua
