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
    const RunDesc* descs;     // device copy of the run descriptors
    uint32_t ndesc;
    uint32_t num_layers;
    uint64_t chunk_bytes;     // C
    uint64_t pool_lstride;    // N * C
    uint32_t max_workgroups;  // 0: one workgroup per (layer, run)
};

// Enqueues the copy on `stream`; returns the first launch error.
hipError_t launch_swap(const SwapLaunch& a, hipStream_t stream);

}  // namespace aqua
