// swap_kernels.hip -- gfx950 gather (swap-out) and scatter (swap-in) kernels.
//
// The work is pure data movement (Aqua, section 7, "Efficient context
// switching"): no arithmetic on the values, so no MFMA and no LDS.  Each
// workgroup of 1024 lanes (16 wave64s) copies one run of chunks of one
// layer; every lane moves 16-byte vectors, a wave covers 1 KiB contiguous
// per instruction, and UNROLL = 4 independent loads are issued before the
// first store, so a workgroup has 64 KiB -- one bf16 chunk -- in flight.
// The run descriptor is uniform across the workgroup and is fetched with
// scalar loads.  The offload side is written (swap-out) or read (swap-in) with
// nontemporal hints: it is touched once and should not displace the pool's
// working set in L2 and MALL.  The gather's pool loads are nontemporal too;
// the scatter's pool stores are nontemporal for chunks of 64 KiB and more,
// where that measured faster, and ordinary stores below.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "aqua_core.h"
#include "swap_kernels.h"

namespace aqua {

namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// Launch shape and cache hints.  The defaults are the shipped
// configuration; the macros exist so that measurement sweeps can build
// variants.
#ifndef AQUA_THREADS
#define AQUA_THREADS 1024
#endif
#ifndef AQUA_UNROLL
#define AQUA_UNROLL 4
#endif
#ifndef AQUA_NT_OUT_LD   // swap-out: pool loads
#define AQUA_NT_OUT_LD 1
#endif
#ifndef AQUA_NT_OUT_ST   // swap-out: image stores
#define AQUA_NT_OUT_ST 1
#endif
#ifndef AQUA_NT_IN_LD    // swap-in: image loads
#define AQUA_NT_IN_LD 1
#endif
// Swap-in pool stores: nontemporal or not is chosen per launch
// (SwapLaunch::nt_pool_store).

constexpr int kThreads = AQUA_THREADS;
constexpr int kUnroll = AQUA_UNROLL;

template <bool NT>
__device__ __forceinline__ v4u ld(const v4u* p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}

template <bool NT>
__device__ __forceinline__ void st(v4u* p, v4u v) {
    if constexpr (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}

// Copies nvec 16-byte vectors from s to d with the whole workgroup.
template <int UNROLL, bool NT_LD, bool NT_ST>
__device__ __forceinline__ void copy_span(const v4u* __restrict__ s,
                                          v4u* __restrict__ d, uint32_t nvec) {
    const uint32_t t = threadIdx.x;
    constexpr uint32_t step = kThreads * UNROLL;
    uint32_t base = 0;
    for (; base + step <= nvec; base += step) {
        v4u r[UNROLL];
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) r[j] = ld<NT_LD>(s + base + j * kThreads + t);
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) st<NT_ST>(d + base + j * kThreads + t, r[j]);
    }
    if (base < nvec) {  // ragged tail, still UNROLL loads in flight
        v4u r[UNROLL];
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) {
            const uint32_t i = base + j * kThreads + t;
            if (i < nvec) r[j] = ld<NT_LD>(s + i);
        }
#pragma unroll
        for (int j = 0; j < UNROLL; ++j) {
            const uint32_t i = base + j * kThreads + t;
            if (i < nvec) st<NT_ST>(d + i, r[j]);
        }
    }
}

// OUT: pool -> image (gather).  !OUT: image -> pool (scatter), with
// nontemporal pool stores when NT_POOL_ST.
// Work unit u in [0, units) is (layer l0 + u / ndesc, descriptor u % ndesc);
// layer l of the image side starts img_l0 layers before img_off's origin
// (0 for whole images, the first staged layer for a staging slot);
// consecutive workgroups take consecutive runs of one layer, so the image
// side of a gather is written front to back.
template <bool OUT, int UNROLL, bool NT_POOL_ST>
__global__ __launch_bounds__(kThreads) void swap_runs_kernel(
    uint8_t* __restrict__ pool, uint8_t* __restrict__ img,
    const RunDesc* __restrict__ descs, uint32_t ndesc, uint32_t l0, uint32_t img_l0,
    uint32_t units, uint64_t chunk_bytes, uint64_t pool_lstride) {
    for (uint32_t u = blockIdx.x; u < units; u += gridDim.x) {
        const uint32_t l = l0 + u / ndesc;
        const uint32_t k = u - (u / ndesc) * ndesc;
        const RunDesc dsc = descs[k];
        uint8_t* p = pool + (uint64_t)l * pool_lstride + (uint64_t)dsc.block * chunk_bytes;
        uint8_t* m = img + dsc.img_off + (uint64_t)(l - img_l0) * dsc.img_lstride;
        const uint32_t nvec = (uint32_t)((uint64_t)dsc.nchunks * chunk_bytes / 16);
        if constexpr (OUT)
            copy_span<UNROLL, AQUA_NT_OUT_LD, AQUA_NT_OUT_ST>(
                reinterpret_cast<const v4u*>(p), reinterpret_cast<v4u*>(m), nvec);
        else
            copy_span<UNROLL, AQUA_NT_IN_LD, NT_POOL_ST>(
                reinterpret_cast<const v4u*>(m), reinterpret_cast<v4u*>(p), nvec);
    }
}

// Range copy between two offload buffers (image migration): work unit u
// copies descs[u].len bytes from src + src_off to dst + dst_off.
template <int UNROLL>
__global__ __launch_bounds__(kThreads) void copy_ranges_kernel(
    const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
    const CopyDesc* __restrict__ descs, uint32_t n) {
    for (uint32_t u = blockIdx.x; u < n; u += gridDim.x) {
        const CopyDesc dsc = descs[u];
        copy_span<UNROLL, true, true>(reinterpret_cast<const v4u*>(src + dsc.src_off),
                                      reinterpret_cast<v4u*>(dst + dsc.dst_off),
                                      (uint32_t)(dsc.len / 16));
    }
}

}  // namespace

hipError_t launch_copy(const uint8_t* src, uint8_t* dst, const CopyDesc* descs, uint32_t n,
                       uint32_t max_workgroups, hipStream_t stream) {
    if (!n) return hipSuccess;
    uint32_t grid = n;
    if (max_workgroups && grid > max_workgroups) grid = max_workgroups;
    hipLaunchKernelGGL((copy_ranges_kernel<kUnroll>), dim3(grid), dim3(kThreads), 0, stream,
                       src, dst, descs, n);
    return hipGetLastError();
}

hipError_t launch_swap(const SwapLaunch& a, hipStream_t stream) {
    if (!a.ndesc || !a.num_layers) return hipSuccess;
    // Split by layers so that every launch has fewer than 2^31 units.
    const uint32_t per = (uint32_t)std::max<uint64_t>(1, (1ull << 31) / a.ndesc);
    const uint32_t end = a.first_layer + a.num_layers;
    for (uint32_t l0 = a.first_layer; l0 < end; l0 += per) {
        const uint32_t nl = std::min<uint32_t>(per, end - l0);
        const uint32_t units = nl * a.ndesc;
        uint32_t grid = units;
        if (a.max_workgroups && grid > a.max_workgroups) grid = a.max_workgroups;
        if (a.out)
            hipLaunchKernelGGL((swap_runs_kernel<true, kUnroll, false>), dim3(grid),
                               dim3(kThreads), 0, stream, a.pool, a.img, a.descs, a.ndesc, l0,
                               a.img_l0, units, a.chunk_bytes, a.pool_lstride);
        else if (a.nt_pool_store)
            hipLaunchKernelGGL((swap_runs_kernel<false, kUnroll, true>), dim3(grid),
                               dim3(kThreads), 0, stream, a.pool, a.img, a.descs, a.ndesc, l0,
                               a.img_l0, units, a.chunk_bytes, a.pool_lstride);
        else
            hipLaunchKernelGGL((swap_runs_kernel<false, kUnroll, false>), dim3(grid),
                               dim3(kThreads), 0, stream, a.pool, a.img, a.descs, a.ndesc, l0,
                               a.img_l0, units, a.chunk_bytes, a.pool_lstride);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace aqua
