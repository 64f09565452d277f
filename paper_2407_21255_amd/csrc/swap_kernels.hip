// swap_kernels.hip -- gfx950 gather (swap-out) and scatter (swap-in) kernels.
//
// The work is pure data movement (Aqua, section 7, "Efficient context
// switching"): no arithmetic on the values, so no MFMA and no LDS.  Each
// workgroup copies one run of chunks of one layer at a time; every lane
// moves 16-byte vectors, a wave covers 1 KiB contiguous per instruction,
// and kUnroll = 4 independent loads are issued before the first store, so a
// workgroup of 1024 lanes (16 wave64s) holds one 64 KiB bf16 chunk in flight.
// The kernels also come in 512, 256, 128 and 64 lanes, so that a launch can
// size the workgroup to a smaller chunk and keep kUnroll loads in flight
// per lane; on MI355X that measured no faster for 32 KiB chunks and 4 %
// slower for 16 KiB ones than 1024 lanes with idle lanes in the last pass,
// so the library launches 1024 lanes by default (swap_threads).
// The run descriptor is uniform across the workgroup and is fetched with
// scalar loads.  The offload side is written (swap-out) or read (swap-in) with
// nontemporal hints: it is touched once and should not displace the pool's
// working set in L2 and MALL.  The gather's pool loads are nontemporal too;
// the scatter's pool stores are nontemporal for chunks of 64 KiB and more
// and for calls that write 2 GiB or more, where that measured faster, and
// ordinary otherwise (nt_pool_store).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "aqua_core.h"
#include "swap_kernels.h"

namespace aqua {

namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// Cache hints.  The defaults are the shipped configuration; the macros
// exist so that measurement sweeps can build variants.
#ifndef AQUA_NT_OUT_LD   // swap-out: pool loads
#define AQUA_NT_OUT_LD 1
#endif
#ifndef AQUA_NT_OUT_ST   // swap-out: image stores
#define AQUA_NT_OUT_ST 1
#endif
#ifndef AQUA_NT_IN_LD    // swap-in: image loads
#define AQUA_NT_IN_LD 1
#endif
// Swap-in pool stores: nontemporal or not is chosen per call
// (SwapLaunch::nt_pool_store).
#ifndef AQUA_YS_NT       // yardsticks: nontemporal loads and stores
#define AQUA_YS_NT 1
#endif

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

// Copies nvec 16-byte vectors from s to d with the whole workgroup of
// THREADS lanes: full passes of THREADS * kUnroll vectors, each lane's loads
// all issued before its first store, then one partial pass in which a lane
// copies only those of its kUnroll vectors that fall inside the span.  In the
// partial pass the gfx950 code waits for each conditional load before issuing
// the next; a form without lane branches that kept them all in flight
// measured no faster on 32 and 16 KiB chunks (within 1 %; one 32 KiB
// gather 2.5 % slower), and neither did workgroups that copy two 32 KiB
// units with all four loads of each lane in flight (1.5-8 % slower).
template <int THREADS, bool NT_LD, bool NT_ST>
__device__ __forceinline__ void copy_span(const v4u* __restrict__ s,
                                          v4u* __restrict__ d, uint32_t nvec) {
    const uint32_t t = threadIdx.x;
    constexpr uint32_t step = THREADS * kUnroll;
    uint32_t base = 0;
    for (; base + step <= nvec; base += step) {
        v4u r[kUnroll];
#pragma unroll
        for (int j = 0; j < (int)kUnroll; ++j) r[j] = ld<NT_LD>(s + base + j * THREADS + t);
#pragma unroll
        for (int j = 0; j < (int)kUnroll; ++j) st<NT_ST>(d + base + j * THREADS + t, r[j]);
    }
    if (base < nvec) {
        v4u r[kUnroll];
#pragma unroll
        for (int j = 0; j < (int)kUnroll; ++j) {
            const uint32_t i = base + j * THREADS + t;
            if (i < nvec) r[j] = ld<NT_LD>(s + i);
        }
#pragma unroll
        for (int j = 0; j < (int)kUnroll; ++j) {
            const uint32_t i = base + j * THREADS + t;
            if (i < nvec) st<NT_ST>(d + i, r[j]);
        }
    }
}

// OUT: pool -> image (gather).  !OUT: image -> pool (scatter), with
// nontemporal pool stores when NT_POOL_ST.
// Work unit u in [0, units) is (layer l0 + u / ndesc, descriptor u % ndesc);
// layer l of the image side starts img_l0 layers before img_off's origin
// (0 for whole images, the first staged layer for a staging slot).  In
// plain order consecutive workgroups take consecutive units; with xcd_order
// each XCD takes a contiguous eighth of them (xcd_unit), and the host may
// have dealt each layer's runs out to the XCDs already (interleave_runs).
template <bool OUT, bool NT_POOL_ST, int THREADS>
__global__ __launch_bounds__(THREADS) void swap_runs_kernel(
    uint8_t* __restrict__ pool, uint8_t* __restrict__ img,
    const RunDesc* __restrict__ descs, uint32_t ndesc, uint32_t l0, uint32_t img_l0,
    uint32_t units, uint64_t chunk_bytes, uint64_t pool_lstride, uint32_t xcd_order) {
    // With one workgroup per unit, xcd_order gives each XCD (workgroups go
    // to the 8 XCDs in turn) a contiguous eighth of the units.
    const uint32_t u0 =
        (xcd_order && gridDim.x == units) ? xcd_unit(blockIdx.x, units) : blockIdx.x;
    for (uint32_t u = u0; u < units; u += gridDim.x) {
        const uint32_t l = l0 + u / ndesc;
        const uint32_t k = u - (u / ndesc) * ndesc;
        const RunDesc dsc = descs[k];
        uint8_t* p = pool + (uint64_t)l * pool_lstride + (uint64_t)dsc.block * chunk_bytes;
        uint8_t* m = img + dsc.img_off + (uint64_t)(l - img_l0) * dsc.img_lstride;
        const uint32_t nvec = (uint32_t)((uint64_t)dsc.nchunks * chunk_bytes / 16);
        if constexpr (OUT)
            copy_span<THREADS, AQUA_NT_OUT_LD, AQUA_NT_OUT_ST>(
                reinterpret_cast<const v4u*>(p), reinterpret_cast<v4u*>(m), nvec);
        else
            copy_span<THREADS, AQUA_NT_IN_LD, NT_POOL_ST>(
                reinterpret_cast<const v4u*>(m), reinterpret_cast<v4u*>(p), nvec);
    }
}

// Range copy between two offload buffers (image migration): work unit u
// copies descs[u].len bytes from src + src_off to dst + dst_off.
__global__ __launch_bounds__(kMaxThreads) void copy_ranges_kernel(
    const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
    const CopyDesc* __restrict__ descs, uint32_t n) {
    for (uint32_t u = blockIdx.x; u < n; u += gridDim.x) {
        const CopyDesc dsc = descs[u];
        copy_span<kMaxThreads, true, true>(reinterpret_cast<const v4u*>(src + dsc.src_off),
                                           reinterpret_cast<v4u*>(dst + dsc.dst_off),
                                           (uint32_t)(dsc.len / 16));
    }
}

// HBM yardsticks over nvec contiguous vectors, in 64 KiB pieces with the
// swap kernels' lane shape and hints.  MODE 0 copies src to dst, MODE 1 only
// reads src (the vectors are folded together and stored to dst only if the
// fold equals a key no real input produces, so the loads stay), MODE 2 only
// writes dst: vector i holds {i low, i high, key, ~key}.
template <int MODE>
__global__ __launch_bounds__(kMaxThreads) void yardstick_kernel(
    const v4u* __restrict__ src, v4u* __restrict__ dst, uint64_t nvec, uint32_t key) {
    constexpr uint32_t per = kMaxThreads * kUnroll;
    const uint64_t units = (nvec + per - 1) / per;
    const uint32_t t = threadIdx.x;
    v4u acc = {0u, 0u, 0u, 0u};
    for (uint64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const uint64_t base = u * per;
        const uint32_t n = (uint32_t)std::min<uint64_t>(per, nvec - base);
        if constexpr (MODE == 0) {
            copy_span<kMaxThreads, AQUA_YS_NT, AQUA_YS_NT>(src + base, dst + base, n);
        } else if constexpr (MODE == 1) {
            v4u r[kUnroll];
#pragma unroll
            for (int j = 0; j < (int)kUnroll; ++j) {
                const uint32_t i = j * kMaxThreads + t;
                r[j] = i < n ? ld<AQUA_YS_NT>(src + base + i) : v4u{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int j = 0; j < (int)kUnroll; ++j) acc ^= r[j];
        } else {
#pragma unroll
            for (int j = 0; j < (int)kUnroll; ++j) {
                const uint32_t i = j * kMaxThreads + t;
                const uint64_t g = base + i;
                if (i < n)
                    st<AQUA_YS_NT>(dst + g, v4u{(uint32_t)g, (uint32_t)(g >> 32), key, ~key});
            }
        }
    }
    if constexpr (MODE == 1) {
        if (acc.x == key && acc.y == ~key && acc.z == key && acc.w == ~key) dst[0] = acc;
    }
}

template <int THREADS>
void launch_swap_t(const SwapLaunch& a, uint32_t grid, uint32_t l0, uint32_t units,
                   hipStream_t stream) {
    if (a.out)
        hipLaunchKernelGGL((swap_runs_kernel<true, false, THREADS>), dim3(grid), dim3(THREADS),
                           0, stream, a.pool, a.img, a.descs, a.ndesc, l0, a.img_l0, units,
                           a.chunk_bytes, a.pool_lstride, (uint32_t)a.xcd_order);
    else if (a.nt_pool_store)
        hipLaunchKernelGGL((swap_runs_kernel<false, true, THREADS>), dim3(grid), dim3(THREADS),
                           0, stream, a.pool, a.img, a.descs, a.ndesc, l0, a.img_l0, units,
                           a.chunk_bytes, a.pool_lstride, (uint32_t)a.xcd_order);
    else
        hipLaunchKernelGGL((swap_runs_kernel<false, false, THREADS>), dim3(grid), dim3(THREADS),
                           0, stream, a.pool, a.img, a.descs, a.ndesc, l0, a.img_l0, units,
                           a.chunk_bytes, a.pool_lstride, (uint32_t)a.xcd_order);
}

}  // namespace

hipError_t launch_copy(const uint8_t* src, uint8_t* dst, const CopyDesc* descs, uint32_t n,
                       uint32_t max_workgroups, hipStream_t stream) {
    if (!n) return hipSuccess;
    hipLaunchKernelGGL(copy_ranges_kernel, dim3(launch_grid(n, max_workgroups)),
                       dim3(kMaxThreads), 0, stream, src, dst, descs, n);
    return hipGetLastError();
}

hipError_t launch_swap(const SwapLaunch& a, hipStream_t stream, uint64_t* launches) {
    if (!a.ndesc || !a.num_layers) return hipSuccess;
    // Whole layers per launch, fewer than 2^31 units each.
    const uint32_t per = layers_per_launch(a.ndesc);
    const uint32_t end = a.first_layer + a.num_layers;
    for (uint32_t l0 = a.first_layer; l0 < end; l0 += per) {
        const uint32_t nl = std::min<uint32_t>(per, end - l0);
        const uint32_t units = nl * a.ndesc;
        const uint32_t grid = launch_grid(units, a.max_workgroups);
        switch (a.threads) {
            case 1024: launch_swap_t<1024>(a, grid, l0, units, stream); break;
            case 512: launch_swap_t<512>(a, grid, l0, units, stream); break;
            case 256: launch_swap_t<256>(a, grid, l0, units, stream); break;
            case 128: launch_swap_t<128>(a, grid, l0, units, stream); break;
            case 64: launch_swap_t<64>(a, grid, l0, units, stream); break;
            default: return hipErrorInvalidValue;
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (launches) ++*launches;
    }
    return hipSuccess;
}

hipError_t launch_yardstick(int mode, const uint8_t* src, uint8_t* dst, uint64_t bytes,
                            uint32_t key, hipStream_t stream) {
    const uint64_t nvec = bytes / 16;
    if (!nvec) return hipSuccess;
    const uint64_t per = (uint64_t)kMaxThreads * kUnroll;
    const uint32_t grid = launch_grid((nvec + per - 1) / per, 0);
    const v4u* s = reinterpret_cast<const v4u*>(src);
    v4u* d = reinterpret_cast<v4u*>(dst);
    switch (mode) {
        case 0: hipLaunchKernelGGL(yardstick_kernel<0>, dim3(grid), dim3(kMaxThreads), 0, stream,
                                   s, d, nvec, key); break;
        case 1: hipLaunchKernelGGL(yardstick_kernel<1>, dim3(grid), dim3(kMaxThreads), 0, stream,
                                   s, d, nvec, key); break;
        case 2: hipLaunchKernelGGL(yardstick_kernel<2>, dim3(grid), dim3(kMaxThreads), 0, stream,
                                   s, d, nvec, key); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace aqua
