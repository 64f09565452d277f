/*
 * c_abi_client.c -- a plain C program that uses the swap library through
 * include/aqua.h alone, with memory and streams from the HIP runtime: no
 * Python and no torch in the process.
 *
 * It swaps two sequences of a small fp16 pool (4 layers, 64 blocks, 64 KiB
 * chunks) out to an HBM region and to pinned host memory, then back from the
 * host copy into fresh blocks, on two streams, and writes the bytes it holds
 * before and after into a directory, where the test that runs it compares
 * them with the CPU oracle:
 *
 *   pool_before.bin  the pool as filled here (xorshift64 bytes, seed 1)
 *   image_hbm.bin    the swap-out image in the HBM region
 *   image_host.bin   the swap-out image in pinned host memory
 *   pool_after.bin   the pool after the swap-in
 *
 * The block tables are fixed below (OUT_IDS, IN_IDS, OFFS).  Exit status 0
 * and a last line "c_abi_client: ok" mean every call returned AQUA_OK.
 */
#define _POSIX_C_SOURCE 200112L
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "aqua.h"

#define L 4u
#define N 64u
#define H 8u
#define T 16u
#define D 128u
#define ELEM 2u
#define CHUNK (2ull * H * T * D * ELEM)
#define POOL_BYTES ((uint64_t)L * N * CHUNK)
#define NSEQ 2u
#define NBLK 17u
#define IMG_BYTES ((uint64_t)L * NBLK * CHUNK)

static const int32_t OUT_IDS[NBLK] = {5, 9, 10, 11, 40, 2, 63, 0, 33, 34,
                                      7, 8, 20, 61, 62, 1, 3};
static const int32_t IN_IDS[NBLK] = {41, 42, 43, 44, 45, 46, 47, 48, 49, 50,
                                     51, 52, 53, 54, 55, 56, 57};
static const uint64_t OFFS[NSEQ + 1] = {0, 10, 17};

static int check_hip(hipError_t e, const char* what) {
    if (e != hipSuccess) {
        fprintf(stderr, "c_abi_client: %s: %s\n", what, hipGetErrorString(e));
        return 1;
    }
    return 0;
}

static int check_aqua(aqua_status s, const char* what) {
    if (s != AQUA_OK) {
        fprintf(stderr, "c_abi_client: %s: %s\n", what, aqua_status_str(s));
        return 1;
    }
    return 0;
}

static int dump(const char* dir, const char* name, const void* p, uint64_t n) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "wb");
    if (!f || fwrite(p, 1, n, f) != n) {
        fprintf(stderr, "c_abi_client: cannot write %s\n", path);
        if (f) fclose(f);
        return 1;
    }
    return fclose(f) != 0;
}

int main(int argc, char** argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: %s OUT_DIR\n", argv[0]);
        return 2;
    }
    const char* dir = argv[1];
    /* Before the HIP runtime starts: stream waits on the copy engines are
     * then held by the command processor (see the staged host path). */
    setenv("GPU_STREAMOPS_CP_WAIT", "1", 0);
    uint8_t* pool_h = malloc(POOL_BYTES);
    uint8_t* back = malloc(POOL_BYTES);
    uint8_t* img_h = malloc(IMG_BYTES);
    if (!pool_h || !back || !img_h) return 1;
    uint64_t x = 1;
    for (uint64_t i = 0; i < POOL_BYTES; ++i) {
        x ^= x << 13;
        x ^= x >> 7;
        x ^= x << 17;
        pool_h[i] = (uint8_t)(x >> 24);
    }

    void *pool = NULL, *region = NULL, *pinned = NULL;
    hipStream_t s_out = NULL, s_in = NULL;
    if (check_hip(hipSetDevice(0), "hipSetDevice") ||
        check_hip(hipMalloc(&pool, POOL_BYTES), "hipMalloc pool") ||
        check_hip(hipMalloc(&region, IMG_BYTES), "hipMalloc region") ||
        check_hip(hipHostMalloc(&pinned, IMG_BYTES, hipHostMallocDefault), "hipHostMalloc") ||
        check_hip(hipStreamCreate(&s_out), "hipStreamCreate") ||
        check_hip(hipStreamCreate(&s_in), "hipStreamCreate") ||
        check_hip(hipMemcpy(pool, pool_h, POOL_BYTES, hipMemcpyHostToDevice), "upload pool") ||
        check_hip(hipMemset(region, 0, IMG_BYTES), "clear region"))
        return 1;
    memset(pinned, 0, IMG_BYTES);

    const aqua_kv_desc d = {L, N, H, T, D, AQUA_F16};
    aqua_kv_pool_t kv = NULL;
    uint64_t t_dev = 0, t_host = 0, t_in = 0;
    if (check_aqua(aqua_kv_pool_create(&d, pool, POOL_BYTES, &kv), "aqua_kv_pool_create"))
        return 1;
    /* Two swap-outs of the same blocks on one stream, then a swap-in from
     * the host image on another stream: the library orders the swap-in after
     * the swap-out that writes its source. */
    if (check_aqua(aqua_swap_out(kv, NSEQ, OUT_IDS, OFFS, region, IMG_BYTES, NULL,
                                 AQUA_TARGET_DEVICE, s_out, &t_dev), "aqua_swap_out (HBM)") ||
        check_aqua(aqua_swap_out(kv, NSEQ, OUT_IDS, OFFS, pinned, IMG_BYTES, NULL,
                                 AQUA_TARGET_HOST, s_out, &t_host), "aqua_swap_out (host)") ||
        check_aqua(aqua_swap_in(kv, NSEQ, IN_IDS, OFFS, pinned, IMG_BYTES, NULL,
                                AQUA_TARGET_HOST, s_in, &t_in), "aqua_swap_in (host)") ||
        check_aqua(aqua_sync(kv, 0), "aqua_sync"))
        return 1;
    if (!(t_dev < t_host && t_host < t_in)) {
        fprintf(stderr, "c_abi_client: tickets out of order\n");
        return 1;
    }
    if (check_hip(hipMemcpy(img_h, region, IMG_BYTES, hipMemcpyDeviceToHost), "read region") ||
        check_hip(hipMemcpy(back, pool, POOL_BYTES, hipMemcpyDeviceToHost), "read pool") ||
        check_aqua(aqua_kv_pool_destroy(kv), "aqua_kv_pool_destroy"))
        return 1;
    if (dump(dir, "pool_before.bin", pool_h, POOL_BYTES) ||
        dump(dir, "image_hbm.bin", img_h, IMG_BYTES) ||
        dump(dir, "image_host.bin", pinned, IMG_BYTES) ||
        dump(dir, "pool_after.bin", back, POOL_BYTES))
        return 1;
    (void)hipStreamDestroy(s_out);
    (void)hipStreamDestroy(s_in);
    (void)hipHostFree(pinned);
    (void)hipFree(region);
    (void)hipFree(pool);
    free(pool_h);
    free(back);
    free(img_h);
    printf("c_abi_client: ok\n");
    return 0;
}
