/*
 * The loader used from plain C, with no Python and no torch in the process:
 * open a converted checkpoint, load it into hipMalloc'd memory with both
 * engines (cached in a pool and streamed from the file, file layout and a
 * 256-byte device layout), copy the image back and compare it with the
 * expected bytes, look tensors up through the index, and check that
 * destinations outside one device allocation are refused.
 *
 *   c_load <checkpoint dir> <expected file image> <expected A2=256 image> <chunk size>
 *
 * The expected images are written by the test from the oracle.  Prints
 * "ok" and exits 0 when every byte matches.
 */
#define __HIP_PLATFORM_AMD__
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "sllm.h"

static unsigned char* slurp(const char* path, size_t* n) {
    FILE* f = fopen(path, "rb");
    if (!f) return NULL;
    fseek(f, 0, SEEK_END);
    long len = ftell(f);
    fseek(f, 0, SEEK_SET);
    unsigned char* p = (unsigned char*)malloc(len > 0 ? (size_t)len : 1);
    if (p && len > 0 && fread(p, 1, (size_t)len, f) != (size_t)len) {
        free(p);
        p = NULL;
    }
    fclose(f);
    *n = (size_t)(len > 0 ? len : 0);
    return p;
}

#define CHECK(cond, ...)                  \
    do {                                  \
        if (!(cond)) {                    \
            printf("FAIL: " __VA_ARGS__); \
            printf("\n");                 \
            return 1;                     \
        }                                 \
    } while (0)

/* one load through a fresh handle; compares the whole image */
static int load_and_compare(const char* dir, sllm_pool* pool, uint32_t engine, uint64_t a2, uint64_t chunk,
                            const unsigned char* want, size_t want_n) {
    sllm_open_opts o;
    memset(&o, 0, sizeof o);
    o.pool = pool;
    o.engine = engine;
    o.dev_alignment = a2;
    o.chunk_size = pool ? 0 : chunk;
    o.ring_slots = 3;
    o.io_threads = 2;
    sllm_ckpt* h = NULL;
    int32_t st = sllm_open(dir, &o, &h);
    CHECK(st == SLLM_OK, "sllm_open: %s", sllm_last_error());
    const uint64_t total = sllm_total_bytes(h);
    CHECK(total == want_n, "total %llu, expected %zu", (unsigned long long)total, want_n);
    unsigned char* dev = NULL;
    CHECK(hipMalloc((void**)&dev, total + 64) == hipSuccess, "hipMalloc");
    CHECK(hipMemset(dev, 0xA5, total + 64) == hipSuccess, "hipMemset");
    hipStream_t s;
    CHECK(hipStreamCreate(&s) == hipSuccess, "hipStreamCreate");
    st = sllm_load(h, dev, total, s);
    CHECK(st == SLLM_OK, "sllm_load: %s", sllm_last_error());
    CHECK(hipStreamSynchronize(s) == hipSuccess, "hipStreamSynchronize");
    unsigned char* got = (unsigned char*)malloc(total + 64);
    CHECK(got != NULL, "malloc");
    CHECK(hipMemcpy(got, dev, total + 64, hipMemcpyDeviceToHost) == hipSuccess, "hipMemcpy");
    CHECK(memcmp(got, want, total) == 0, "engine %u A2 %llu %s: image differs", engine, (unsigned long long)a2,
          pool ? "cached" : "streamed");
    for (int i = 0; i < 64; ++i) CHECK(got[total + i] == 0xA5, "byte past the image written");

    /* the index: every entry's bytes sit at base + offset */
    uint64_t n = 0;
    CHECK(sllm_tensor_index(h, NULL, 0, &n) == SLLM_OK, "sllm_tensor_index count");
    sllm_tensor_info* info = (sllm_tensor_info*)calloc(n ? n : 1, sizeof *info);
    CHECK(sllm_tensor_index(h, info, n, &n) == SLLM_OK, "sllm_tensor_index");
    for (uint64_t i = 0; i < n; ++i) {
        sllm_tensor_info one;
        CHECK(sllm_tensor_find(h, info[i].name, &one) == SLLM_OK, "sllm_tensor_find %s", info[i].name);
        CHECK(one.offset == info[i].offset && one.nbytes == info[i].nbytes, "find/index disagree for %s",
              info[i].name);
        CHECK(one.offset + one.nbytes <= total, "tensor %s past the image", info[i].name);
    }
    sllm_tensor_info none;
    CHECK(sllm_tensor_find(h, "no such tensor", &none) == SLLM_E_NOTFOUND, "missing tensor found");
    free(info);
    free(got);
    CHECK(hipStreamDestroy(s) == hipSuccess, "hipStreamDestroy");
    CHECK(hipFree(dev) == hipSuccess, "hipFree");
    CHECK(sllm_close(h) == SLLM_OK, "sllm_close: %s", sllm_last_error());
    return 0;
}

/* Destinations the load must refuse before any device work: a range that
 * runs 16 bytes past the end of its allocation (as the runtime reports the
 * allocation), fewer bytes than the image, an address that is not 16-byte
 * aligned, and host memory.  The allocation keeps its fill byte throughout;
 * then a load into the allocation's last `total` bytes succeeds. */
static int refusals(const char* dir, uint64_t chunk, const unsigned char* want, size_t want_n) {
    sllm_open_opts o;
    memset(&o, 0, sizeof o);
    o.chunk_size = chunk;
    o.ring_slots = 3;
    o.io_threads = 2;
    sllm_ckpt* h = NULL;
    CHECK(sllm_open(dir, &o, &h) == SLLM_OK, "sllm_open: %s", sllm_last_error());
    const uint64_t total = sllm_total_bytes(h);
    CHECK(total == want_n && total > 0, "total %llu", (unsigned long long)total);
    const size_t alloc = (size_t)total + 4096;
    unsigned char* dev = NULL;
    CHECK(hipMalloc((void**)&dev, alloc) == hipSuccess, "hipMalloc");
    CHECK(hipMemset(dev, 0x5A, alloc) == hipSuccess, "hipMemset");
    CHECK(hipDeviceSynchronize() == hipSuccess, "hipDeviceSynchronize");
    void* base = NULL;
    size_t size = 0;
    CHECK(hipMemGetAddressRange(&base, &size, dev) == hipSuccess && base == dev && size >= alloc,
          "hipMemGetAddressRange");
    /* 16-byte aligned, ending 1-16 bytes past what the runtime counts as the allocation */
    const size_t over_off = ((size - total) / 16 + 1) * 16;
    unsigned char* over = (unsigned char*)base + over_off;
    CHECK(sllm_load(h, over, total, NULL) == SLLM_E_RANGE, "load past the allocation: %s", sllm_last_error());
    CHECK(sllm_load(h, dev, total - 1, NULL) == SLLM_E_RANGE, "short destination accepted");
    CHECK(sllm_load(h, dev + 8, total, NULL) == SLLM_E_INVAL, "unaligned destination accepted");
    unsigned char* host = (unsigned char*)malloc(total);
    CHECK(host != NULL, "malloc");
    CHECK(sllm_load(h, host, total, NULL) == SLLM_E_INVAL, "host destination accepted");
    CHECK(hipDeviceSynchronize() == hipSuccess, "hipDeviceSynchronize");
    unsigned char* back = (unsigned char*)malloc(alloc);
    CHECK(back != NULL, "malloc");
    CHECK(hipMemcpy(back, dev, alloc, hipMemcpyDeviceToHost) == hipSuccess, "hipMemcpy");
    for (size_t i = 0; i < alloc; ++i) CHECK(back[i] == 0x5A, "a refused load wrote byte %zu", i);
    /* the allocation's last `total` bytes (16-byte aligned as `alloc - total` is) */
    CHECK(sllm_load(h, dev + alloc - total, total, NULL) == SLLM_OK, "load at the end: %s", sllm_last_error());
    CHECK(hipDeviceSynchronize() == hipSuccess, "hipDeviceSynchronize");
    CHECK(hipMemcpy(back, dev, alloc, hipMemcpyDeviceToHost) == hipSuccess, "hipMemcpy");
    CHECK(memcmp(back + alloc - total, want, total) == 0, "load at the end: image differs");
    for (size_t i = 0; i < alloc - total; ++i) CHECK(back[i] == 0x5A, "byte %zu before the image written", i);
    free(back);
    free(host);
    CHECK(hipFree(dev) == hipSuccess, "hipFree");
    CHECK(sllm_close(h) == SLLM_OK, "sllm_close: %s", sllm_last_error());
    return 0;
}

int main(int argc, char** argv) {
    if (argc != 5) {
        printf("usage: c_load <dir> <expected image> <expected A2=256 image> <chunk size>\n");
        return 2;
    }
    const char* dir = argv[1];
    const uint64_t chunk = strtoull(argv[4], NULL, 10);
    size_t n1 = 0, n2 = 0;
    unsigned char* want1 = slurp(argv[2], &n1);
    unsigned char* want2 = slurp(argv[3], &n2);
    CHECK(want1 && want2, "cannot read the expected images");
    CHECK(hipSetDevice(0) == hipSuccess, "hipSetDevice");
    printf("images %zu / %zu bytes\n", n1, n2);
    fflush(stdout);

    sllm_pool* pool = NULL;
    CHECK(sllm_pool_create(chunk, n1 / chunk + 2, 0, &pool) == SLLM_OK, "sllm_pool_create: %s", sllm_last_error());
    CHECK(sllm_pool_cache(pool, dir, 2, 0) == SLLM_OK, "sllm_pool_cache: %s", sllm_last_error());
    const uint32_t engines[2] = {SLLM_ENGINE_KERNEL, SLLM_ENGINE_SDMA};
    for (int e = 0; e < 2; ++e) {
        if (load_and_compare(dir, pool, engines[e], 0, chunk, want1, n1)) return 1;
        if (load_and_compare(dir, pool, engines[e], 256, chunk, want2, n2)) return 1;
        if (load_and_compare(dir, NULL, engines[e], 0, chunk, want1, n1)) return 1;
        if (load_and_compare(dir, NULL, engines[e], 256, chunk, want2, n2)) return 1;
        printf("engine %u ok\n", engines[e]);
        fflush(stdout);
    }
    if (refusals(dir, chunk, want1, n1)) return 1;
    printf("refusals ok\n");
    fflush(stdout);
    CHECK(sllm_pool_evict(pool, dir) == SLLM_OK, "sllm_pool_evict: %s", sllm_last_error());
    CHECK(sllm_pool_destroy(pool) == SLLM_OK, "sllm_pool_destroy: %s", sllm_last_error());
    free(want1);
    free(want2);
    printf("ok\n");
    return 0;
}
