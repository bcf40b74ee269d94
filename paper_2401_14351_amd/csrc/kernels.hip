// gfx950 kernels of the loader.
//
// K1 (chunk gather, file layout): moves partition chunks from pinned host
// chunks, which the GPU reads directly through their device mapping, into the
// HBM image.  It is the kernel alternative to the copy engines for the
// DRAM-to-GPU step of Sec. 4.2, where pinned host memory is copied straight
// into GPU memory.  Reads of host memory cross PCIe with microsecond latency,
// so each lane keeps 16-byte loads in flight and a persistent grid streams
// tiles.
#include <hip/hip_runtime.h>

#include <cstdlib>

#include "common.hpp"
#include "hip_util.hpp"
#include "kernels.hpp"

namespace sllm {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kThreads = 256;  // 4 wave64 per workgroup
constexpr uint32_t kVec = 16;       // bytes per lane access

struct GatherArgs {
    uint8_t* dst;
    const uint8_t* const* table;
    const uint8_t* single;
    uint64_t chunk;
    uint64_t total;
    uint64_t first_chunk;
    uint32_t tiles_per_chunk;
    uint32_t n_tiles;
    // a batch of chunks from separate slots, passed inline (batch_n > 0)
    uint32_t batch_n;
    const uint8_t* batch_src[kGatherBatch];
    uint64_t batch_chunk[kGatherBatch];
};

template <bool NT>
__device__ __forceinline__ u32x4 load16(const uint8_t* p) {
    const u32x4* q = reinterpret_cast<const u32x4*>(p);
    if constexpr (NT) return __builtin_nontemporal_load(q);
    return *q;
}

template <bool NT>
__device__ __forceinline__ void store16(uint8_t* p, u32x4 v) {
    u32x4* q = reinterpret_cast<u32x4*>(p);
    if constexpr (NT) {
        __builtin_nontemporal_store(v, q);
    } else {
        *q = v;
    }
}

// Tile t of the launch covers bytes [j * tile, (j + 1) * tile) of chunk
// first_chunk + c, with c = t / tiles_per_chunk and j = t % tiles_per_chunk.
// Requires C % 16 == 0 and a 16-byte aligned dst, so every 16-byte vector of
// a chunk is aligned on both sides; only the image's last bytes (T % 16) go
// byte by byte.
template <int U, bool NT>
__global__ __launch_bounds__(kThreads) void k1_gather(GatherArgs a) {
    constexpr uint32_t kTile = kThreads * kVec * U;
    for (uint32_t t = blockIdx.x; t < a.n_tiles; t += gridDim.x) {
        const uint32_t c = t / a.tiles_per_chunk;
        const uint32_t j = t - c * a.tiles_per_chunk;
        const uint64_t k = a.batch_n ? a.batch_chunk[c] : a.first_chunk + c;
        const uint64_t base = k * a.chunk;
        if (base >= a.total) continue;
        const uint64_t len = a.total - base < a.chunk ? a.total - base : a.chunk;
        const uint8_t* src = a.batch_n ? a.batch_src[c] : a.table ? a.table[c] : a.single;
        uint8_t* dst = a.dst + base;
        const uint64_t lo = (uint64_t)j * kTile + threadIdx.x * kVec;
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t off = lo + (uint64_t)u * kThreads * kVec;
            if (off + kVec <= len) v[u] = load16<NT>(src + off);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t off = lo + (uint64_t)u * kThreads * kVec;
            if (off + kVec <= len) {
                store16<NT>(dst + off, v[u]);
            } else if (off < len) {
                for (uint64_t b = off; b < len; ++b) dst[b] = src[b];
            }
        }
    }
}

// Byte-granular form for chunk sizes that are not a multiple of 16 (test
// geometries); grid-stride over the launch's bytes.
__global__ __launch_bounds__(kThreads) void k1_gather_bytes(GatherArgs a, uint64_t n_chunks) {
    const uint64_t start = a.first_chunk * a.chunk;
    uint64_t end = start + n_chunks * a.chunk;
    if (end > a.total) end = a.total;
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    for (uint64_t x = start + blockIdx.x * (uint64_t)kThreads + threadIdx.x; x < end; x += stride) {
        const uint64_t rel = x - start;
        const uint64_t c = rel / a.chunk;
        const uint8_t* src = a.table ? a.table[c] : a.single;
        a.dst[x] = src[rel - c * a.chunk];
    }
}

// A non-negative integer from the environment, or dflt when unset or malformed.
uint32_t env_u32(const char* name, uint32_t dflt) {
    const char* s = std::getenv(name);
    if (!s || !*s) return dflt;
    char* end = nullptr;
    const long v = std::strtol(s, &end, 10);
    return (end && *end == '\0' && v >= 0) ? (uint32_t)v : dflt;
}

}  // namespace

GatherShape gather_shape() {
    // read at every launch (a few getenv calls) so one process can compare shapes
    GatherShape s;
    s.blocks = env_u32("SLLM_K1_BLOCKS", 512);
    if (s.blocks == 0) s.blocks = 1;
    s.stream_blocks = env_u32("SLLM_K1_STREAM_BLOCKS", 64);
    if (s.stream_blocks == 0) s.stream_blocks = 1;
    s.unroll = env_u32("SLLM_K1_UNROLL", 4);
    if (s.unroll != 1 && s.unroll != 2 && s.unroll != 4) s.unroll = 4;
    s.nontemporal = env_u32("SLLM_K1_NT", 0) != 0;
    return s;
}

namespace {

int32_t launch_tiles(GatherArgs a, uint64_t tpc, uint64_t n_chunks, const GatherShape& sh, uint32_t blocks,
                     hipStream_t stream) {
    a.tiles_per_chunk = (uint32_t)tpc;
    a.n_tiles = (uint32_t)(n_chunks * tpc);
    const uint32_t grid = a.n_tiles < blocks ? a.n_tiles : blocks;
    const dim3 gd(grid), bd(kThreads);
    switch (sh.unroll * 2 + (sh.nontemporal ? 1 : 0)) {
        case 2: k1_gather<1, false><<<gd, bd, 0, stream>>>(a); break;
        case 3: k1_gather<1, true><<<gd, bd, 0, stream>>>(a); break;
        case 4: k1_gather<2, false><<<gd, bd, 0, stream>>>(a); break;
        case 5: k1_gather<2, true><<<gd, bd, 0, stream>>>(a); break;
        case 8: k1_gather<4, false><<<gd, bd, 0, stream>>>(a); break;
        default: k1_gather<4, true><<<gd, bd, 0, stream>>>(a); break;
    }
    SLLM_HIP(hipGetLastError());
    return SLLM_OK;
}

}  // namespace

int32_t launch_gather_batch(uint8_t* dst, const uint8_t* const* srcs, const uint64_t* chunks, uint32_t n,
                            uint64_t chunk, uint64_t total, hipStream_t stream) {
    if (n == 0) return SLLM_OK;
    if (n > kGatherBatch || chunk == 0) return fail(SLLM_E_INVAL, "gather batch: bad size");
    const uint64_t n_all = ceil_div(total, chunk);
    for (uint32_t i = 0; i < n; ++i)
        if (chunks[i] >= n_all) return fail(SLLM_E_INVAL, "gather batch: chunk past the end of the image");
    const bool vec = (chunk % kVec) == 0 && (reinterpret_cast<uintptr_t>(dst) % kVec) == 0;
    if (!vec) {  // byte geometry: one launch per chunk
        for (uint32_t i = 0; i < n; ++i) {
            GatherLaunch g;
            g.dst = dst;
            g.single = srcs[i];
            g.chunk = chunk;
            g.total = total;
            g.first_chunk = chunks[i];
            g.n_chunks = 1;
            SLLM_TRY(launch_gather(g, stream));
        }
        return SLLM_OK;
    }
    const GatherShape sh = gather_shape();
    GatherArgs a{};
    a.dst = dst;
    a.chunk = chunk;
    a.total = total;
    a.batch_n = n;
    for (uint32_t i = 0; i < n; ++i) {
        a.batch_src[i] = srcs[i];
        a.batch_chunk[i] = chunks[i];
    }
    const uint64_t tpc = ceil_div(chunk, (uint64_t)kThreads * kVec * sh.unroll);
    if (tpc * n >= (1ull << 31)) return fail(SLLM_E_INVAL, "gather batch: chunk size too large");
    return launch_tiles(a, tpc, n, sh, sh.stream_blocks, stream);
}

int32_t launch_gather(const GatherLaunch& g, hipStream_t stream) {
    if (g.n_chunks == 0 || g.first_chunk * g.chunk >= g.total) return SLLM_OK;
    if (!g.table && g.n_chunks != 1) return fail(SLLM_E_INVAL, "gather: a single slot serves one chunk");
    if (g.chunk == 0 || g.n_chunks > ceil_div(g.total, g.chunk) - g.first_chunk)
        return fail(SLLM_E_INVAL, "gather: chunks past the end of the image");
    const GatherShape sh = gather_shape();
    GatherArgs a{};
    a.dst = g.dst;
    a.table = g.table;
    a.single = g.single;
    a.chunk = g.chunk;
    a.total = g.total;
    a.first_chunk = g.first_chunk;
    const bool vec = (g.chunk % kVec) == 0 && (reinterpret_cast<uintptr_t>(g.dst) % kVec) == 0;
    if (!vec) {
        uint64_t bytes = g.n_chunks * g.chunk;
        uint64_t blocks = ceil_div(bytes, kThreads);
        if (blocks > 4096) blocks = 4096;
        k1_gather_bytes<<<dim3((uint32_t)blocks), dim3(kThreads), 0, stream>>>(a, g.n_chunks);
        SLLM_HIP(hipGetLastError());
        return SLLM_OK;
    }
    const uint64_t tile = (uint64_t)kThreads * kVec * sh.unroll;
    const uint64_t tpc = ceil_div(g.chunk, tile);
    const bool whole = g.first_chunk == 0 && g.n_chunks == ceil_div(g.total, g.chunk);
    const uint32_t blocks = whole ? sh.blocks : sh.stream_blocks;
    // launch at most 2^31 tiles at a time
    const uint64_t max_chunks = tpc > (1ull << 31) ? 0 : (1ull << 31) / tpc;
    if (max_chunks == 0) return fail(SLLM_E_INVAL, "gather: chunk size %llu too large", (unsigned long long)g.chunk);
    for (uint64_t c0 = 0; c0 < g.n_chunks; c0 += max_chunks) {
        const uint64_t nc = g.n_chunks - c0 < max_chunks ? g.n_chunks - c0 : max_chunks;
        a.table = g.table ? g.table + c0 : nullptr;
        a.first_chunk = g.first_chunk + c0;
        SLLM_TRY(launch_tiles(a, tpc, nc, sh, blocks, stream));
    }
    return SLLM_OK;
}

}  // namespace sllm
