// gfx950 kernels for device layouts with alignment A2.
//
// K3  offsets scan: d = exclusive prefix sum of align_up(s_i, A2) over the
//     tensor index, one workgroup of 16 wave64s: a shuffle scan inside each
//     wave, the 16 wave totals combined through LDS, a running carry across
//     blocks of 1024 tensors.
// K2  index-driven scatter from HBM (the repack of a file-layout image, and
//     copy-engine loads staged in HBM): destination-driven, one 8 KiB tile of
//     the device image per workgroup of 512 lanes, tiles in dispatch order.
//     A plan built with the layout gives, per 16 KiB block of the device
//     image, the shift from a destination byte to its partition byte when the
//     block lies inside one tensor's data; such tiles copy with one 16-byte
//     vector per lane after a single table load.  The other tiles take the
//     general path below.
// K1-scatter (mapped pinned host source) and K2's general path: each
//     workgroup walks a span of tiles, finds the tensors whose slots meet a
//     tile (a forward search of d), stages those index entries in LDS and
//     keeps them for the following tiles they still cover; every lane
//     produces aligned 16-byte destination vectors: a straight 16-byte load
//     when source and destination agree mod 16, two aligned loads and a byte
//     funnel shift when they do not, zeros for padding.  Only vectors cut by
//     the window's first or last destination byte are written byte by byte.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <mutex>

#include "common.hpp"
#include "device_layout.hpp"
#include "hip_util.hpp"

namespace sllm {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kThreads = 256;
constexpr uint32_t kLdsEntries = 256;                          // index entries staged per tile

// ---------------------------------------------------------------------------
// K3
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint64_t shfl_up64(uint64_t x, uint32_t d) {
    const int lo = __shfl_up((int)(uint32_t)x, d, 64);
    const int hi = __shfl_up((int)(uint32_t)(x >> 32), d, 64);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// inclusive scan across the 64 lanes of a wave
__device__ __forceinline__ uint64_t wave_scan(uint64_t x, uint32_t lane) {
#pragma unroll
    for (uint32_t d = 1; d < 64; d <<= 1) {
        const uint64_t y = shfl_up64(x, d);
        if (lane >= d) x += y;
    }
    return x;
}

__global__ __launch_bounds__(1024) void k3_offsets_scan(const uint64_t* __restrict__ size, uint64_t n,
                                                        uint64_t align, uint64_t* __restrict__ dev) {
    __shared__ uint64_t wave_tot[16];
    const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t carry = 0;
    for (uint64_t base = 0; base < n; base += 1024) {
        const uint64_t i = base + threadIdx.x;
        const uint64_t v = i < n ? (size[i] + align - 1) & ~(align - 1) : 0;
        const uint64_t incl = wave_scan(v, lane);
        if (lane == 63) wave_tot[wave] = incl;
        __syncthreads();
        if (wave == 0) {
            uint64_t w = lane < 16 ? wave_tot[lane] : 0;
            w = wave_scan(w, lane);
            if (lane < 16) wave_tot[lane] = w;
        }
        __syncthreads();
        const uint64_t before = carry + (wave ? wave_tot[wave - 1] : 0);
        if (i < n) dev[i] = before + incl - v;
        carry += wave_tot[15];
        __syncthreads();  // wave_tot is rewritten by the next block
    }
    if (threadIdx.x == 0) dev[n] = carry;
}

// ---------------------------------------------------------------------------
// K2 / K1-scatter
// ---------------------------------------------------------------------------

struct ScatterArgs {
    uint8_t* dst;
    const uint64_t* off;   // o_i
    const uint64_t* size;  // s_i
    const uint64_t* dev;   // d_i, d_n = T2
    uint64_t n;
    uint64_t y0, y1;       // destination bytes written by this launch
    uint64_t tile0, n_tiles;
    // source: a contiguous window ...
    const uint8_t* base;   // partition byte x at base[x - x0]
    uint64_t x0, x1;
    // ... or a table of chunks
    const uint8_t* const* table;  // partition byte x at table[x / chunk][x % chunk]
    uint64_t chunk;
    // ... or a run of chunks passed inline (run_n > 0): byte x of chunk
    // k = x / chunk at run_src[k - run_k0][x % chunk], for x in [x0, x1)
    uint32_t run_n;
    uint64_t run_k0;
    const uint8_t* run_src[kScatterBatch];
    uint64_t total;        // T
    uint32_t vec_ok;       // 16-byte aligned source vectors are addressable as such
    uint64_t plan0;        // K2: plan entry of destination block p is shift[p - plan0]
};

// Where a launch's source bytes are: one contiguous window, a device table
// of chunks, or a run of chunks passed inline.  A kernel instance serves one
// kind, so none of them pays for the others' addressing.
enum SrcKind : int { kWindow = 0, kTable = 1, kRun = 2 };

template <SrcKind K>
struct Src {
    const ScatterArgs& a;
    __device__ __forceinline__ const uint8_t* at(uint64_t x) const {
        if constexpr (K == kRun) {
            const uint64_t k = x / a.chunk;
            return a.run_src[k - a.run_k0] + (x - k * a.chunk);
        } else if constexpr (K == kTable) {
            const uint64_t k = x / a.chunk;
            return a.table[k] + (x - k * a.chunk);
        } else {
            return a.base + (x - a.x0);
        }
    }
    // can the 16-byte aligned vectors covering [x, x + len) be loaded whole?
    __device__ __forceinline__ bool vectors_ok(uint64_t xa, uint64_t len) const {
        if (!a.vec_ok) return false;
        if constexpr (K == kTable) return xa + len <= a.total;
        return xa >= a.x0 && xa + len <= a.x1;
    }
};

__device__ __forceinline__ u32x4 ld16(const uint8_t* p) { return *reinterpret_cast<const u32x4*>(p); }

// bytes [s, s + 16) of the 32 bytes lo:hi, for s in [0, 16)
__device__ __forceinline__ u32x4 funnel(u32x4 lo, u32x4 hi, uint32_t s) {
    const uint32_t w[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    const uint32_t b = s & 3;
    u32x4 r;
    switch (s >> 2) {
        case 0: r = u32x4{__builtin_amdgcn_alignbyte(w[1], w[0], b), __builtin_amdgcn_alignbyte(w[2], w[1], b),
                          __builtin_amdgcn_alignbyte(w[3], w[2], b), __builtin_amdgcn_alignbyte(w[4], w[3], b)}; break;
        case 1: r = u32x4{__builtin_amdgcn_alignbyte(w[2], w[1], b), __builtin_amdgcn_alignbyte(w[3], w[2], b),
                          __builtin_amdgcn_alignbyte(w[4], w[3], b), __builtin_amdgcn_alignbyte(w[5], w[4], b)}; break;
        case 2: r = u32x4{__builtin_amdgcn_alignbyte(w[3], w[2], b), __builtin_amdgcn_alignbyte(w[4], w[3], b),
                          __builtin_amdgcn_alignbyte(w[5], w[4], b), __builtin_amdgcn_alignbyte(w[6], w[5], b)}; break;
        default: r = u32x4{__builtin_amdgcn_alignbyte(w[4], w[3], b), __builtin_amdgcn_alignbyte(w[5], w[4], b),
                           __builtin_amdgcn_alignbyte(w[6], w[5], b), __builtin_amdgcn_alignbyte(w[7], w[6], b)}; break;
    }
    return r;
}

// keep bytes [0, keep) of v, zero the rest
__device__ __forceinline__ u32x4 keep_bytes(u32x4 v, uint32_t keep) {
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (uint32_t j = 0; j < 4; ++j) {
        const uint32_t lo = 4 * j;
        if (keep <= lo) w[j] = 0;
        else if (keep < lo + 4) w[j] &= (1u << (8 * (keep - lo))) - 1u;
    }
    return u32x4{w[0], w[1], w[2], w[3]};
}

__device__ __forceinline__ uint32_t byte_of(u32x4 v, uint32_t b) {
    const uint32_t w = b < 4 ? v.x : b < 8 ? v.y : b < 12 ? v.z : v.w;
    return (w >> (8 * (b & 3))) & 0xFF;
}

// largest m in [lo, hi] with d[m] <= y (d[lo] <= y holds)
__device__ __forceinline__ uint64_t owner_global(const uint64_t* d, uint64_t lo, uint64_t hi, uint64_t y) {
    while (lo < hi) {
        const uint64_t mid = lo + (hi - lo + 1) / 2;
        if (d[mid] <= y) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// the same, searching forward from `from` (d[from] <= y): gallop 1, 2, 4 ...
// entries ahead, then bisect the last step; one load when y is still in the
// slot of tensor `from`, as it is for most tiles of a large tensor
__device__ __forceinline__ uint64_t owner_from(const uint64_t* d, uint64_t from, uint64_t last, uint64_t y) {
    uint64_t lo = from, step = 1;
    while (lo < last) {
        const uint64_t probe = last - lo < step ? last : lo + step;
        if (d[probe] > y) return owner_global(d, lo, probe - 1, y);
        lo = probe;
        step <<= 1;
    }
    return lo;
}

template <bool NT>
__device__ __forceinline__ void st16(uint8_t* p, u32x4 v) {
    if constexpr (NT) {
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
    } else {
        *reinterpret_cast<u32x4*>(p) = v;
    }
}

// Index entries of the tensors meeting a tile, staged in LDS.
struct Staging {
    uint64_t dev[kLdsEntries], off[kLdsEntries], size[kLdsEntries];
    uint64_t lo, hi, next;
};

// Tiles [t_begin, t_end) of the launch, in order (tile t covers destination
// bytes [(tile0 + t) S, (tile0 + t + 1) S), S = L lanes x 16 B x U).  For
// each tile every lane first produces its U destination vectors (all source
// loads in flight together), then stores them.  The index entries of the
// tensors meeting a tile are staged in LDS together with the start of the
// next tensor's slot; while the following tiles end before that start (the
// interior of a large tensor) they reuse the staged entries, with no search,
// no staging and no barrier.  Every lane of the workgroup must call this
// with the same span (it holds barriers).
template <uint32_t L, uint32_t U, bool NT, SrcKind K>
__device__ __forceinline__ void scatter_span(const ScatterArgs& a, Staging& stg, uint64_t t_begin, uint64_t t_end) {
    constexpr uint64_t kTileU = (uint64_t)L * 16 * U;
    uint64_t* const s_dev = stg.dev;
    uint64_t* const s_off = stg.off;
    uint64_t* const s_size = stg.size;
    const Src<K> src{a};
    uint64_t cursor = 0;   // thread 0: owner of the last searched tile's last byte
    bool staged = false;   // LDS holds entries i_lo .. i_lo + cnt - 1 (uniform)
    uint64_t i_lo = 0, cnt = 0, next = 0;  // next: d of the first tensor not staged
    for (uint64_t t = t_begin; t < t_end; ++t) {
        const uint64_t yt = (a.tile0 + t) * kTileU;
        const uint64_t lo = yt > a.y0 ? yt : a.y0;
        const uint64_t hi = yt + kTileU < a.y1 ? yt + kTileU : a.y1;
        if (!staged || hi > next) {
            __syncthreads();  // every wave is done with the entries staged before
            if (threadIdx.x == 0) {
                const uint64_t first =
                    t == t_begin ? owner_global(a.dev, 0, a.n - 1, lo) : owner_from(a.dev, cursor, a.n - 1, lo);
                cursor = owner_from(a.dev, first, a.n - 1, hi - 1);
                stg.lo = first;
                stg.hi = cursor;
            }
            __syncthreads();
            i_lo = stg.lo;
            cnt = stg.hi - stg.lo + 1;
            staged = cnt <= kLdsEntries;
            if (staged)
                for (uint32_t i = threadIdx.x; i < cnt; i += L) {
                    s_dev[i] = a.dev[i_lo + i];
                    s_off[i] = a.off[i_lo + i];
                    s_size[i] = a.size[i_lo + i];
                }
            if (threadIdx.x == 0) stg.next = a.dev[i_lo + cnt];  // d[n] = T2 ends the last slot
            __syncthreads();
            next = stg.next;
        }
        u32x4 v[U];
        uint32_t whole_mask = 0, in_mask = 0;
#pragma unroll
        for (uint32_t u = 0; u < U; ++u) {
            v[u] = u32x4{0, 0, 0, 0};
            const uint64_t y = yt + ((uint64_t)u * L + threadIdx.x) * 16;
            if (y + 16 <= lo || y >= hi) continue;
            in_mask |= 1u << u;
            uint64_t dm, om, sm;
            if (cnt == 1) {
                dm = s_dev[0]; om = s_off[0]; sm = s_size[0];
            } else if (staged) {
                uint32_t l = 0, h = (uint32_t)cnt - 1;
                while (l < h) {
                    const uint32_t mid = (l + h + 1) >> 1;
                    if (s_dev[mid] <= y) l = mid;
                    else h = mid - 1;
                }
                dm = s_dev[l]; om = s_off[l]; sm = s_size[l];
            } else {
                const uint64_t m = owner_global(a.dev, i_lo, i_lo + cnt - 1, y);
                dm = a.dev[m]; om = a.off[m]; sm = a.size[m];
            }
            const uint64_t r = y - dm;                   // byte of the slot
            const uint32_t dn = sm > r ? (sm - r < 16 ? (uint32_t)(sm - r) : 16u) : 0u;  // data bytes in vector
            const uint64_t x = om + r;                   // source of the vector's first byte
            const bool whole = y >= lo && y + 16 <= hi;  // vector entirely ours to write
            if (whole) whole_mask |= 1u << u;
            if (!dn) continue;
            const uint64_t xa = x & ~15ull;
            const uint32_t sh = (uint32_t)(x & 15);
            const uint64_t need = sh + dn > 16 ? 32 : 16;  // aligned source bytes spanned
            if (whole && src.vectors_ok(xa, need)) {
                const u32x4 v0 = ld16(src.at(xa));
                u32x4 w = sh == 0 ? v0 : funnel(v0, need == 32 ? ld16(src.at(xa + 16)) : v0, sh);
                v[u] = dn < 16 ? keep_bytes(w, dn) : w;
            } else {
                uint32_t w[4] = {0, 0, 0, 0};
                for (uint32_t b = 0; b < dn; ++b) {
                    if (y + b < lo || y + b >= hi) continue;
                    w[b >> 2] |= (uint32_t)*src.at(x + b) << (8 * (b & 3));
                }
                v[u] = u32x4{w[0], w[1], w[2], w[3]};
            }
        }
#pragma unroll
        for (uint32_t u = 0; u < U; ++u) {
            if (!(in_mask >> u & 1)) continue;
            const uint64_t y = yt + ((uint64_t)u * L + threadIdx.x) * 16;
            if (whole_mask >> u & 1) {
                st16<NT>(a.dst + y, v[u]);
            } else {
                for (uint32_t b = 0; b < 16; ++b)
                    if (y + b >= lo && y + b < hi) a.dst[y + b] = (uint8_t)byte_of(v[u], b);
            }
        }
    }
}

// K1-scatter (host sources): each workgroup of a persistent grid walks a
// contiguous span of tiles, so the owner of the next tile is found by
// searching forward from the last one.
template <uint32_t U, bool NT, SrcKind K>
__global__ __launch_bounds__(kThreads) void k_scatter(ScatterArgs a) {
    __shared__ Staging stg;
    const uint64_t per_block = (a.n_tiles + gridDim.x - 1) / gridDim.x;
    const uint64_t t_begin = (uint64_t)blockIdx.x * per_block;
    const uint64_t t_end = t_begin + per_block < a.n_tiles ? t_begin + per_block : a.n_tiles;
    scatter_span<kThreads, U, NT, K>(a, stg, t_begin, t_end);
}

// K2 from HBM: one kTileBytes destination tile per workgroup of kK2Lanes
// lanes, tiles in dispatch order, so the workgroups in flight sweep a
// contiguous window of both images (HBM serves that order best).  A tile
// whose plan block lies inside one tensor's data, and whose source bytes all
// lie in the window, copies straight from source byte y + shift: one table
// load, then the data loads.  Every other tile (tensor boundaries, padding,
// window edges) takes the general path of scatter_span.
template <bool NT>
__global__ __launch_bounds__(kK2Lanes) void k2_tiles(ScatterArgs a, const int64_t* __restrict__ shift) {
    constexpr uint32_t U = kK2Vecs;
    __shared__ Staging stg;
    const uint64_t t = a.tile0 + blockIdx.x;
    const uint64_t yt = t * kTileBytes;
    const int64_t sh = shift[yt / kPlanBytes - a.plan0];
    if (sh != kMixedTile && yt >= a.y0 && yt + kTileBytes <= a.y1) {
        const uint64_t xs = yt + (uint64_t)sh;  // source of the tile's first byte
        // aligned 16-byte source vectors spanning [xs, xs + S)
        const uint64_t xa0 = xs & ~15ull, xa1 = (xs + kTileBytes + 15) & ~15ull;
        if (a.vec_ok && xa0 >= a.x0 && xa1 <= a.x1) {
            const uint32_t r = (uint32_t)(xs & 15);  // the same for every vector of the tile
            u32x4 v[U];
#pragma unroll
            for (uint32_t u = 0; u < U; ++u) {
                // partition byte x sits at base + (x - x0); base and x0 are 16-byte aligned
                const uint8_t* p = a.base + (xs - a.x0) + ((uint64_t)u * kK2Lanes + threadIdx.x) * 16 - r;
                v[u] = r == 0 ? ld16(p) : funnel(ld16(p), ld16(p + 16), r);
            }
#pragma unroll
            for (uint32_t u = 0; u < U; ++u) st16<NT>(a.dst + yt + ((uint64_t)u * kK2Lanes + threadIdx.x) * 16, v[u]);
            return;
        }
    }
    scatter_span<kK2Lanes, U, NT, kWindow>(a, stg, blockIdx.x, blockIdx.x + 1);
}

// K2's plan for destination blocks p0 .. p0 + n_blocks - 1: shift[p - p0] =
// o_m - d_m when block p (kPlanBytes) lies inside the data bytes of tensor
// m, else kMixedTile.
__global__ __launch_bounds__(256) void k3_tile_shift(const uint64_t* __restrict__ dev, const uint64_t* __restrict__ off,
                                                     const uint64_t* __restrict__ size, uint64_t n, uint64_t p0,
                                                     uint64_t n_blocks, int64_t* __restrict__ shift) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n_blocks; p += stride) {
        const uint64_t y = (p0 + p) * kPlanBytes;
        const uint64_t m = owner_global(dev, 0, n - 1, y);  // d_0 = 0 <= y
        shift[p] = y + kPlanBytes <= dev[m] + size[m] ? (int64_t)(off[m] - dev[m]) : kMixedTile;
    }
}

// A non-negative integer from the environment, or dflt when unset or malformed.
uint32_t env_uint(const char* name, uint32_t dflt) {
    const char* s = std::getenv(name);
    if (!s || !*s) return dflt;
    char* end = nullptr;
    const long v = std::strtol(s, &end, 10);
    return (end && *end == '\0' && v >= 0) ? (uint32_t)v : dflt;
}

// first device byte owned by partition byte x: the first tensor whose data
// ends after x starts owning there (padding belongs to a tensor's last byte)
uint64_t y_of(const DeviceLayout& l, uint64_t x) {
    auto it = std::upper_bound(l.h_end.begin(), l.h_end.end(), x);
    if (it == l.h_end.end()) return l.dev_total;
    const size_t i = (size_t)(it - l.h_end.begin());
    return l.h_dev[i] + (x > l.h_off[i] ? x - l.h_off[i] : 0);
}

// Launch shape, read at every launch so that one process can compare shapes:
// SLLM_K2_NT (streaming stores) and SLLM_K2_MAX_GRID (workgroups a launch)
// for HBM sources; SLLM_K2_UNROLL (4 or 8 vectors per lane) and
// SLLM_K1_BLOCKS / SLLM_K1_STREAM_BLOCKS (grid of a launch that moves the
// whole image / part of it, as for K1) for host sources.
int32_t launch(const DeviceLayout& l, ScatterArgs a, bool src_is_host, hipStream_t stream) {
    a.off = l.d_off;
    a.size = l.d_size;
    a.dev = l.d_dev;
    a.n = l.n;
    a.total = l.total;
    if (a.y0 >= a.y1 || l.n == 0) return SLLM_OK;
    if (a.y1 > l.dev_total) return fail(SLLM_E_INVAL, "scatter: destination range past the image");
    if (!src_is_host) {  // HBM source (K2): one tile per workgroup
        if (!l.d_shift) return fail(SLLM_E_INVAL, "scatter: the layout has no tile plan");
        const bool nt = env_uint("SLLM_K2_NT", 1) != 0;
        const uint64_t t_end = ceil_div(a.y1, kTileBytes);
        // at most 2^31 lanes a launch (SLLM_K2_MAX_GRID lowers it, to exercise
        // the split on small images)
        constexpr uint64_t kMaxGrid = (1ull << 31) / kK2Lanes;
        const uint64_t max_grid = std::max<uint64_t>(1, std::min<uint64_t>(kMaxGrid, env_uint("SLLM_K2_MAX_GRID", kMaxGrid)));
        for (uint64_t t0 = a.y0 / kTileBytes; t0 < t_end; t0 += max_grid) {
            a.tile0 = t0;
            a.n_tiles = std::min(max_grid, t_end - t0);
            const dim3 grid((uint32_t)a.n_tiles);
            if (nt) k2_tiles<true><<<grid, dim3(kK2Lanes), 0, stream>>>(a, l.d_shift);
            else k2_tiles<false><<<grid, dim3(kK2Lanes), 0, stream>>>(a, l.d_shift);
            SLLM_HIP(hipGetLastError());
        }
        return SLLM_OK;
    }
    // host sources are PCIe-latency bound like K1: a persistent grid of spans
    const uint32_t unroll = env_uint("SLLM_K2_UNROLL", 8) >= 8 ? 8 : 4;
    const uint64_t tile = (uint64_t)kThreads * 16 * unroll;
    a.tile0 = a.y0 / tile;
    a.n_tiles = ceil_div(a.y1, tile) - a.tile0;
    // a chunk table carries the whole image; runs and windows are parts of it
    const uint32_t want = std::max<uint32_t>(
        1, a.table ? env_uint("SLLM_K1_BLOCKS", 512) : env_uint("SLLM_K1_STREAM_BLOCKS", 64));
    const dim3 grid((uint32_t)std::min<uint64_t>(a.n_tiles, want)), block(kThreads);
    const bool u8 = unroll == 8;
    if (a.run_n) u8 ? k_scatter<8, false, kRun><<<grid, block, 0, stream>>>(a) : k_scatter<4, false, kRun><<<grid, block, 0, stream>>>(a);
    else if (a.table) u8 ? k_scatter<8, false, kTable><<<grid, block, 0, stream>>>(a) : k_scatter<4, false, kTable><<<grid, block, 0, stream>>>(a);
    else u8 ? k_scatter<8, false, kWindow><<<grid, block, 0, stream>>>(a) : k_scatter<4, false, kWindow><<<grid, block, 0, stream>>>(a);
    SLLM_HIP(hipGetLastError());
    return SLLM_OK;
}

}  // namespace

int32_t device_layout_build(const std::vector<uint64_t>& file_off, const std::vector<uint64_t>& sizes,
                            const std::vector<uint64_t>& dev_off, uint64_t total, uint64_t dev_total,
                            uint64_t dev_align, uint64_t staging_chunks, uint64_t chunk, DeviceLayout* out) {
    DeviceLayout& l = *out;
    l.n = sizes.size();
    l.total = total;
    l.dev_total = dev_total;
    l.dev_align = dev_align;
    l.h_off = file_off;
    l.h_dev = dev_off;
    l.h_end.resize(l.n);
    for (uint64_t i = 0; i < l.n; ++i) l.h_end[i] = file_off[i] + sizes[i];
    if (staging_chunks) {
        if (!align_up(chunk, 256, &l.staging_stride)) return fail(SLLM_E_INVAL, "chunk size overflows");
        SLLM_HIP(hipMalloc(reinterpret_cast<void**>(&l.staging), staging_chunks * l.staging_stride));
    }
    if (l.n == 0) return SLLM_OK;
    const size_t bytes = l.n * sizeof(uint64_t);
    SLLM_HIP(hipMalloc(reinterpret_cast<void**>(&l.d_off), bytes));
    SLLM_HIP(hipMalloc(reinterpret_cast<void**>(&l.d_size), bytes));
    SLLM_HIP(hipMalloc(reinterpret_cast<void**>(&l.d_dev), bytes + sizeof(uint64_t)));
    SLLM_HIP(hipMemcpy(l.d_off, file_off.data(), bytes, hipMemcpyHostToDevice));
    SLLM_HIP(hipMemcpy(l.d_size, sizes.data(), bytes, hipMemcpyHostToDevice));
    k3_offsets_scan<<<dim3(1), dim3(1024), 0, nullptr>>>(l.d_size, l.n, dev_align, l.d_dev);
    SLLM_HIP(hipGetLastError());
    // K2's tile plan, from the scanned offsets (same stream, so in order)
    l.n_shift = ceil_div(dev_total, kPlanBytes);
    if (l.n_shift) {
        SLLM_HIP(hipMalloc(reinterpret_cast<void**>(&l.d_shift), l.n_shift * sizeof(int64_t)));
        const uint64_t blocks = std::min<uint64_t>(ceil_div(l.n_shift, 256), 4096);
        k3_tile_shift<<<dim3((uint32_t)blocks), dim3(256), 0, nullptr>>>(l.d_dev, l.d_off, l.d_size, l.n, 0,
                                                                         l.n_shift, l.d_shift);
        SLLM_HIP(hipGetLastError());
    }
    std::vector<uint64_t> got(l.n + 1);
    SLLM_HIP(hipMemcpy(got.data(), l.d_dev, bytes + sizeof(uint64_t), hipMemcpyDeviceToHost));
    for (uint64_t i = 0; i < l.n; ++i)
        if (got[i] != dev_off[i])
            return fail(SLLM_E_HIP, "device offsets scan disagrees at tensor %llu: %llu vs %llu", (unsigned long long)i,
                        (unsigned long long)got[i], (unsigned long long)dev_off[i]);
    if (got[l.n] != dev_total) return fail(SLLM_E_HIP, "device offsets scan total disagrees");
    return SLLM_OK;
}

void device_layout_free(DeviceLayout* l) {
    for (void* p : {(void*)l->d_off, (void*)l->d_size, (void*)l->d_dev, (void*)l->d_shift, (void*)l->staging})
        if (p) (void)hipFree(p);
    *l = DeviceLayout{};
}

int32_t launch_scatter_window(const DeviceLayout& l, uint8_t* dst, const uint8_t* src, uint64_t x0, uint64_t x1,
                              bool src_is_host, hipStream_t stream) {
    ScatterArgs a{};
    a.dst = dst;
    a.base = src;
    a.x0 = x0;
    a.x1 = x1;
    a.vec_ok = (reinterpret_cast<uintptr_t>(src) % 16 == 0) && (x0 % 16 == 0);
    a.y0 = y_of(l, x0);
    a.y1 = y_of(l, x1);
    return launch(l, a, src_is_host, stream);
}

int32_t launch_scatter_run(const DeviceLayout& l, uint8_t* dst, const uint8_t* const* srcs, uint64_t k0, uint32_t m,
                           uint64_t chunk, hipStream_t stream) {
    if (m == 0) return SLLM_OK;
    if (m > kScatterBatch || chunk == 0) return fail(SLLM_E_INVAL, "scatter run: bad size");
    if (k0 >= ceil_div(l.total, chunk) || m > ceil_div(l.total, chunk) - k0)
        return fail(SLLM_E_INVAL, "scatter run: chunks past the end of the image");
    ScatterArgs a{};
    a.dst = dst;
    a.chunk = chunk;
    a.run_n = m;
    a.run_k0 = k0;
    bool aligned = chunk % 16 == 0;
    for (uint32_t j = 0; j < m; ++j) {
        a.run_src[j] = srcs[j];
        aligned = aligned && reinterpret_cast<uintptr_t>(srcs[j]) % 16 == 0;
    }
    a.vec_ok = aligned;
    a.x0 = k0 * chunk;
    a.x1 = std::min((k0 + m) * chunk, l.total);
    a.y0 = y_of(l, a.x0);
    a.y1 = y_of(l, a.x1);
    return launch(l, a, /*src_is_host=*/true, stream);
}

int32_t launch_scatter_table(const DeviceLayout& l, uint8_t* dst, const uint8_t* const* table, uint64_t chunk,
                             hipStream_t stream) {
    ScatterArgs a{};
    a.dst = dst;
    a.table = table;
    a.chunk = chunk;
    a.vec_ok = chunk % 16 == 0;
    a.y0 = 0;
    a.y1 = l.dev_total;
    return launch(l, a, /*src_is_host=*/true, stream);
}

}  // namespace sllm

// ---------------------------------------------------------------------------
// Allocation-free repack
// ---------------------------------------------------------------------------

// The device memory of the allocation-free repack: the size table, the two
// scanned offset tables and one window of K2's plan (layout in
// device_layout.hpp).  Every device holds its own copy from the library's
// first kernel launch on it until the process ends.  Host code reaches a
// device's copy only through the address hipGetSymbolAddress returns with
// that device current; the name itself is not a device address on the host.
static __device__ __align__(256) uint8_t scratch[sllm::kNoAllocScratchBytes];

namespace sllm {

namespace {

// Tensor sizes travel to the device as kernel arguments, kSizeBatch a launch.
constexpr uint32_t kSizeBatch = 256;
struct SizeBatch {
    uint64_t* dst;
    uint32_t m;
    uint64_t s[kSizeBatch];
};

__global__ __launch_bounds__(kSizeBatch) void k_put_sizes(SizeBatch b) {
    if (threadIdx.x < b.m) b.dst[threadIdx.x] = b.s[threadIdx.x];
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch[kMaxDevices] = {};

// The scratch area's address on `device`, looked up once per device (the
// caller has made `device` current).
int32_t scratch_of(int device, uint8_t** out) {
    if (device < 0 || device >= kMaxDevices) return fail(SLLM_E_INVAL, "device %d is out of range", device);
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch[device]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(SLLM_E_HIP, "hipGetSymbolAddress(scratch) on device %d failed: %s", device, hipGetErrorString(e));
        g_scratch[device] = static_cast<uint8_t*>(p);
    }
    *out = g_scratch[device];
    return SLLM_OK;
}

}  // namespace

int32_t repack_noalloc(const IndexData& ix, int device, uint64_t dev_align, uint64_t dev_total, const uint8_t* src,
                       uint8_t* dst, hipStream_t stream) {
    const uint64_t n = ix.tensors.size();
    if (n > kNoAllocMaxTensors)
        return fail(SLLM_E_RANGE, "%llu tensors exceed the %llu of the allocation-free repack", (unsigned long long)n,
                    (unsigned long long)kNoAllocMaxTensors);
    if (n == 0 || dev_total == 0) return SLLM_OK;
    uint8_t* base = nullptr;
    SLLM_TRY(scratch_of(device, &base));
    uint64_t* d_size = reinterpret_cast<uint64_t*>(base + kNoAllocSizeOffset);
    uint64_t* d_off = reinterpret_cast<uint64_t*>(base + kNoAllocFileOffset);
    uint64_t* d_dev = reinterpret_cast<uint64_t*>(base + kNoAllocDevOffset);
    int64_t* plan = reinterpret_cast<int64_t*>(base + kNoAllocPlanOffset);

    // s, then o (file layout, A) and d (device layout, A2) by the K3 scan;
    // the index was validated against the same closed form when it was read
    for (uint64_t i0 = 0; i0 < n; i0 += kSizeBatch) {
        SizeBatch b{};
        b.dst = d_size + i0;
        b.m = (uint32_t)std::min<uint64_t>(kSizeBatch, n - i0);
        for (uint32_t j = 0; j < b.m; ++j) b.s[j] = ix.tensors[i0 + j].nbytes;
        k_put_sizes<<<dim3(1), dim3(kSizeBatch), 0, stream>>>(b);
        SLLM_HIP(hipGetLastError());
    }
    k3_offsets_scan<<<dim3(1), dim3(1024), 0, stream>>>(d_size, n, ix.alignment, d_off);
    SLLM_HIP(hipGetLastError());
    k3_offsets_scan<<<dim3(1), dim3(1024), 0, stream>>>(d_size, n, dev_align, d_dev);
    SLLM_HIP(hipGetLastError());

    // windows of the device image, each planned into the plan area and then
    // moved by K2; one stream orders each window's plan after the previous
    // window's K2 (SLLM_NOALLOC_PLAN_BLOCKS lowers the window, to exercise
    // several on small images)
    DeviceLayout l;  // views of the scratch tables: owns nothing, never freed
    l.n = n;
    l.total = ix.total;
    l.dev_total = dev_total;
    l.dev_align = dev_align;
    l.d_off = d_off;
    l.d_size = d_size;
    l.d_dev = d_dev;
    l.d_shift = plan;
    const uint64_t n_blocks = ceil_div(dev_total, kPlanBytes);
    const uint64_t window = std::max<uint64_t>(
        1, std::min<uint64_t>(kNoAllocPlanEntries, env_uint("SLLM_NOALLOC_PLAN_BLOCKS", (uint32_t)kNoAllocPlanEntries)));
    for (uint64_t p0 = 0; p0 < n_blocks; p0 += window) {
        const uint64_t nb = std::min(window, n_blocks - p0);
        const uint64_t blocks = std::min<uint64_t>(ceil_div(nb, 256), 4096);
        k3_tile_shift<<<dim3((uint32_t)blocks), dim3(256), 0, stream>>>(d_dev, d_off, d_size, n, p0, nb, plan);
        SLLM_HIP(hipGetLastError());
        ScatterArgs a{};
        a.dst = dst;
        a.base = src;
        a.x0 = 0;
        a.x1 = ix.total;
        a.vec_ok = reinterpret_cast<uintptr_t>(src) % 16 == 0;
        a.y0 = p0 * kPlanBytes;
        a.y1 = std::min((p0 + nb) * kPlanBytes, dev_total);
        a.plan0 = p0;
        SLLM_TRY(launch(l, a, /*src_is_host=*/false, stream));
    }
    return SLLM_OK;
}

}  // namespace sllm
