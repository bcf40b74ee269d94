// Host-side launchers of the gfx950 kernels.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace sllm {

// Chunk gather in the file layout: for every chunk k in
// [first_chunk, first_chunk + n_chunks), copy bytes [kC, min(kC + C, T)) of
// the partition from that chunk's mapped pinned slot into dst + kC.
// Slots come from `table` (a device array of n_chunks device-visible host
// addresses, indexed from first_chunk) or, when table is null, `single`
// (n_chunks must then be 1).
struct GatherLaunch {
    uint8_t* dst = nullptr;                  // device base of the whole image
    const uint8_t* const* table = nullptr;   // device memory
    const uint8_t* single = nullptr;         // device-visible host address
    uint64_t chunk = 0;                      // C
    uint64_t total = 0;                      // T
    uint64_t first_chunk = 0;
    uint64_t n_chunks = 0;
};
int32_t launch_gather(const GatherLaunch& g, hipStream_t stream);

// Up to this many chunks, each from its own slot, in one gather launch.
constexpr uint32_t kGatherBatch = 64;

// Gather n (<= kGatherBatch) chunks: chunk chunks[i] of the partition from
// the device-visible slot srcs[i] into dst + chunks[i] * C.
int32_t launch_gather_batch(uint8_t* dst, const uint8_t* const* srcs, const uint64_t* chunks, uint32_t n,
                            uint64_t chunk, uint64_t total, hipStream_t stream);

// Kernel launch shape knobs, read from the environment at every launch:
// SLLM_K1_BLOCKS, SLLM_K1_STREAM_BLOCKS, SLLM_K1_UNROLL, SLLM_K1_NT.
struct GatherShape {
    uint32_t blocks;         // persistent grid of a launch that moves the whole image
    uint32_t stream_blocks;  // persistent grid of a launch that moves part of it
                             // (a streamed batch, run or chunk): such launches
                             // overlap on the copy streams, and a small grid
                             // each keeps the reads in flight near what the
                             // link needs
    uint32_t unroll;         // 16-byte vectors per lane per tile: 1, 2 or 4
    bool nontemporal;        // streaming (non-temporal) loads and stores
};
GatherShape gather_shape();

}  // namespace sllm
