// Device layouts with their own alignment A2: tensor i of the partition goes
// to d_i = sum_{j<i} align_up(s_j, A2) of the device buffer, zero padded (the
// closed form of Sec. 4.1's aligned packing, applied with A2).
//
// The device keeps the index as three u64 tables (file offsets o, sizes s and
// device offsets d, the last computed on the GPU by a wave64 prefix sum) and
// a scatter kernel moves a window [x0, x1) of partition bytes to the device
// bytes that window owns: the data bytes whose source lies in the window plus
// the padding after every tensor whose last byte lies in it.  Windows that
// tile [0, T) therefore write every byte of [0, T2) exactly once.
#pragma once

#include <hip/hip_runtime_api.h>

#include <climits>
#include <cstdint>
#include <vector>

#include "format.hpp"

namespace sllm {

struct DeviceLayout {
    uint64_t n = 0;                 // tensors
    uint64_t total = 0;             // T: bytes of the partition image
    uint64_t dev_total = 0;         // T2: bytes of the device image
    uint64_t dev_align = 0;         // A2
    uint64_t* d_off = nullptr;      // device: o_i
    uint64_t* d_size = nullptr;     // device: s_i
    uint64_t* d_dev = nullptr;      // device: d_i for i < n, d_n = T2
    std::vector<uint64_t> h_off, h_dev, h_end;  // host: o_i, d_i, o_i + s_i
    int64_t* d_shift = nullptr;     // device: K2's plan, one entry per kPlanBytes of the device image
    uint64_t n_shift = 0;           // entries of d_shift: ceil(T2 / kPlanBytes)
    uint8_t* staging = nullptr;     // HBM staging chunks for copy-engine loads
    uint64_t staging_stride = 0;
};

// K2 from HBM moves the device image in tiles of kTileBytes (kK2Lanes lanes x
// kK2Vecs 16-byte vectors), one per workgroup.  Its plan holds, for each
// block of kPlanBytes, the shift o_m - d_m from a destination byte to its
// partition byte when the block lies inside the data bytes of one tensor m,
// or kMixedTile when it meets a boundary or padding.
constexpr uint32_t kK2Lanes = 512;
constexpr uint32_t kK2Vecs = 1;
constexpr uint64_t kTileBytes = (uint64_t)kK2Lanes * 16 * kK2Vecs;
constexpr uint64_t kPlanBytes = 16384;
static_assert(kPlanBytes % kTileBytes == 0, "a tile lies in one plan block");
constexpr int64_t kMixedTile = INT64_MIN;

// Upload the tables, compute d on the device and check it against the host
// plan `dev_off`/`dev_total`; allocate `staging_chunks` HBM chunks of `chunk`
// bytes when asked.
int32_t device_layout_build(const std::vector<uint64_t>& file_off, const std::vector<uint64_t>& sizes,
                            const std::vector<uint64_t>& dev_off, uint64_t total, uint64_t dev_total,
                            uint64_t dev_align, uint64_t staging_chunks, uint64_t chunk, DeviceLayout* out);
void device_layout_free(DeviceLayout* l);

// Move partition window [x0, x1), held contiguously at `src` (device memory,
// or a device-visible mapping of pinned host memory), into the device image.
int32_t launch_scatter_window(const DeviceLayout& l, uint8_t* dst, const uint8_t* src, uint64_t x0, uint64_t x1,
                              bool src_is_host, hipStream_t stream);

// Move the whole partition, held in pinned chunks listed by `table` (device
// array; chunk k holds partition bytes [kC, kC + C)), into the device image.
int32_t launch_scatter_table(const DeviceLayout& l, uint8_t* dst, const uint8_t* const* table, uint64_t chunk,
                             hipStream_t stream);

// Up to this many chunks, each from its own slot, in one scatter launch.
constexpr uint32_t kScatterBatch = 64;

// Move the run of m (<= kScatterBatch) consecutive chunks k0 .. k0 + m - 1,
// chunk k0 + j held at the device-visible host address srcs[j], into the
// device image (the window [k0 C, min((k0 + m) C, T))).
int32_t launch_scatter_run(const DeviceLayout& l, uint8_t* dst, const uint8_t* const* srcs, uint64_t k0, uint32_t m,
                           uint64_t chunk, hipStream_t stream);

// The allocation-free repack works in a fixed device area of
// kNoAllocScratchBytes per device: the sizes s_i, the file offsets o_i and the
// device offsets d_i (n + 1 entries each for the two scans) of at most
// kNoAllocMaxTensors tensors, then K2's plan for one window of the device
// image (kNoAllocPlanEntries blocks of kPlanBytes, 28 GiB).
constexpr uint64_t kNoAllocScratchBytes = SLLM_NOALLOC_SCRATCH_BYTES;
constexpr uint64_t kNoAllocMaxTensors = SLLM_NOALLOC_MAX_TENSORS;
constexpr uint64_t kNoAllocSizeOffset = 0;
constexpr uint64_t kNoAllocFileOffset = kNoAllocSizeOffset + 8 * kNoAllocMaxTensors;
constexpr uint64_t kNoAllocDevOffset = kNoAllocFileOffset + 8 * (kNoAllocMaxTensors + 1);
constexpr uint64_t kNoAllocPlanOffset = 2ull << 20;
constexpr uint64_t kNoAllocPlanEntries = (kNoAllocScratchBytes - kNoAllocPlanOffset) / sizeof(int64_t);
static_assert(kNoAllocDevOffset + 8 * (kNoAllocMaxTensors + 1) <= kNoAllocPlanOffset, "tables fit before the plan");

// Repack the file-layout image at src (T = ix.total bytes) into dst (T2 =
// dev_total bytes at alignment dev_align) with every device table in the
// scratch area: no allocation.  Calls that overlap on one device race for
// that area.  The current device must be `device`.
int32_t repack_noalloc(const IndexData& ix, int device, uint64_t dev_align, uint64_t dev_total, const uint8_t* src,
                       uint8_t* dst, hipStream_t stream);

}  // namespace sllm
