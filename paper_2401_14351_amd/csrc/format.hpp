// The loading-optimized checkpoint format (Sec. 4.1): layout planning, the
// tensor index codec and its validation.  Host-only (no HIP).
#pragma once

#include <cstdint>
#include <string>
#include <string_view>
#include <unordered_map>
#include <vector>

#include "common.hpp"

namespace sllm {

constexpr char kMagic[8] = {'S', 'L', 'L', 'M', 'I', 'D', 'X', '1'};
constexpr uint32_t kVersion = 1;
constexpr uint64_t kFileBlock = 4096;        // the data file is padded to whole blocks
constexpr uint64_t kHeaderBytes = 56;        // fixed header before the records
constexpr uint64_t kMaxName = 65535;
constexpr const char* kIndexName = "sllm.index";
constexpr const char* kDataName = "sllm.part0";

uint32_t itemsize(uint32_t dtype);  // 0 for an unknown dtype

struct TensorRec {
    uint64_t name_off = 0;  // the name's first byte in IndexData::names
    uint32_t name_len = 0;  // bytes, without the NUL that follows it there
    uint32_t dtype = 0;
    uint32_t ndim = 0;
    int64_t shape[SLLM_MAX_NDIM] = {};
    uint64_t offset = 0;   // o_i in the partition file
    uint64_t nbytes = 0;   // s_i, unpadded
};

struct IndexData {
    uint64_t alignment = 0;   // A
    uint64_t chunk_size = 0;  // default C
    uint64_t total = 0;       // T = sum align_up(s_i, A)
    uint64_t file_bytes = 0;  // F = align_up(T, 4096)
    std::vector<TensorRec> tensors;
    // every tensor's name followed by a NUL, in record order: one buffer for
    // all names instead of an allocation per name
    std::string names;

    const char* name(size_t i) const { return names.data() + tensors[i].name_off; }
    std::string_view name_view(size_t i) const { return {names.data() + tensors[i].name_off, tensors[i].name_len}; }
    // record t's name (len bytes at s)
    void set_name(TensorRec& t, const char* s, size_t len) {
        t.name_off = names.size();
        t.name_len = (uint32_t)len;
        names.append(s, len);
        names.push_back('\0');
    }
};

// CRC-32, IEEE 802.3 polynomial (reflected 0xEDB88320), as used by zlib/PNG.
uint32_t crc32(const void* data, size_t n, uint32_t crc = 0);

// Check one source tensor's metadata (name, dtype, ndim, shape, nbytes) and
// return its numel-based byte size in *nbytes_out.
int32_t check_tensor_meta(const char* name, uint32_t dtype, uint32_t ndim, const int64_t* shape,
                          uint64_t nbytes);

// Offsets of tensors packed in order at `align`-aligned offsets:
// out[i] = sum_{j<i} align_up(s_j, align); *total = sum align_up(s_i, align).
int32_t plan_layout(const uint64_t* sizes, size_t n, uint64_t align, uint64_t* out, uint64_t* total);

// Serialize / parse sllm.index.  decode_index validates everything the format
// fixes (magic, version, CRC, names, dtypes, sizes, offsets, totals).
std::string encode_index(const IndexData& ix);
int32_t decode_index(const void* data, size_t n, IndexData* out);

}  // namespace sllm
