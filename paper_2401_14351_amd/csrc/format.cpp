#include "format.hpp"

#include <cstring>

namespace sllm {

uint32_t itemsize(uint32_t dtype) {
    switch (dtype) {
        case SLLM_DTYPE_F32: return 4;
        case SLLM_DTYPE_F16: return 2;
        case SLLM_DTYPE_BF16: return 2;
        case SLLM_DTYPE_I8: return 1;
        default: return 0;
    }
}

namespace {

struct CrcTable {
    uint32_t t[8][256];
    CrcTable() {
        for (uint32_t i = 0; i < 256; ++i) {
            uint32_t c = i;
            for (int k = 0; k < 8; ++k) c = (c & 1) ? 0xEDB88320u ^ (c >> 1) : c >> 1;
            t[0][i] = c;
        }
        // slicing-by-8 tables: t[k][i] is the CRC of byte i followed by k zero bytes
        for (uint32_t i = 0; i < 256; ++i)
            for (int k = 1; k < 8; ++k) t[k][i] = (t[k - 1][i] >> 8) ^ t[0][t[k - 1][i] & 0xFF];
    }
};
const CrcTable kCrc;

inline void put_u16(std::string& s, uint16_t v) { s.append(reinterpret_cast<const char*>(&v), 2); }
inline void put_u32(std::string& s, uint32_t v) { s.append(reinterpret_cast<const char*>(&v), 4); }
inline void put_u64(std::string& s, uint64_t v) { s.append(reinterpret_cast<const char*>(&v), 8); }

// Bounds-checked little-endian reader over the index bytes.
struct Cursor {
    const uint8_t* p;
    size_t n, pos = 0;
    bool take(void* dst, size_t k) {
        if (k > n - pos) return false;
        std::memcpy(dst, p + pos, k);
        pos += k;
        return true;
    }
};

// 64-bit hash of a name, eight bytes at a time (multiply-xorshift mixing).
inline uint64_t name_hash(const std::string& s) {
    const unsigned char* p = reinterpret_cast<const unsigned char*>(s.data());
    size_t n = s.size();
    uint64_t h = 0x9E3779B97F4A7C15ull ^ n;
    auto mix = [&h](uint64_t w) {
        h ^= w * 0xBF58476D1CE4E5B9ull;
        h = (h ^ (h >> 31)) * 0x94D049BB133111EBull;
    };
    for (; n >= 8; p += 8, n -= 8) {
        uint64_t w;
        std::memcpy(&w, p, 8);
        mix(w);
    }
    uint64_t tail = 0;
    std::memcpy(&tail, p, n);
    mix(tail);
    return h ^ (h >> 29);
}

// The duplicate-name check of decode_index without an allocation per name:
// open addressing over record positions, probing by a 64-bit hash of the
// name and comparing names only when hashes match.
class NameSet {
  public:
    explicit NameSet(const std::vector<TensorRec>& recs) : recs_(recs) {
        size_t cap = 16;
        while (cap < 2 * recs.size()) cap <<= 1;
        slot_.assign(cap, kEmpty);
        hash_.resize(recs.size());
    }
    // false if record i's name is already in the set
    bool insert(uint32_t i) {
        const std::string& name = recs_[i].name;
        const uint64_t h = name_hash(name);
        hash_[i] = h;
        for (size_t k = h & (slot_.size() - 1);; k = (k + 1) & (slot_.size() - 1)) {
            const uint32_t j = slot_[k];
            if (j == kEmpty) {
                slot_[k] = i;
                return true;
            }
            if (hash_[j] == h && recs_[j].name == name) return false;
        }
    }

  private:
    static constexpr uint32_t kEmpty = UINT32_MAX;
    const std::vector<TensorRec>& recs_;
    std::vector<uint32_t> slot_;
    std::vector<uint64_t> hash_;
};

}  // namespace

uint32_t crc32(const void* data, size_t n, uint32_t crc) {
    const uint8_t* p = static_cast<const uint8_t*>(data);
    uint32_t c = ~crc;
    while (n >= 8) {
        uint32_t lo, hi;
        std::memcpy(&lo, p, 4);
        std::memcpy(&hi, p + 4, 4);
        lo ^= c;
        c = kCrc.t[7][lo & 0xFF] ^ kCrc.t[6][(lo >> 8) & 0xFF] ^ kCrc.t[5][(lo >> 16) & 0xFF] ^
            kCrc.t[4][lo >> 24] ^ kCrc.t[3][hi & 0xFF] ^ kCrc.t[2][(hi >> 8) & 0xFF] ^
            kCrc.t[1][(hi >> 16) & 0xFF] ^ kCrc.t[0][hi >> 24];
        p += 8;
        n -= 8;
    }
    while (n--) c = kCrc.t[0][(c ^ *p++) & 0xFF] ^ (c >> 8);
    return ~c;
}

int32_t check_tensor_meta(const char* name, uint32_t dtype, uint32_t ndim, const int64_t* shape,
                          uint64_t nbytes) {
    if (!name) return fail(SLLM_E_INVAL, "tensor name is NULL");
    size_t len = std::strlen(name);
    if (len == 0 || len > kMaxName) return fail(SLLM_E_INVAL, "tensor name length %zu not in [1, %llu]", len, (unsigned long long)kMaxName);
    uint32_t isz = itemsize(dtype);
    if (!isz) return fail(SLLM_E_INVAL, "tensor '%s': unknown dtype %u", name, dtype);
    if (ndim > SLLM_MAX_NDIM) return fail(SLLM_E_INVAL, "tensor '%s': ndim %u > %d", name, ndim, SLLM_MAX_NDIM);
    if (ndim && !shape) return fail(SLLM_E_INVAL, "tensor '%s': shape is NULL", name);
    uint64_t numel = 1;
    for (uint32_t d = 0; d < ndim; ++d) {
        if (shape[d] < 0) return fail(SLLM_E_INVAL, "tensor '%s': negative dimension", name);
        if (!mul_ok(numel, (uint64_t)shape[d], &numel))
            return fail(SLLM_E_INVAL, "tensor '%s': element count overflows", name);
    }
    uint64_t want;
    if (!mul_ok(numel, isz, &want)) return fail(SLLM_E_INVAL, "tensor '%s': byte size overflows", name);
    if (want != nbytes)
        return fail(SLLM_E_INVAL, "tensor '%s': nbytes %llu != numel * itemsize = %llu", name,
                    (unsigned long long)nbytes, (unsigned long long)want);
    return SLLM_OK;
}

int32_t plan_layout(const uint64_t* sizes, size_t n, uint64_t align, uint64_t* out, uint64_t* total) {
    if (!is_pow2(align)) return fail(SLLM_E_INVAL, "alignment %llu is not a power of two", (unsigned long long)align);
    uint64_t cursor = 0;
    for (size_t i = 0; i < n; ++i) {
        uint64_t padded;
        if (out) out[i] = cursor;
        if (!align_up(sizes[i], align, &padded) || !add_ok(cursor, padded, &cursor))
            return fail(SLLM_E_INVAL, "layout size overflows 64 bits");
    }
    *total = cursor;
    return SLLM_OK;
}

std::string encode_index(const IndexData& ix) {
    std::string s;
    size_t est = kHeaderBytes + 4;
    for (const auto& t : ix.tensors) est += 24 + 8 * t.ndim + t.name.size();
    s.reserve(est);
    s.append(kMagic, 8);
    put_u32(s, kVersion);
    put_u32(s, 1);  // one partition
    put_u64(s, ix.alignment);
    put_u64(s, ix.chunk_size);
    put_u64(s, ix.total);
    put_u64(s, ix.file_bytes);
    put_u64(s, ix.tensors.size());
    for (const auto& t : ix.tensors) {
        put_u32(s, (uint32_t)t.name.size());
        s.append(t.name);
        s.push_back((char)t.dtype);
        s.push_back((char)t.ndim);
        put_u16(s, 0);  // partition (GPU id) 0
        for (uint32_t d = 0; d < t.ndim; ++d) put_u64(s, (uint64_t)t.shape[d]);
        put_u64(s, t.offset);
        put_u64(s, t.nbytes);
    }
    put_u32(s, crc32(s.data(), s.size()));
    return s;
}

int32_t decode_index(const void* data, size_t n, IndexData* out) {
    if (n < kHeaderBytes + 4) return fail(SLLM_E_FORMAT, "index is %zu bytes, shorter than its header", n);
    const uint8_t* p = static_cast<const uint8_t*>(data);
    uint32_t stored;
    std::memcpy(&stored, p + n - 4, 4);
    if (crc32(p, n - 4) != stored) return fail(SLLM_E_FORMAT, "index CRC mismatch");
    if (std::memcmp(p, kMagic, 8) != 0) return fail(SLLM_E_FORMAT, "bad index magic");
    Cursor c{p, n - 4, 8};
    uint32_t version, nparts;
    uint64_t count;
    IndexData ix;
    c.take(&version, 4);
    c.take(&nparts, 4);
    c.take(&ix.alignment, 8);
    c.take(&ix.chunk_size, 8);
    c.take(&ix.total, 8);
    c.take(&ix.file_bytes, 8);
    c.take(&count, 8);
    if (version != kVersion) return fail(SLLM_E_FORMAT, "unsupported index version %u", version);
    if (nparts != 1) return fail(SLLM_E_FORMAT, "index has %u partitions, expected 1", nparts);
    if (!is_pow2(ix.alignment)) return fail(SLLM_E_FORMAT, "index alignment is not a power of two");
    if (ix.chunk_size == 0) return fail(SLLM_E_FORMAT, "index chunk size is 0");
    // each record takes at least 25 bytes, which bounds a sane count
    if (count > (n - kHeaderBytes) / 25) return fail(SLLM_E_FORMAT, "index tensor count %llu is impossible", (unsigned long long)count);
    ix.tensors.resize(count);
    NameSet names(ix.tensors);
    uint64_t padded_sum = 0;
    for (uint64_t i = 0; i < count; ++i) {
        TensorRec& t = ix.tensors[i];
        uint32_t len;
        uint8_t dtype, ndim;
        uint16_t part;
        if (!c.take(&len, 4) || len == 0 || len > kMaxName || len > c.n - c.pos)
            return fail(SLLM_E_FORMAT, "record %llu: bad name length", (unsigned long long)i);
        t.name.assign(reinterpret_cast<const char*>(p + c.pos), len);
        c.pos += len;
        if (std::memchr(t.name.data(), 0, len)) return fail(SLLM_E_FORMAT, "record %llu: NUL in name", (unsigned long long)i);
        if (!c.take(&dtype, 1) || !c.take(&ndim, 1) || !c.take(&part, 2))
            return fail(SLLM_E_FORMAT, "record %llu truncated", (unsigned long long)i);
        if (part != 0) return fail(SLLM_E_FORMAT, "record '%s': partition %u, expected 0", t.name.c_str(), part);
        if (ndim > SLLM_MAX_NDIM) return fail(SLLM_E_FORMAT, "record '%s': ndim %u", t.name.c_str(), ndim);
        t.dtype = dtype;
        t.ndim = ndim;
        for (uint32_t d = 0; d < ndim; ++d)
            if (!c.take(&t.shape[d], 8)) return fail(SLLM_E_FORMAT, "record '%s' truncated", t.name.c_str());
        if (!c.take(&t.offset, 8) || !c.take(&t.nbytes, 8))
            return fail(SLLM_E_FORMAT, "record '%s' truncated", t.name.c_str());
        if (check_tensor_meta(t.name.c_str(), t.dtype, t.ndim, t.shape, t.nbytes) != SLLM_OK)
            return fail(SLLM_E_FORMAT, "record '%s': %s", t.name.c_str(), sllm_last_error());
        if (!names.insert((uint32_t)i)) return fail(SLLM_E_FORMAT, "duplicate tensor name '%s'", t.name.c_str());
        // tensors packed in order: o_i is the end of the previous padded slot
        if (t.offset != padded_sum)
            return fail(SLLM_E_FORMAT, "record '%s': offset %llu, expected %llu", t.name.c_str(),
                        (unsigned long long)t.offset, (unsigned long long)padded_sum);
        uint64_t slot;
        if (!align_up(t.nbytes, ix.alignment, &slot) || !add_ok(padded_sum, slot, &padded_sum))
            return fail(SLLM_E_FORMAT, "index sizes overflow");
    }
    if (c.pos != c.n) return fail(SLLM_E_FORMAT, "%zu trailing bytes in index", c.n - c.pos);
    if (padded_sum != ix.total)
        return fail(SLLM_E_FORMAT, "index total %llu != padded sum %llu", (unsigned long long)ix.total,
                    (unsigned long long)padded_sum);
    uint64_t f;
    if (!align_up(ix.total, kFileBlock, &f) || f != ix.file_bytes)
        return fail(SLLM_E_FORMAT, "index file length %llu != T rounded up to 4 KiB", (unsigned long long)ix.file_bytes);
    *out = std::move(ix);
    return SLLM_OK;
}

}  // namespace sllm
