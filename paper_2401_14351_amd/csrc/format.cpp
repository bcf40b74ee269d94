#include "format.hpp"

#include <immintrin.h>

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
inline uint64_t name_hash(std::string_view s) {
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
    explicit NameSet(const IndexData& ix) : ix_(ix) {
        size_t cap = 16;
        while (cap < 2 * ix.tensors.size()) cap <<= 1;
        slot_.assign(cap, kEmpty);
        hash_.resize(ix.tensors.size());
    }
    // false if record i's name is already in the set
    bool insert(uint32_t i) {
        const std::string_view name = ix_.name_view(i);
        const uint64_t h = name_hash(name);
        hash_[i] = h;
        for (size_t k = h & (slot_.size() - 1);; k = (k + 1) & (slot_.size() - 1)) {
            const uint32_t j = slot_[k];
            if (j == kEmpty) {
                slot_[k] = i;
                return true;
            }
            if (hash_[j] == h && ix_.name_view(j) == name) return false;
        }
    }

  private:
    static constexpr uint32_t kEmpty = UINT32_MAX;
    const IndexData& ix_;
    std::vector<uint32_t> slot_;
    std::vector<uint64_t> hash_;
};

}  // namespace

namespace {

// Raw (uninverted) CRC state c advanced over n bytes by table lookups:
// slicing-by-8, then one byte at a time.
uint32_t crc_tables(uint32_t c, const uint8_t* p, size_t n) {
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
    return c;
}

// Carry-less-multiply folding (Gopal et al., "Fast CRC Computation for
// Generic Polynomials Using PCLMULQDQ Instruction", Intel, 2009), in the
// bit-reflected order of this CRC.  A 128-bit block loaded little-endian
// holds the message polynomial with byte 0's bit 0 as its highest
// coefficient: bit k stands for x^(127-k).  Folding block A over the next
// block D uses A x^128 + D = U x^192 + U' x^128 + D, where U (the low 64
// bits) and U' (the high 64) are A's halves.  The product of a reflected
// 64-bit U and a reflected constant shifted up one bit lands with bit k for
// x^(95-k), i.e. it carries an extra x^32 in the block's frame, so the
// constants are x^(192-32) and x^(128-32) mod P; folding over 512 bits uses
// x^(576-32) and x^(512-32).  The folded remainder S is congruent to the
// message, so the raw CRC (message x^32 mod P) is the table CRC of S's 16
// bytes from state 0; the bytes past the last whole block follow by table.
struct FoldKeys {
    uint64_t lo1, hi1, lo4, hi4;  // (x^160, x^96), (x^544, x^480) mod P, reflected, << 1
    FoldKeys() {
        lo1 = key(160);
        hi1 = key(96);
        lo4 = key(544);
        hi4 = key(480);
    }
    // x^e mod P as the reflected 32-bit value (bit j for x^(31-j)), shifted
    // up one bit: start from x^0 and multiply by x e times
    static uint64_t key(int e) {
        uint32_t r = 0x80000000u;
        for (int i = 0; i < e; ++i) r = (r & 1) ? (r >> 1) ^ 0xEDB88320u : r >> 1;
        return (uint64_t)r << 1;
    }
};
const FoldKeys kFold;

__attribute__((target("pclmul,sse4.1"))) inline __m128i fold(__m128i a, __m128i k) {
    return _mm_xor_si128(_mm_clmulepi64_si128(a, k, 0x00), _mm_clmulepi64_si128(a, k, 0x11));
}

__attribute__((target("pclmul,sse4.1"))) uint32_t crc_fold(uint32_t c, const uint8_t* p, size_t n) {
    auto load = [](const uint8_t* q) { return _mm_loadu_si128(reinterpret_cast<const __m128i*>(q)); };
    // n >= 64: four blocks 512 bits apart, the state injected into the first
    __m128i x0 = _mm_xor_si128(load(p), _mm_cvtsi32_si128((int)c));
    __m128i x1 = load(p + 16), x2 = load(p + 32), x3 = load(p + 48);
    p += 64;
    n -= 64;
    const __m128i k4 = _mm_set_epi64x((long long)kFold.hi4, (long long)kFold.lo4);
    for (; n >= 64; p += 64, n -= 64) {
        x0 = _mm_xor_si128(fold(x0, k4), load(p));
        x1 = _mm_xor_si128(fold(x1, k4), load(p + 16));
        x2 = _mm_xor_si128(fold(x2, k4), load(p + 32));
        x3 = _mm_xor_si128(fold(x3, k4), load(p + 48));
    }
    const __m128i k1 = _mm_set_epi64x((long long)kFold.hi1, (long long)kFold.lo1);
    x1 = _mm_xor_si128(fold(x0, k1), x1);
    x2 = _mm_xor_si128(fold(x1, k1), x2);
    x3 = _mm_xor_si128(fold(x2, k1), x3);
    for (; n >= 16; p += 16, n -= 16) x3 = _mm_xor_si128(fold(x3, k1), load(p));
    alignas(16) uint8_t s[16];
    _mm_store_si128(reinterpret_cast<__m128i*>(s), x3);
    return crc_tables(crc_tables(0, s, 16), p, n);
}

bool have_clmul() {
    static const bool ok = __builtin_cpu_supports("pclmul") && __builtin_cpu_supports("sse4.1");
    return ok;
}

}  // namespace

uint32_t crc32(const void* data, size_t n, uint32_t crc) {
    const uint8_t* p = static_cast<const uint8_t*>(data);
    if (n >= 64 && have_clmul()) return ~crc_fold(~crc, p, n);
    return ~crc_tables(~crc, p, n);
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
    for (const auto& t : ix.tensors) est += 24 + 8 * t.ndim + t.name_len;
    s.reserve(est);
    s.append(kMagic, 8);
    put_u32(s, kVersion);
    put_u32(s, 1);  // one partition
    put_u64(s, ix.alignment);
    put_u64(s, ix.chunk_size);
    put_u64(s, ix.total);
    put_u64(s, ix.file_bytes);
    put_u64(s, ix.tensors.size());
    for (size_t i = 0; i < ix.tensors.size(); ++i) {
        const TensorRec& t = ix.tensors[i];
        put_u32(s, t.name_len);
        s.append(ix.name_view(i));
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
    ix.names.reserve(n);  // the names fit in the index, so the buffer never moves
    NameSet names(ix);
    uint64_t padded_sum = 0;
    for (uint64_t i = 0; i < count; ++i) {
        TensorRec& t = ix.tensors[i];
        uint32_t len;
        uint8_t dtype, ndim;
        uint16_t part;
        if (!c.take(&len, 4) || len == 0 || len > kMaxName || len > c.n - c.pos)
            return fail(SLLM_E_FORMAT, "record %llu: bad name length", (unsigned long long)i);
        if (std::memchr(p + c.pos, 0, len)) return fail(SLLM_E_FORMAT, "record %llu: NUL in name", (unsigned long long)i);
        ix.set_name(t, reinterpret_cast<const char*>(p + c.pos), len);
        c.pos += len;
        const char* name = ix.name(i);
        if (!c.take(&dtype, 1) || !c.take(&ndim, 1) || !c.take(&part, 2))
            return fail(SLLM_E_FORMAT, "record %llu truncated", (unsigned long long)i);
        if (part != 0) return fail(SLLM_E_FORMAT, "record '%s': partition %u, expected 0", name, part);
        if (ndim > SLLM_MAX_NDIM) return fail(SLLM_E_FORMAT, "record '%s': ndim %u", name, ndim);
        t.dtype = dtype;
        t.ndim = ndim;
        for (uint32_t d = 0; d < ndim; ++d)
            if (!c.take(&t.shape[d], 8)) return fail(SLLM_E_FORMAT, "record '%s' truncated", name);
        if (!c.take(&t.offset, 8) || !c.take(&t.nbytes, 8))
            return fail(SLLM_E_FORMAT, "record '%s' truncated", name);
        if (check_tensor_meta(name, t.dtype, t.ndim, t.shape, t.nbytes) != SLLM_OK)
            return fail(SLLM_E_FORMAT, "record '%s': %s", name, sllm_last_error());
        if (!names.insert((uint32_t)i)) return fail(SLLM_E_FORMAT, "duplicate tensor name '%s'", name);
        // tensors packed in order: o_i is the end of the previous padded slot
        if (t.offset != padded_sum)
            return fail(SLLM_E_FORMAT, "record '%s': offset %llu, expected %llu", name,
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
