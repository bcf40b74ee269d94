// CPU-only driver for the host-side format code, built with AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_sanitize.py.
//
//  1. Random checkpoints go through the streaming writer; their index must
//     decode, describe the aligned packed layout, and the data file must hold
//     every tensor's bytes with zero padding.
//  0. crc32 (table and carry-less-multiply paths) equals the bit-at-a-time
//     definition of the reflected IEEE CRC-32 on every length up to 300,
//     random longer buffers, unaligned starts, any initial value, and
//     chained calls.
//  2. A valid index is mutated (byte flips, truncation, growth), with its CRC
//     recomputed half of the time so that field validation is reached.  The
//     decoder must never fault, and any index it accepts must re-encode to
//     exactly the same bytes.
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <fstream>
#include <random>
#include <sstream>
#include <string>
#include <vector>

#include "format.hpp"
#include "json.hpp"
#include "sllm.h"

using namespace sllm;

// The CRC-32 of zlib by its definition: a 32-bit shift register over the
// message bits, least significant bit of each byte first, reflected
// polynomial 0xEDB88320, register and result inverted.
static uint32_t crc_bitwise(const uint8_t* p, size_t n, uint32_t crc) {
    uint32_t c = ~crc;
    for (size_t i = 0; i < n; ++i) {
        c ^= p[i];
        for (int b = 0; b < 8; ++b) c = (c & 1) ? (c >> 1) ^ 0xEDB88320u : c >> 1;
    }
    return ~c;
}

static std::string slurp(const std::string& path) {
    std::ifstream f(path, std::ios::binary);
    std::stringstream ss;
    ss << f.rdbuf();
    return ss.str();
}

#define CHECK(c)                                                             \
    do {                                                                     \
        if (!(c)) {                                                          \
            std::fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            return 1;                                                        \
        }                                                                    \
    } while (0)

int main(int argc, char** argv) {
    if (argc < 3) return 2;
    const std::string dir = argv[1];
    const long iters = std::atol(argv[2]);
    std::mt19937_64 rng(20240125);
    std::string valid;

    {  // 0. CRC-32 against its definition
        const char* check = "123456789";
        CHECK(crc32(check, 9) == 0xCBF43926u);
        std::vector<uint8_t> buf(4096 + 16);
        for (auto& b : buf) b = (uint8_t)rng();
        for (size_t n = 0; n <= 4096; n = n < 300 ? n + 1 : n + 1 + rng() % 97) {
            const size_t off = rng() % 16;
            const uint32_t init = (n % 3 == 0) ? 0u : (uint32_t)rng();
            const uint8_t* p = buf.data() + off;
            const uint32_t want = crc_bitwise(p, n, init);
            CHECK(crc32(p, n, init) == want);
            const size_t cut = n ? rng() % (n + 1) : 0;  // chained: crc of a then b == crc of a + b
            CHECK(crc32(p + cut, n - cut, crc32(p, cut, init)) == want);
        }
    }

    for (int round = 0; round < 60; ++round) {
        sllm_convert_opts o{1ull << (rng() % 13), 1 + rng() % 5000, 0, 0};
        sllm_writer* w = nullptr;
        CHECK(sllm_writer_open(dir.c_str(), &o, &w) == SLLM_OK);
        const int n = (int)(rng() % 24);
        std::vector<std::vector<uint8_t>> data(n);
        std::vector<uint64_t> sizes(n);
        for (int i = 0; i < n; ++i) {
            const uint32_t dtype = (uint32_t)(rng() % 4);
            const uint32_t ndim = (uint32_t)(rng() % 4);
            int64_t shape[4] = {1, 1, 1, 1};
            uint64_t numel = 1;
            for (uint32_t d = 0; d < ndim; ++d) {
                shape[d] = (int64_t)(rng() % 9);
                numel *= (uint64_t)shape[d];
            }
            sizes[i] = numel * itemsize(dtype);
            data[i].resize(sizes[i]);
            for (auto& b : data[i]) b = (uint8_t)(rng() & 0xFF);
            const std::string name = "t" + std::to_string(round) + "." + std::to_string(i);
            sllm_src_tensor t{name.c_str(), dtype, ndim, shape, data[i].data(), sizes[i]};
            CHECK(sllm_writer_add(w, &t) == SLLM_OK);
        }
        CHECK(sllm_writer_close(w) == SLLM_OK);
        const std::string blob = slurp(dir + "/sllm.index");
        const std::string part = slurp(dir + "/sllm.part0");
        IndexData ix;
        CHECK(decode_index(blob.data(), blob.size(), &ix) == SLLM_OK);
        CHECK(encode_index(ix) == blob);
        std::vector<uint64_t> off(n);
        uint64_t T = 0;
        CHECK(plan_layout(sizes.data(), (size_t)n, o.alignment, off.data(), &T) == SLLM_OK);
        CHECK(ix.total == T && part.size() == ix.file_bytes && ix.file_bytes % 4096 == 0 && ix.file_bytes - T < 4096);
        std::vector<uint8_t> used(part.size(), 0);
        for (int i = 0; i < n; ++i) {
            CHECK(ix.tensors[i].offset == off[i] && ix.tensors[i].nbytes == sizes[i]);
            if (!sizes[i]) continue;
            CHECK(std::memcmp(part.data() + off[i], data[i].data(), sizes[i]) == 0);
            std::memset(used.data() + off[i], 1, sizes[i]);
        }
        for (size_t x = 0; x < part.size(); ++x) CHECK(used[x] || part[x] == 0);
        if (n > 3) valid = blob;
    }
    CHECK(!valid.empty());

    long accepted = 0;
    for (long it = 0; it < iters; ++it) {
        std::string m = valid;
        const int kind = (int)(rng() % 4);
        if (kind == 0) {
            m.resize(rng() % (m.size() + 1));
        } else if (kind == 1) {
            const size_t extra = 1 + rng() % 64;
            for (size_t k = 0; k < extra; ++k) m.insert(m.begin() + (long)(rng() % (m.size() + 1)), (char)(rng() & 0xFF));
        } else {
            const int flips = 1 + (int)(rng() % 4);
            for (int k = 0; k < flips; ++k) m[rng() % m.size()] ^= (char)(1u << (rng() % 8));
        }
        if ((rng() & 1) && m.size() >= 4) {  // recompute the CRC so the fields themselves are checked
            const uint32_t c = crc32(m.data(), m.size() - 4);
            std::memcpy(&m[m.size() - 4], &c, 4);
        }
        IndexData ix;
        if (decode_index(m.data(), m.size(), &ix) == SLLM_OK) {
            ++accepted;
            CHECK(encode_index(ix) == m);
        }
    }
    // 3. The safetensors header reader: mutations of a realistic header must
    //    parse or fail cleanly, never read out of bounds.
    const std::string header =
        "{\"__metadata__\":{\"format\":\"pt\"},\"model.embed.weight\":{\"dtype\":\"BF16\","
        "\"shape\":[32000,4096],\"data_offsets\":[0,262144000]},\"a\\u00e9\\ud83d\\ude00\":{\"dtype\":"
        "\"F32\",\"shape\":[],\"data_offsets\":[262144000,262144004]},\"n\":[1.5e3,-0,true,false,null]}";
    {
        json::Value v;
        json::Parser p(header.data(), header.size());
        CHECK(p.parse(&v) && v.kind == json::Value::Object && v.fields.size() == 4);
        CHECK(v.fields[2].first == "a\xc3\xa9\xf0\x9f\x98\x80");
    }
    long parsed = 0;
    for (long it = 0; it < iters / 2; ++it) {
        std::string m = header;
        const int edits = 1 + (int)(rng() % 6);
        for (int k = 0; k < edits; ++k) {
            const int kind = (int)(rng() % 3);
            const size_t at = rng() % (m.size() + 1);
            if (kind == 0 && !m.empty()) m.erase(rng() % m.size(), 1 + rng() % 8);
            else if (kind == 1) {
                static const char alphabet[] = "{}[],:\"\\u0e-1 ";
                m.insert(m.begin() + (long)std::min(at, m.size()), alphabet[rng() % (sizeof alphabet - 1)]);
            }
            else if (!m.empty()) m[rng() % m.size()] = (char)(rng() & 0xFF);
        }
        json::Value v;
        json::Parser p(m.data(), m.size());
        parsed += p.parse(&v);
    }
    std::printf("ok rounds=60 mutants=%ld accepted=%ld json_parsed=%ld\n", iters, accepted, parsed);
    return 0;
}
