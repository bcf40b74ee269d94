// CPU-only check of the chunk reader (csrc/io.cpp), built with AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_sanitize.py.
//
// For buffered files read with pread, read with pread through a small buffer
// copied with streaming stores (SLLM_READ_STREAM=1), and read through the file
// mapping with streaming stores (SLLM_READ_MAPPED=1): random chunk offsets and lengths,
// destinations at every alignment mod 32, the bytes equal the file's; after
// the file is truncated, a chunk past the new end is an I/O error (not a
// fault) and a chunk before it still reads.
#include <fcntl.h>
#include <unistd.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <vector>

#include "common.hpp"
#include "io.hpp"

using namespace sllm;

// mode 0: pread, 1: pread through the streaming buffer, 2: mapped
static int check(const std::string& path, const std::vector<uint8_t>& bytes, int mode, std::mt19937_64& rng) {
    const bool mapped = mode == 2;
    setenv("SLLM_READ_MAPPED", mapped ? "1" : "0", 1);
    setenv("SLLM_READ_STREAM", mode == 1 ? "1" : "0", 1);
    DataFile f;
    if (open_data(path, false, &f) != SLLM_OK) {
        std::printf("open failed: %s\n", sllm_last_error());
        return 1;
    }
    if ((f.map != nullptr) != mapped) {
        std::printf("mapping %s expected\n", mapped ? "" : "not");
        return 1;
    }
    std::vector<uint8_t> buf(bytes.size() + 64);
    for (int it = 0; it < 400; ++it) {
        const uint64_t off = rng() % bytes.size();
        const uint64_t n = 1 + rng() % std::min<uint64_t>(bytes.size() - off, (it % 4 == 0) ? 9u << 20 : 70000);
        const uint64_t shift = rng() % 33;
        std::memset(buf.data(), 0xEE, n + shift + 8);
        if (read_chunk(f, buf.data() + shift, n, off, path, nullptr) != SLLM_OK) {
            std::printf("read at %llu (%llu bytes) failed: %s\n", (unsigned long long)off, (unsigned long long)n,
                        sllm_last_error());
            return 1;
        }
        if (std::memcmp(buf.data() + shift, bytes.data() + off, n) != 0 || buf[shift + n] != 0xEE ||
            (shift && buf[shift - 1] != 0xEE)) {
            std::printf("bytes differ at %llu (%llu bytes, shift %llu, mode %d)\n", (unsigned long long)off,
                        (unsigned long long)n, (unsigned long long)shift, mode);
            return 1;
        }
    }
    // past the end of the file as opened
    if (read_chunk(f, buf.data(), 100, bytes.size() - 50, path, nullptr) != SLLM_E_IO) {
        std::printf("read past the end was not an I/O error\n");
        return 1;
    }
    // truncated while open: a chunk past the new end fails cleanly
    const uint64_t cut = bytes.size() / 2;
    if (truncate(path.c_str(), (off_t)cut) != 0) return 1;
    const int32_t st = read_chunk(f, buf.data(), 1 << 20, cut + 8192, path, nullptr);
    if (st != SLLM_E_IO) {
        std::printf("read past a truncation returned %d (mode %d)\n", st, mode);
        return 1;
    }
    if (read_chunk(f, buf.data(), 4096, 0, path, nullptr) != SLLM_OK || std::memcmp(buf.data(), bytes.data(), 4096)) {
        std::printf("read before the truncation failed\n");
        return 1;
    }
    close_data(&f);
    return 0;
}

int main(int argc, char** argv) {
    if (argc < 2) return 2;
    const std::string dir = argv[1];
    std::mt19937_64 rng(20261202);
    for (int mode = 0; mode < 3; ++mode) {
        std::vector<uint8_t> bytes((24u << 20) + 1234);
        for (auto& b : bytes) b = (uint8_t)rng();
        const std::string path = dir + "/data" + std::to_string(mode);
        FILE* fp = std::fopen(path.c_str(), "wb");
        if (!fp || std::fwrite(bytes.data(), 1, bytes.size(), fp) != bytes.size()) return 1;
        std::fclose(fp);
        if (check(path, bytes, mode, rng)) return 1;
    }
    std::printf("ok\n");
    return 0;
}
