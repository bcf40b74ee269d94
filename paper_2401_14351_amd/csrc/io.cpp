#include "io.hpp"

#include <fcntl.h>
#include <immintrin.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <cerrno>
#include <cstdlib>
#include <cstring>

#include "common.hpp"

#ifndef STATX_DIOALIGN
#define STATX_DIOALIGN 0x00002000U
#endif
#ifndef MADV_POPULATE_READ
#define MADV_POPULATE_READ 22
#endif

namespace sllm {

namespace {

// The O_DIRECT alignment the kernel reports for this file (statx with
// STATX_DIOALIGN, Linux 6.1+), else the 4 KiB that common block devices
// accept.  The two fields are read from the kernel's struct statx layout
// (u32 stx_dio_mem_align at byte 152, u32 stx_dio_offset_align at 156) so
// that older C library headers still build.
uint64_t query_dio_align(int fd) {
#ifdef SYS_statx
    alignas(8) unsigned char sx[256];
    std::memset(sx, 0, sizeof sx);
    if (syscall(SYS_statx, fd, "", AT_EMPTY_PATH, STATX_DIOALIGN, sx) == 0) {
        uint32_t mask, mem_align, off_align;
        std::memcpy(&mask, sx + 0, 4);
        std::memcpy(&mem_align, sx + 152, 4);
        std::memcpy(&off_align, sx + 156, 4);
        if ((mask & STATX_DIOALIGN) && off_align) return mem_align > off_align ? mem_align : off_align;
    }
#endif
    return 4096;
}

}  // namespace

int32_t open_data(const std::string& path, bool want_direct, DataFile* out) {
    DataFile f;
    if (want_direct) {
        f.fd = ::open(path.c_str(), O_RDONLY | O_CLOEXEC | O_DIRECT);
        if (f.fd >= 0) {
            f.direct = true;
        } else if (errno != EINVAL) {
            return fail(SLLM_E_IO, "open %s: %s", path.c_str(), std::strerror(errno));
        } else {
            log_msg(1, "O_DIRECT refused for %s; reading buffered", path.c_str());
        }
    }
    if (f.fd < 0) {
        f.fd = ::open(path.c_str(), O_RDONLY | O_CLOEXEC);
        if (f.fd < 0) return fail(SLLM_E_IO, "open %s: %s", path.c_str(), std::strerror(errno));
    }
    struct stat st;
    if (::fstat(f.fd, &st) != 0) {
        int32_t r = fail(SLLM_E_IO, "fstat %s: %s", path.c_str(), std::strerror(errno));
        ::close(f.fd);
        return r;
    }
    f.size = (uint64_t)st.st_size;
    f.dev = (uint64_t)st.st_dev;
    f.ino = (uint64_t)st.st_ino;
    f.mtime_ns = (uint64_t)st.st_mtim.tv_sec * 1000000000ull + (uint64_t)st.st_mtim.tv_nsec;
    f.dio_align = f.direct ? query_dio_align(f.fd) : 1;
    if (!f.direct && f.size && mapped_reads()) {
        void* m = ::mmap(nullptr, f.size, PROT_READ, MAP_SHARED, f.fd, 0);
        if (m != MAP_FAILED) {
            const uint64_t len = f.size;
            f.map = std::shared_ptr<const uint8_t>(static_cast<const uint8_t*>(m),
                                                   [len](const uint8_t* p) { ::munmap((void*)p, len); });
        } else {
            log_msg(1, "mmap %s failed (%s); reading with pread", path.c_str(), std::strerror(errno));
        }
    }
    *out = f;
    return SLLM_OK;
}

void close_data(DataFile* f) {
    if (f->fd >= 0) ::close(f->fd);
    f->fd = -1;
    f->map.reset();
}

namespace {

// dst <- src, n bytes, with non-temporal 32-byte stores where dst is
// aligned (the pinned chunks are page-aligned), then a store fence so the
// bytes are globally visible before the chunk is handed on.
__attribute__((target("avx2"))) void copy_stream_avx2(uint8_t* dst, const uint8_t* src, uint64_t n) {
    uint64_t head = (32 - (reinterpret_cast<uintptr_t>(dst) & 31)) & 31;
    if (head > n) head = n;
    std::memcpy(dst, src, head);
    dst += head;
    src += head;
    n -= head;
    uint64_t i = 0;
    for (; i + 128 <= n; i += 128) {
        const __m256i a = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(src + i));
        const __m256i b = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(src + i + 32));
        const __m256i c = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(src + i + 64));
        const __m256i d = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(src + i + 96));
        _mm256_stream_si256(reinterpret_cast<__m256i*>(dst + i), a);
        _mm256_stream_si256(reinterpret_cast<__m256i*>(dst + i + 32), b);
        _mm256_stream_si256(reinterpret_cast<__m256i*>(dst + i + 64), c);
        _mm256_stream_si256(reinterpret_cast<__m256i*>(dst + i + 96), d);
    }
    std::memcpy(dst + i, src + i, n - i);
    _mm_sfence();
}

void copy_stream(uint8_t* dst, const uint8_t* src, uint64_t n) {
    static const bool avx2 = __builtin_cpu_supports("avx2");
    if (avx2) copy_stream_avx2(dst, src, n);
    else std::memcpy(dst, src, n);
}

// Chunk copies per populate call: a populate of a whole 64 MiB chunk would
// hold the file's page-table lock for long; 4 MiB steps keep copy and
// populate interleaved.
constexpr uint64_t kMapStep = 4u << 20;

// 0 on success, else the errno of the failing read (-1 for end of file).
int pread_exact(int fd, void* buf, uint64_t n, uint64_t off) {
    uint8_t* p = static_cast<uint8_t*>(buf);
    while (n) {
        ssize_t r = ::pread(fd, p, n, (off_t)off);
        if (r < 0) {
            if (errno == EINTR) continue;
            return errno;
        }
        if (r == 0) return -1;
        p += r;
        off += (uint64_t)r;
        n -= (uint64_t)r;
    }
    return 0;
}

int32_t read_error(int e, const std::string& path, uint64_t off) {
    if (e < 0) return fail(SLLM_E_IO, "read %s at %llu: unexpected end of file", path.c_str(), (unsigned long long)off);
    return fail(SLLM_E_IO, "read %s at %llu: %s", path.c_str(), (unsigned long long)off, std::strerror(e));
}

// 16 MiB: one read of a 16 MiB chunk, which the block layer splits into
// several requests in flight at once (a deeper queue than 4 MiB reads give)
constexpr uint64_t kBounceBytes = 16u << 20;

struct Bounce {
    void* p = nullptr;
    ~Bounce() { std::free(p); }
};

uint8_t* bounce_buffer() {
    thread_local Bounce b;
    if (!b.p && posix_memalign(&b.p, 4096, kBounceBytes) != 0) b.p = nullptr;
    return static_cast<uint8_t*>(b.p);
}

}  // namespace

int32_t pread_full(const DataFile& f, void* buf, uint64_t n, uint64_t off, const std::string& path) {
    int e = pread_exact(f.fd, buf, n, off);
    return e ? read_error(e, path, off) : SLLM_OK;
}

namespace {

// 1 MiB: small enough to stay in the reader core's caches between the read
// into it and the copy out of it
constexpr uint64_t kStreamBytes = 1u << 20;

uint8_t* stream_buffer() {
    thread_local Bounce b;
    if (!b.p && posix_memalign(&b.p, 4096, kStreamBytes) != 0) b.p = nullptr;
    return static_cast<uint8_t*>(b.p);
}

// Buffered read through a small cache-resident buffer, copied into dst with
// streaming stores: a pinned chunk then holds its bytes in DRAM rather than
// dirty in the CPU's caches, where the GPU's reads of it would have to be
// served by snoops (measured slower at the start of a streamed load).
int32_t pread_streamed(const DataFile& f, void* dst, uint64_t n, uint64_t off, const std::string& path) {
    uint8_t* b = stream_buffer();
    if (!b) return pread_full(f, dst, n, off, path);
    uint8_t* d = static_cast<uint8_t*>(dst);
    for (uint64_t done = 0; done < n;) {
        const uint64_t k = n - done < kStreamBytes ? n - done : kStreamBytes;
        const int e = pread_exact(f.fd, b, k, off + done);
        if (e) return read_error(e, path, off + done);
        copy_stream(d + done, b, k);
        done += k;
    }
    return SLLM_OK;
}

}  // namespace

int32_t read_chunk(const DataFile& f, void* dst, uint64_t n, uint64_t off, const std::string& path,
                   uint64_t* bounced) {
    if (!f.direct && f.map) {
        if (off > f.size || n > f.size - off)
            return fail(SLLM_E_IO, "read %s at %llu: unexpected end of file", path.c_str(), (unsigned long long)off);
        const uintptr_t page = 4096;
        uint8_t* d = static_cast<uint8_t*>(dst);
        for (uint64_t done = 0; done < n;) {
            const uint64_t k = n - done < kMapStep ? n - done : kMapStep;
            const uint8_t* s = f.map.get() + off + done;
            // populate the pages first: a range the file no longer covers
            // (truncated since it was opened) fails here instead of faulting
            const uintptr_t a0 = reinterpret_cast<uintptr_t>(s) & ~(page - 1);
            const uintptr_t a1 = reinterpret_cast<uintptr_t>(s + k);
            if (::madvise(reinterpret_cast<void*>(a0), a1 - a0, MADV_POPULATE_READ) != 0) {
                // a kernel without MADV_POPULATE_READ (EINVAL) reads the rest with pread
                if (errno == EINVAL) return pread_full(f, d + done, n - done, off + done, path);
                return read_error(errno == EFAULT ? -1 : errno, path, off + done);
            }
            copy_stream(d + done, s, k);
            // drop the page-table entries again (the pages stay in the page
            // cache): the reader thread pays that teardown while the GPU
            // moves earlier chunks, instead of the caller at close
            (void)::madvise(reinterpret_cast<void*>(a0), a1 - a0, MADV_DONTNEED);
            done += k;
        }
        return SLLM_OK;
    }
    if (!f.direct) return stream_reads() ? pread_streamed(f, dst, n, off, path) : pread_full(f, dst, n, off, path);
    if (f.direct_into_pinned->load() != 0) {
        int e = pread_exact(f.fd, dst, n, off);
        if (e == 0) {
            f.direct_into_pinned->store(1);
            return SLLM_OK;
        }
        if (e != EFAULT) return read_error(e, path, off);
        if (f.direct_into_pinned->exchange(0) != 0)
            log_msg(1, "direct reads cannot target pinned chunks; staging through a bounce buffer");
    }
    uint8_t* b = bounce_buffer();
    if (!b) return fail(SLLM_E_NOMEM, "no memory for a direct-read bounce buffer");
    uint8_t* d = static_cast<uint8_t*>(dst);
    for (uint64_t done = 0; done < n;) {
        const uint64_t k = n - done < kBounceBytes ? n - done : kBounceBytes;
        int e = pread_exact(f.fd, b, k, off + done);
        if (e) return read_error(e, path, off + done);
        copy_stream(d + done, b, k);  // streaming stores, as for buffered reads
        done += k;
    }
    if (bounced) *bounced += n;
    return SLLM_OK;
}

void drop_cache(const DataFile& f) { (void)::posix_fadvise(f.fd, 0, 0, POSIX_FADV_DONTNEED); }

bool mapped_reads() {
    const char* s = std::getenv("SLLM_READ_MAPPED");
    return s && *s == '1';
}

bool stream_reads() {
    const char* s = std::getenv("SLLM_READ_STREAM");
    return !(s && *s == '0');
}

}  // namespace sllm
