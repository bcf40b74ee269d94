// Pinned host chunk pool (the DRAM tier of Sec. 4.2) and the partitions
// cached in it.
#include "pool.hpp"

#include <fcntl.h>
#include <limits.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cerrno>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <thread>

#include "hip_util.hpp"
#include "workers.hpp"

using namespace sllm;

namespace sllm {

int32_t pool_take(sllm_pool* p, uint64_t n, std::vector<uint32_t>* out) {
    if (n > p->free_ids.size())
        return fail(SLLM_E_NOMEM, "pool has %zu free chunks, %llu needed", p->free_ids.size(), (unsigned long long)n);
    out->clear();
    out->reserve(n);
    for (uint64_t i = 0; i < n; ++i) {
        out->push_back(p->free_ids.back());
        p->free_ids.pop_back();
    }
    return SLLM_OK;
}

void pool_give(sllm_pool* p, const std::vector<uint32_t>& ids) {
    p->free_ids.insert(p->free_ids.end(), ids.begin(), ids.end());
    // keep the lowest ids at the back so later takes get address-ordered runs
    std::sort(p->free_ids.begin(), p->free_ids.end(), std::greater<uint32_t>());
}

CacheEntry* pool_find(sllm_pool* p, const DataFile& f) {
    for (auto& e : p->cache)
        if (e->dev == f.dev && e->ino == f.ino && e->size == f.size && e->mtime_ns == f.mtime_ns) return e.get();
    return nullptr;
}

// Read a whole file into a string.
int32_t read_small_file(const std::string& path, std::string* out) {
    int fd = ::open(path.c_str(), O_RDONLY | O_CLOEXEC);
    if (fd < 0) return fail(SLLM_E_IO, "open %s: %s", path.c_str(), std::strerror(errno));
    struct stat st;
    if (::fstat(fd, &st) != 0) {
        ::close(fd);
        return fail(SLLM_E_IO, "fstat %s: %s", path.c_str(), std::strerror(errno));
    }
    if (st.st_size > (1ll << 32)) {
        ::close(fd);
        return fail(SLLM_E_FORMAT, "%s is implausibly large", path.c_str());
    }
    out->resize((size_t)st.st_size);
    size_t got = 0;
    while (got < out->size()) {
        ssize_t r = ::read(fd, &(*out)[got], out->size() - got);
        if (r < 0 && errno == EINTR) continue;
        if (r <= 0) {
            ::close(fd);
            return fail(SLLM_E_IO, "read %s: %s", path.c_str(), r < 0 ? std::strerror(errno) : "short read");
        }
        got += (size_t)r;
    }
    ::close(fd);
    return SLLM_OK;
}

// Run fn(k) for k in [0, n) on `threads` threads; stop at the first failure
// and return its status (with its message re-recorded on the calling thread).
int32_t parallel_chunks(uint64_t n, uint32_t threads, const std::function<int32_t(uint64_t)>& fn) {
    std::atomic<uint64_t> next{0};
    std::atomic<int32_t> status{SLLM_OK};
    std::mutex mu;
    std::string msg;
    auto worker = [&] {
        for (;;) {
            if (status.load() != SLLM_OK) return;
            uint64_t k = next.fetch_add(1);
            if (k >= n) return;
            int32_t st = fn(k);
            if (st != SLLM_OK) {
                std::lock_guard<std::mutex> g(mu);
                if (status.load() == SLLM_OK) {
                    msg = sllm_last_error();
                    status.store(st);
                }
                return;
            }
        }
    };
    uint32_t nt = (uint32_t)std::min<uint64_t>(threads ? threads : 1, n ? n : 1);
    {
        // the caller is one of the workers; fewer threads than asked is fine
        // (the ones running finish the work)
        TaskGroup helpers;
        if (nt > 1 && helpers.start(nt - 1, [&](uint32_t) { worker(); }) != SLLM_OK) clear_error();
        worker();
        helpers.wait();
    }
    if (status.load() != SLLM_OK) return fail(status.load(), "%s", msg.c_str());
    return SLLM_OK;
}

std::string canonical_dir(const char* dir) {
    char buf[PATH_MAX];
    return ::realpath(dir, buf) ? std::string(buf) : std::string(dir);
}

int32_t pool_chunk_table(sllm_pool* p, const std::vector<uint32_t>& ids, const uint8_t*** out) {
    *out = nullptr;
    if (ids.empty()) return SLLM_OK;
    DeviceGuard guard(p->device);
    std::vector<const uint8_t*> table(ids.size());
    for (size_t k = 0; k < ids.size(); ++k) table[k] = p->mapped[ids[k]];
    const uint8_t** d = nullptr;
    hipError_t he = hipMalloc(reinterpret_cast<void**>(&d), table.size() * sizeof(void*));
    if (he == hipSuccess) he = hipMemcpy(d, table.data(), table.size() * sizeof(void*), hipMemcpyHostToDevice);
    if (he != hipSuccess) {
        if (d) (void)hipFree(d);
        return fail(SLLM_E_HIP, "chunk table upload failed: %s", hipGetErrorString(he));
    }
    *out = d;
    return SLLM_OK;
}

void pool_free_table(sllm_pool* p, const uint8_t** d_table) {
    if (!d_table) return;
    DeviceGuard guard(p->device);
    (void)hipFree(const_cast<uint8_t**>(d_table));
}

int32_t pool_adopt(sllm_pool* p, const char* dir, const DataFile& f, uint64_t total, const std::vector<uint32_t>& ids,
                   const uint8_t** d_table, int refs, CacheEntry** out) {
    auto e = std::make_unique<CacheEntry>();
    e->dir = canonical_dir(dir);
    e->dev = f.dev;
    e->ino = f.ino;
    e->size = f.size;
    e->mtime_ns = f.mtime_ns;
    e->total = total;
    e->chunks = ids;
    e->d_table = d_table;
    e->refs = refs;
    std::lock_guard<std::mutex> g(p->mu);
    if (pool_find(p, f)) return fail(SLLM_E_BUSY, "%s is already cached", dir);
    if (out) *out = e.get();
    p->cache.push_back(std::move(e));
    return SLLM_OK;
}

}  // namespace sllm

namespace {

uint64_t arena_target_bytes() {
    const char* s = std::getenv("SLLM_POOL_ARENA_MB");
    long mb = s ? std::strtol(s, nullptr, 10) : 0;
    return (mb > 0 ? (uint64_t)mb : 1024ull) << 20;
}

void destroy_pool(sllm_pool* p) {
    for (auto& e : p->cache)
        if (e->d_table) (void)hipFree(e->d_table);
    for (void* a : p->arenas) (void)hipHostFree(a);
    delete p;
}

// Touch every 4 KiB page of the new arenas once, from several threads, so
// that the CPU page tables of the pinned memory are populated when the pool
// is created: the first CPU write to a page of a fresh pinned allocation
// takes a page fault, which would otherwise be paid by the first fill of
// each chunk (the pool is a pre-allocated tier, Sec. 4.2).
void prefault(const std::vector<void*>& arenas, uint64_t arena_bytes_last, uint64_t arena_bytes) {
    constexpr uint64_t kPiece = 64ull << 20;
    struct Piece {
        uint8_t* p;
        uint64_t n;
    };
    std::vector<Piece> pieces;
    for (size_t a = 0; a < arenas.size(); ++a) {
        const uint64_t n = a + 1 == arenas.size() ? arena_bytes_last : arena_bytes;
        for (uint64_t o = 0; o < n; o += kPiece)
            pieces.push_back({static_cast<uint8_t*>(arenas[a]) + o, std::min(kPiece, n - o)});
    }
    const unsigned hw = std::thread::hardware_concurrency();
    (void)parallel_chunks(pieces.size(), std::min(16u, hw ? hw : 1u), [&](uint64_t k) {
        volatile uint8_t* p = pieces[k].p;
        for (uint64_t o = 0; o < pieces[k].n; o += 4096) p[o] = 0;
        return SLLM_OK;
    });
}

}  // namespace

extern "C" int32_t sllm_pool_create(uint64_t chunk_size, uint64_t n_chunks, int32_t device, sllm_pool** out) try {
    clear_error();
    if (!out) return fail(SLLM_E_INVAL, "out is NULL");
    *out = nullptr;
    if (chunk_size == 0 || n_chunks == 0) return fail(SLLM_E_INVAL, "chunk size and chunk count must be >= 1");
    if (n_chunks > 0xFFFFFFFFull) return fail(SLLM_E_INVAL, "too many chunks");
    uint64_t stride, total;
    if (!align_up(chunk_size, 4096, &stride) || !mul_ok(stride, n_chunks, &total))
        return fail(SLLM_E_INVAL, "pool size overflows");
    int count = 0;
    SLLM_HIP(hipGetDeviceCount(&count));
    if (device < 0 || device >= count) return fail(SLLM_E_INVAL, "device %d not present (%d devices)", device, count);
    DeviceGuard guard(device);
    if (!guard.ok()) return fail(SLLM_E_HIP, "cannot make device %d current", device);
    auto* p = new (std::nothrow) sllm_pool;
    if (!p) return fail(SLLM_E_NOMEM, "out of host memory");
    p->device = device;
    p->chunk = chunk_size;
    p->stride = stride;
    const uint64_t per_arena = std::max<uint64_t>(1, arena_target_bytes() / stride);
    p->host.reserve(n_chunks);
    p->mapped.reserve(n_chunks);
    p->arena_of.reserve(n_chunks);
    for (uint64_t done = 0; done < n_chunks;) {
        const uint64_t k = std::min(per_arena, n_chunks - done);
        void* h = nullptr;
        hipError_t e = hipHostMalloc(&h, k * stride, hipHostMallocDefault);
        if (e != hipSuccess) {
            destroy_pool(p);
            return fail(SLLM_E_HIP, "hipHostMalloc(%llu bytes) failed: %s", (unsigned long long)(k * stride), hipGetErrorString(e));
        }
        p->arenas.push_back(h);
        void* d = nullptr;
        e = hipHostGetDevicePointer(&d, h, 0);
        if (e != hipSuccess) {
            destroy_pool(p);
            return fail(SLLM_E_HIP, "hipHostGetDevicePointer failed: %s", hipGetErrorString(e));
        }
        for (uint64_t i = 0; i < k; ++i) {
            p->host.push_back(static_cast<uint8_t*>(h) + i * stride);
            p->mapped.push_back(static_cast<const uint8_t*>(d) + i * stride);
            p->arena_of.push_back((uint32_t)(p->arenas.size() - 1));
        }
        done += k;
    }
    const double t0 = now_s();
    const uint64_t last = n_chunks - (p->arenas.size() - 1) * per_arena;
    prefault(p->arenas, last * stride, per_arena * stride);
    log_msg(2, "pool: %llu x %llu B pinned in %zu arenas, pages touched in %.3f s", (unsigned long long)n_chunks,
            (unsigned long long)stride, p->arenas.size(), now_s() - t0);
    p->free_ids.resize(n_chunks);
    for (uint64_t i = 0; i < n_chunks; ++i) p->free_ids[i] = (uint32_t)(n_chunks - 1 - i);
    *out = p;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_pool_destroy(sllm_pool* p) try {
    clear_error();
    if (!p) return SLLM_OK;
    {
        std::lock_guard<std::mutex> g(p->mu);
        if (p->users) return fail(SLLM_E_BUSY, "pool still used by %d open handle(s)", p->users);
    }
    DeviceGuard guard(p->device);
    destroy_pool(p);
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_pool_query(const sllm_pool* pc, sllm_pool_info* out) try {
    clear_error();
    if (!pc || !out) return fail(SLLM_E_INVAL, "pool and out must be non-NULL");
    auto* p = const_cast<sllm_pool*>(pc);
    std::lock_guard<std::mutex> g(p->mu);
    out->chunk_size = p->chunk;
    out->n_chunks = p->host.size();
    out->free_chunks = p->free_ids.size();
    out->cached_checkpoints = p->cache.size();
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_pool_cache(sllm_pool* p, const char* dir, uint32_t io_threads, uint32_t flags) try {
    Range range_("sllm_pool_cache");
    clear_error();
    if (!p || !dir) return fail(SLLM_E_INVAL, "pool and dir must be non-NULL");
    if (flags & ~SLLM_OPEN_DIRECT_IO) return fail(SLLM_E_INVAL, "unknown flags 0x%x", flags);
    const std::string data_path = std::string(dir) + "/" + kDataName;
    std::string blob;
    IndexData ix;
    SLLM_TRY(read_small_file(std::string(dir) + "/" + kIndexName, &blob));
    SLLM_TRY(decode_index(blob.data(), blob.size(), &ix));
    DataFile f;
    SLLM_TRY(open_data(data_path, (flags & SLLM_OPEN_DIRECT_IO) != 0, &f));
    struct Closer {
        DataFile* f;
        ~Closer() { close_data(f); }
    } closer{&f};
    if (f.size != ix.file_bytes)
        return fail(SLLM_E_FORMAT, "%s is %llu bytes, the index says %llu", data_path.c_str(),
                    (unsigned long long)f.size, (unsigned long long)ix.file_bytes);
    const uint64_t C = p->chunk;
    if (f.direct && (C % f.dio_align || ix.file_bytes % f.dio_align))
        return fail(SLLM_E_INVAL, "direct reads need chunk size %llu to be a multiple of %llu", (unsigned long long)C,
                    (unsigned long long)f.dio_align);
    const uint64_t n = ceil_div(ix.total, C);
    std::vector<uint32_t> ids;
    {
        std::lock_guard<std::mutex> g(p->mu);
        if (pool_find(p, f)) return fail(SLLM_E_BUSY, "%s is already cached", dir);
        SLLM_TRY(pool_take(p, n, &ids));
    }
    auto give_back = [&] {
        std::lock_guard<std::mutex> g(p->mu);
        pool_give(p, ids);
    };
    // read chunk k into its pool chunk; direct reads run to the 4 KiB-padded
    // file end so that their lengths stay block multiples
    const uint64_t read_end = f.direct ? ix.file_bytes : ix.total;
    int32_t st = parallel_chunks(n, io_threads ? io_threads : 4, [&](uint64_t k) {
        const uint64_t off = k * C;
        return read_chunk(f, p->host[ids[k]], std::min(C, read_end - off), off, data_path, nullptr);
    });
    if (st != SLLM_OK) {
        give_back();
        return st;
    }
    const uint8_t** d_table = nullptr;
    st = pool_chunk_table(p, ids, &d_table);
    if (st == SLLM_OK) st = pool_adopt(p, dir, f, ix.total, ids, d_table, 0, nullptr);
    if (st != SLLM_OK) {  // nothing was adopted: the chunks and the table are still ours
        pool_free_table(p, d_table);
        give_back();
        return st;
    }
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_pool_evict(sllm_pool* p, const char* dir) try {
    clear_error();
    if (!p || !dir) return fail(SLLM_E_INVAL, "pool and dir must be non-NULL");
    const std::string canon = canonical_dir(dir);
    struct stat st;
    const bool have = ::stat((std::string(dir) + "/" + kDataName).c_str(), &st) == 0;
    std::lock_guard<std::mutex> g(p->mu);
    for (size_t i = 0; i < p->cache.size(); ++i) {
        CacheEntry& e = *p->cache[i];
        const bool same = have ? (e.dev == (uint64_t)st.st_dev && e.ino == (uint64_t)st.st_ino) : e.dir == canon;
        if (!same) continue;
        if (e.refs) return fail(SLLM_E_BUSY, "%s is loaded by %d open handle(s)", dir, e.refs);
        if (e.d_table) {
            DeviceGuard guard(p->device);
            (void)hipFree(e.d_table);
        }
        pool_give(p, e.chunks);
        p->cache.erase(p->cache.begin() + (long)i);
        return SLLM_OK;
    }
    return fail(SLLM_E_NOTFOUND, "%s is not cached", dir);
} SLLM_CATCH_ALL
