// Pinned host chunk pool: the DRAM tier of Sec. 4.2.  Fixed-size chunks avoid
// fragmentation; the application allocates and frees them explicitly, and
// whole partitions can stay cached in them between loads.
#pragma once

#include <cstdint>
#include <functional>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "format.hpp"
#include "io.hpp"

namespace sllm {

// A partition kept in pool chunks (chunk k of the partition in chunks[k]).
struct CacheEntry {
    std::string dir;
    uint64_t dev = 0, ino = 0, size = 0, mtime_ns = 0;  // identity of the data file
    uint64_t total = 0;                                 // T of the cached partition
    std::vector<uint32_t> chunks;                       // pool chunk ids, partition order
    const uint8_t** d_table = nullptr;                  // device array: mapped address of each chunk
    int refs = 0;                                       // open handles that load from it
};

}  // namespace sllm

struct sllm_pool {
    int device = 0;
    uint64_t chunk = 0;   // usable bytes per chunk
    uint64_t stride = 0;  // distance between chunk starts: align_up(chunk, 4096)
    std::vector<void*> arenas;            // pinned allocations
    std::vector<uint8_t*> host;           // per chunk: host address
    std::vector<const uint8_t*> mapped;   // per chunk: device-visible address
    std::vector<uint32_t> arena_of;       // per chunk: index of the arena holding it
    std::vector<uint32_t> free_ids;
    std::vector<std::unique_ptr<sllm::CacheEntry>> cache;
    int users = 0;                        // open handles attached to the pool
    std::mutex mu;
};

namespace sllm {

// Chunk b's bytes follow chunk a's in one pinned allocation, so one copy can
// read both.  Two arenas may happen to sit back to back in the address
// space, but a copy must not run from one allocation into another.
inline bool pool_follows(const sllm_pool* p, uint32_t a, uint32_t b) {
    return p->stride == p->chunk && p->arena_of[a] == p->arena_of[b] && p->host[b] == p->host[a] + p->chunk;
}

// Take n free chunks (NOMEM if fewer are free) / give them back.
int32_t pool_take(sllm_pool* p, uint64_t n, std::vector<uint32_t>* out);
void pool_give(sllm_pool* p, const std::vector<uint32_t>& ids);

// The cache entry for this data file, or null (caller holds p->mu).
CacheEntry* pool_find(sllm_pool* p, const DataFile& f);

// A device array holding the mapped address of chunk ids[k] at k (null for
// no ids); free it with pool_free_table unless a cache entry adopts it.
int32_t pool_chunk_table(sllm_pool* p, const std::vector<uint32_t>& ids, const uint8_t*** out);
void pool_free_table(sllm_pool* p, const uint8_t** d_table);

// Register chunks `ids` (chunk k of the partition of data file `f` in
// ids[k]) and their device table as the pool's cached copy of checkpoint
// `dir`, with `refs` handles already loading from it.  On success the entry
// owns the chunks and the table (*out, if given, points to it); BUSY if that
// file is cached already, and then nothing is taken.  Caller must not hold
// p->mu.
int32_t pool_adopt(sllm_pool* p, const char* dir, const DataFile& f, uint64_t total, const std::vector<uint32_t>& ids,
                   const uint8_t** d_table, int refs, CacheEntry** out);

// realpath of dir, or dir itself if that fails.
std::string canonical_dir(const char* dir);

}  // namespace sllm

namespace sllm {

// Read a whole (small) file.
int32_t read_small_file(const std::string& path, std::string* out);

// Run fn(k) for every k in [0, n) on `threads` threads (the caller's among
// them), stopping at the first failure.
int32_t parallel_chunks(uint64_t n, uint32_t threads, const std::function<int32_t(uint64_t)>& fn);

}  // namespace sllm
