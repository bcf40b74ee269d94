// Opening a converted checkpoint and loading it into one device buffer
// (Sec. 4.1 direct tensor addressing; Sec. 4.2 multi-tier loading).
//
// Two sources feed a load:
//  * cached: the partition already sits in pool chunks (the DRAM tier); the
//    whole image moves in one K1 launch or in merged SDMA copies.
//  * streamed: the task-queue pipeline of pipeline.cpp.  I/O threads take
//    the next chunk number, read that chunk from the file into a free pinned
//    slot and queue (chunk, slot); the issue loop moves ready chunks to the
//    GPU in batches (GpuSink below: one batch per copy stream in turn, then
//    one event).  A slot is refilled only after its batch's event has fired.
#include <algorithm>
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <mutex>
#include <string_view>
#include <unordered_map>

#include "device_layout.hpp"
#include "hip_util.hpp"
#include "kernels.hpp"
#include "pipeline.hpp"
#include "pool.hpp"

using namespace sllm;

namespace {

struct Slot {
    uint32_t id = 0;                  // pool chunk id
    uint8_t* host = nullptr;
    const uint8_t* mapped = nullptr;  // device-visible address of the same bytes
    hipEvent_t done = nullptr;        // the event of a batch this slot heads
};

}  // namespace

struct sllm_ckpt {
    std::string dir, data_path;
    IndexData ix;
    // name -> position, built at the first lookup by name (keys view the
    // names in ix, which never change after open)
    mutable std::unordered_map<std::string_view, uint32_t> by_name;
    mutable std::once_flag by_name_once;
    int device = 0;
    uint64_t chunk = 0;             // C of this handle's loads
    uint64_t dev_align = 0;         // A2, 0 for the file layout
    std::vector<uint64_t> dev_off;  // offset of each tensor in the device buffer
    uint64_t dev_total = 0;         // bytes a load writes (T or T2)
    sllm_pool* pool = nullptr;
    bool own_pool = false;
    CacheEntry* cached = nullptr;
    DataFile file;
    uint32_t io_threads = 4, n_streams = 2, ring_slots = 8, engine = SLLM_ENGINE_KERNEL, flags = 0;
    std::vector<Slot> slots;
    std::vector<uint32_t> slot_ids;
    std::deque<InFlightBatch> inflight;  // batches of the last streamed load not yet seen done
                                         // (token = the slot whose event ends the batch)
    std::vector<hipStream_t> streams;
    std::vector<hipEvent_t> join_ev;
    hipEvent_t fork_ev = nullptr, t0_ev = nullptr, t1_ev = nullptr;
    // recorded on the caller's stream after each load or repack, so that
    // close waits for device work that ran on such a stream alone (a cached
    // kernel-engine load, a repack) before the pool chunks and tables it
    // reads go back: the events of loads and repacks that may still run, and
    // completed ones for reuse
    mutable std::vector<hipEvent_t> end_evs, end_free;
    bool timed = false;             // t0/t1 bracket the last load
    DeviceLayout layout;            // device tables for A2 layouts
    bool keep = false;              // SLLM_OPEN_CACHE: chunk k streams into slot k, kept afterwards
    const uint8_t** keep_table = nullptr;  // device table of the kept slots, until the pool adopts it
    std::atomic<bool> busy{false};
    sllm_stats stats{};
};

namespace {

// Copy streams outlive the handles that use them.  Creating a handle's
// streams and destroying them again at close costs most of a millisecond,
// as long as a small checkpoint's whole transfer, so a closed handle leaves
// its streams, idle, with their fork/join events here for the next handle
// on the same device.  They live until the process ends.
struct StreamSet {
    int device = 0;
    std::vector<hipStream_t> streams;
    std::vector<hipEvent_t> join_ev;
    hipEvent_t fork_ev = nullptr;
};
constexpr size_t kMaxIdleStreamSets = 32;
std::mutex g_idle_mu;
std::vector<StreamSet> g_idle_sets;

// Take an idle set of n streams of `device`; false if there is none.
bool take_stream_set(int device, uint32_t n, sllm_ckpt* h);

// Park the handle's copy streams (synchronized by the caller); false if the
// list is full or the set is incomplete, and then the caller destroys them.
bool park_stream_set(sllm_ckpt* h);

void release(sllm_ckpt* h) {
    const bool used_hip = !h->streams.empty() || !h->slots.empty() || h->fork_ev || h->t0_ev || h->t1_ev ||
                          !h->end_evs.empty() || !h->end_free.empty() || h->layout.d_off || h->layout.staging;
    if (used_hip) {
        DeviceGuard guard(h->device);
        for (hipEvent_t e : h->end_evs) (void)hipEventSynchronize(e);
        for (hipEvent_t e : h->end_evs) (void)hipEventDestroy(e);
        for (hipEvent_t e : h->end_free) (void)hipEventDestroy(e);
        for (hipStream_t s : h->streams)
            if (s) (void)hipStreamSynchronize(s);
        for (const InFlightBatch& b : h->inflight) (void)hipEventSynchronize(h->slots[b.token].done);
        for (Slot& s : h->slots)
            if (s.done) (void)hipEventDestroy(s.done);
        if (!park_stream_set(h)) {
            for (hipEvent_t e : h->join_ev)
                if (e) (void)hipEventDestroy(e);
            if (h->fork_ev) (void)hipEventDestroy(h->fork_ev);
            for (hipStream_t s : h->streams)
                if (s) (void)hipStreamDestroy(s);
        }
        for (hipEvent_t e : {h->t0_ev, h->t1_ev})
            if (e) (void)hipEventDestroy(e);
        device_layout_free(&h->layout);
    }
    if (h->keep_table) pool_free_table(h->pool, h->keep_table);
    if (h->pool) {
        std::lock_guard<std::mutex> g(h->pool->mu);
        if (!h->slot_ids.empty()) pool_give(h->pool, h->slot_ids);
        if (h->cached) --h->cached->refs;
        --h->pool->users;
    }
    if (h->own_pool) (void)sllm_pool_destroy(h->pool);
    close_data(&h->file);
    delete h;
}

bool take_stream_set(int device, uint32_t n, sllm_ckpt* h) {
    std::lock_guard<std::mutex> g(g_idle_mu);
    for (auto it = g_idle_sets.begin(); it != g_idle_sets.end(); ++it) {
        if (it->device != device || it->streams.size() != n) continue;
        h->streams = std::move(it->streams);
        h->join_ev = std::move(it->join_ev);
        h->fork_ev = it->fork_ev;
        g_idle_sets.erase(it);
        return true;
    }
    return false;
}

bool park_stream_set(sllm_ckpt* h) {
    if (h->streams.empty() || !h->fork_ev || h->join_ev.size() != h->streams.size()) return false;
    for (size_t i = 0; i < h->streams.size(); ++i)
        if (!h->streams[i] || !h->join_ev[i]) return false;
    std::lock_guard<std::mutex> g(g_idle_mu);
    if (g_idle_sets.size() >= kMaxIdleStreamSets) return false;
    StreamSet set;
    set.device = h->device;
    set.streams = std::move(h->streams);
    set.join_ev = std::move(h->join_ev);
    set.fork_ev = h->fork_ev;
    g_idle_sets.push_back(std::move(set));
    h->streams.clear();
    h->join_ev.clear();
    h->fork_ev = nullptr;
    return true;
}

// The copy streams and their fork/join events, taken at the first load that
// needs them (a cached load by the kernel engine runs on the caller's stream
// alone, so opening such a handle creates no HIP objects): an idle set a
// closed handle left, else new ones.
int32_t ensure_streams(sllm_ckpt* h) {
    if (!h->streams.empty()) return SLLM_OK;
    if (take_stream_set(h->device, h->n_streams, h)) return SLLM_OK;
    std::vector<hipStream_t> streams(h->n_streams, nullptr);
    std::vector<hipEvent_t> join_ev(h->n_streams, nullptr);
    hipEvent_t fork_ev = nullptr;
    hipError_t e = hipSuccess;
    for (uint32_t i = 0; i < h->n_streams && e == hipSuccess; ++i) {
        e = hipStreamCreateWithFlags(&streams[i], hipStreamNonBlocking);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&join_ev[i], hipEventDisableTiming);
    }
    if (e == hipSuccess) e = hipEventCreateWithFlags(&fork_ev, hipEventDisableTiming);
    if (e != hipSuccess) {
        // all or nothing: a handle left with a null stream would queue its
        // copies on the device's null stream at the next load
        for (hipEvent_t ev : join_ev)
            if (ev) (void)hipEventDestroy(ev);
        for (hipStream_t s : streams)
            if (s) (void)hipStreamDestroy(s);
        return fail(SLLM_E_HIP, "creating %u copy streams: %s", h->n_streams, hipGetErrorString(e));
    }
    h->streams = std::move(streams);
    h->join_ev = std::move(join_ev);
    h->fork_ev = fork_ev;
    return SLLM_OK;
}

// Record an end event on `s` after a load's or repack's work (events of
// earlier ones that have completed are reused).
int32_t mark_end(const sllm_ckpt* h, hipStream_t s) {
    for (size_t i = 0; i < h->end_evs.size();) {
        if (hipEventQuery(h->end_evs[i]) == hipSuccess) {
            h->end_free.push_back(h->end_evs[i]);
            h->end_evs[i] = h->end_evs.back();
            h->end_evs.pop_back();
        } else {
            ++i;
        }
    }
    (void)hipGetLastError();  // a query of pending work is not an error
    hipEvent_t e = nullptr;
    if (!h->end_free.empty()) {
        e = h->end_free.back();
    } else {
        SLLM_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
        h->end_free.push_back(e);
    }
    SLLM_HIP(hipEventRecord(e, s));
    h->end_free.pop_back();
    h->end_evs.push_back(e);
    return SLLM_OK;
}

// Make the copy streams wait for work already queued on `user`.
int32_t fork_streams(sllm_ckpt* h, hipStream_t user) {
    SLLM_HIP(hipEventRecord(h->fork_ev, user));
    for (hipStream_t s : h->streams) SLLM_HIP(hipStreamWaitEvent(s, h->fork_ev, 0));
    return SLLM_OK;
}

// Make `user` wait for everything queued on the copy streams.
int32_t join_streams(sllm_ckpt* h, hipStream_t user) {
    for (size_t i = 0; i < h->streams.size(); ++i) {
        SLLM_HIP(hipEventRecord(h->join_ev[i], h->streams[i]));
        SLLM_HIP(hipStreamWaitEvent(user, h->join_ev[i], 0));
    }
    return SLLM_OK;
}

// [p, p + bytes) must be device memory of `device` inside one allocation: a
// kernel or copy that wrote to a host address or past an allocation would
// fault the GPU instead of failing the call.
int32_t check_device_range(const void* p, uint64_t bytes, int device, const char* what) {
    if (!bytes) return SLLM_OK;
    hipPointerAttribute_t at{};
    if (hipPointerGetAttributes(&at, p) != hipSuccess) {
        (void)hipGetLastError();  // leave no error behind for later launch checks
        return fail(SLLM_E_INVAL, "%s %p is not device memory", what, p);
    }
    if (at.type != hipMemoryTypeDevice && at.type != hipMemoryTypeManaged)
        return fail(SLLM_E_INVAL, "%s %p is not device memory", what, p);
    if (at.type == hipMemoryTypeDevice && at.device != device)
        return fail(SLLM_E_INVAL, "%s is memory of device %d, not of the handle's device %d", what, at.device, device);
    void* base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void*>(p)) != hipSuccess || !base) {
        // no allocation range known (e.g. managed memory): the call cannot
        // show that the whole range is inside one allocation, so refuse it
        (void)hipGetLastError();
        return fail(SLLM_E_INVAL, "%s %p: the runtime reports no allocation range for it; pass memory from hipMalloc",
                    what, p);
    }
    const uint64_t off = (uint64_t)(static_cast<const uint8_t*>(p) - static_cast<const uint8_t*>(base));
    if (bytes > size || off > size - bytes)
        return fail(SLLM_E_RANGE, "%s: %llu bytes from %p run past the end of its allocation", what,
                    (unsigned long long)bytes, p);
    return SLLM_OK;
}

// Largest merged copy of a cached partition (SLLM_SDMA_MAX_COPY_MB, default
// 256), read at every load so that one process can compare sizes.
uint64_t sdma_max_copy() {
    const char* s = std::getenv("SLLM_SDMA_MAX_COPY_MB");
    const long mb = s ? std::strtol(s, nullptr, 10) : 0;
    return (mb > 0 ? (uint64_t)mb : 256ull) << 20;
}

// Move one chunk (partition bytes [x0, x0 + len)) from a pinned slot to the
// device on stream s, in the handle's device layout.
int32_t move_chunk(sllm_ckpt* h, uint8_t* dst, uint64_t k, const uint8_t* host, const uint8_t* mapped, uint64_t len,
                   uint32_t si, hipStream_t s) {
    const uint64_t x0 = k * h->chunk;
    if (h->dev_align) {
        if (h->engine == SLLM_ENGINE_KERNEL)
            return launch_scatter_window(h->layout, dst, mapped, x0, x0 + len, /*src_is_host=*/true, s);
        // SDMA into this stream's HBM staging chunk, then repack on the same stream
        uint8_t* stage = h->layout.staging + (uint64_t)si * h->layout.staging_stride;
        SLLM_HIP(hipMemcpyAsync(stage, host, len, hipMemcpyHostToDevice, s));
        return launch_scatter_window(h->layout, dst, stage, x0, x0 + len, /*src_is_host=*/false, s);
    }
    if (h->engine == SLLM_ENGINE_SDMA) {
        SLLM_HIP(hipMemcpyAsync(dst + x0, host, len, hipMemcpyHostToDevice, s));
        return SLLM_OK;
    }
    GatherLaunch g;
    g.dst = dst;
    g.single = mapped;
    g.chunk = h->chunk;
    g.total = h->ix.total;
    g.first_chunk = k;
    g.n_chunks = 1;
    return launch_gather(g, s);
}

int32_t load_cached(sllm_ckpt* h, uint8_t* dst, hipStream_t user) {
    CacheEntry* e = h->cached;
    sllm_pool* p = h->pool;
    const uint64_t C = h->chunk, T = h->ix.total, n = e->chunks.size();
    h->stats.n_chunks = n;
    h->stats.from_cache = 1;
    if (h->engine == SLLM_ENGINE_KERNEL) {
        h->stats.n_launches = 1;
        if (h->dev_align) return launch_scatter_table(h->layout, dst, e->d_table, C, user);
        GatherLaunch g;
        g.dst = dst;
        g.table = e->d_table;
        g.chunk = C;
        g.total = T;
        g.first_chunk = 0;
        g.n_chunks = n;
        return launch_gather(g, user);
    }
    SLLM_TRY(ensure_streams(h));
    SLLM_TRY(fork_streams(h, user));
    // merge chunks that follow each other in one pinned arena into one copy;
    // with a device layout a merged run goes to this stream's HBM staging
    // chunk and one scatter launch repacks it
    const uint64_t max_copy = h->dev_align ? h->layout.staging_stride : std::max(sdma_max_copy(), C);
    uint64_t issued = 0;
    for (uint64_t k = 0; k < n;) {
        uint64_t j = k + 1;
        while (j < n && pool_follows(p, e->chunks[j - 1], e->chunks[j]) && (j + 1 - k) * C <= max_copy) ++j;
        const uint64_t x0 = k * C, x1 = std::min(j * C, T);
        const uint32_t si = (uint32_t)(issued % h->streams.size());
        hipStream_t s = h->streams[si];
        if (h->dev_align) {
            uint8_t* stage = h->layout.staging + (uint64_t)si * h->layout.staging_stride;
            SLLM_HIP(hipMemcpyAsync(stage, p->host[e->chunks[k]], x1 - x0, hipMemcpyHostToDevice, s));
            SLLM_TRY(launch_scatter_window(h->layout, dst, stage, x0, x1, /*src_is_host=*/false, s));
        } else {
            SLLM_HIP(hipMemcpyAsync(dst + x0, p->host[e->chunks[k]], x1 - x0, hipMemcpyHostToDevice, s));
        }
        ++issued;
        k = j;
    }
    h->stats.n_launches = issued;
    return join_streams(h, user);
}

// Bytes a streamed gather batch waits to collect (SLLM_BATCH_TARGET_MB,
// default 64; 0 launches whatever is ready).
uint64_t batch_target_bytes() {
    constexpr uint64_t kDefault = 64ull << 20;
    const char* s = std::getenv("SLLM_BATCH_TARGET_MB");
    if (!s || !*s) return kDefault;
    char* end = nullptr;
    const long v = std::strtol(s, &end, 10);
    return (end && *end == '\0' && v >= 0) ? (uint64_t)v << 20 : kDefault;
}

// Leading chunks of a streamed load read in pieces (SLLM_SPLIT_CHUNKS;
// default: as many as there are I/O threads).
uint64_t split_chunks(uint32_t io_threads) {
    const char* s = std::getenv("SLLM_SPLIT_CHUNKS");
    if (!s || !*s) return io_threads;
    char* end = nullptr;
    const long v = std::strtol(s, &end, 10);
    return (end && *end == '\0' && v >= 0) ? (uint64_t)v : io_threads;
}

// After a successful streamed load with kept slots, hand them to the pool as
// its cached copy of the checkpoint; the handle then loads from the cache.
// If another handle cached the same file meanwhile, the slots stay with this
// handle and its loads keep streaming.
void adopt_kept(sllm_ckpt* h) {
    CacheEntry* e = nullptr;
    if (pool_adopt(h->pool, h->dir.c_str(), h->file, h->ix.total, h->slot_ids, h->keep_table, 1, &e) != SLLM_OK) {
        log_msg(1, "%s was cached by another handle; this one keeps streaming", h->dir.c_str());
        clear_error();
        return;
    }
    h->cached = e;
    h->slot_ids.clear();  // owned by the cache entry now
    h->keep_table = nullptr;
    h->keep = false;
}

// The GPU side of a streamed load.  Batch `seq` goes to copy stream
// seq mod S: the kernel engine moves the batch in one batched gather (file
// layout) or one K1-scatter launch per run of consecutive chunks (device
// layout); the copy engines take one copy per run of consecutive chunks
// whose slots follow each other in one pinned arena (slots are handed out
// in order, so runs are common), or, with a device layout, one chunk per batch through
// the stream's HBM staging chunk and K2.  The event of the batch's first
// slot, recorded after its work on the same stream, ends the batch.
class GpuSink final : public BatchSink {
  public:
    GpuSink(sllm_ckpt* h, uint8_t* dst, uint32_t max_batch) : h_(h), dst_(dst), max_batch_(max_batch) {}

    int32_t move(const ChunkSlot* b, uint32_t n, uint64_t seq, uint64_t* token) override {
        const uint64_t C = h_->chunk, T = h_->ix.total;
        const uint32_t si = (uint32_t)(seq % h_->streams.size());
        hipStream_t st = h_->streams[si];
        if (max_batch_ > 1 && h_->dev_align) {
            const uint8_t* srcs[kScatterBatch];
            for (uint32_t b0 = 0; b0 < n;) {
                uint32_t b1 = b0 + 1;
                while (b1 < n && b[b1].chunk == b[b1 - 1].chunk + 1) ++b1;
                for (uint32_t j = b0; j < b1; ++j) srcs[j - b0] = h_->slots[b[j].slot].mapped;
                ++calls;
                SLLM_TRY(launch_scatter_run(h_->layout, dst_, srcs, b[b0].chunk, b1 - b0, C, st));
                b0 = b1;
            }
        } else if (max_batch_ > 1 && h_->engine == SLLM_ENGINE_SDMA) {
            for (uint32_t b0 = 0; b0 < n;) {
                uint32_t b1 = b0 + 1;
                while (b1 < n && b[b1].chunk == b[b1 - 1].chunk + 1 &&
                       pool_follows(h_->pool, h_->slots[b[b1 - 1].slot].id, h_->slots[b[b1].slot].id))
                    ++b1;
                const uint64_t x0 = b[b0].chunk * C, x1 = std::min(b[b1 - 1].chunk * C + C, T);
                ++calls;
                SLLM_HIP(hipMemcpyAsync(dst_ + x0, h_->slots[b[b0].slot].host, x1 - x0, hipMemcpyHostToDevice, st));
                b0 = b1;
            }
        } else if (max_batch_ > 1) {
            const uint8_t* srcs[kGatherBatch];
            uint64_t ks[kGatherBatch];
            for (uint32_t j = 0; j < n; ++j) {
                srcs[j] = h_->slots[b[j].slot].mapped;
                ks[j] = b[j].chunk;
            }
            ++calls;
            SLLM_TRY(launch_gather_batch(dst_, srcs, ks, n, C, T, st));
        } else {
            const Slot& s0 = h_->slots[b[0].slot];
            ++calls;
            SLLM_TRY(move_chunk(h_, dst_, b[0].chunk, s0.host, s0.mapped, std::min(C, T - b[0].chunk * C), si, st));
        }
        SLLM_HIP(hipEventRecord(h_->slots[b[0].slot].done, st));
        *token = b[0].slot;
        return SLLM_OK;
    }

    int32_t done(uint64_t token, bool block) override {
        hipEvent_t ev = h_->slots[token].done;
        const hipError_t e = block ? hipEventSynchronize(ev) : hipEventQuery(ev);
        if (e == hipErrorNotReady) return 0;
        if (e != hipSuccess) return fail(SLLM_E_HIP, "waiting for a batch: %s", hipGetErrorString(e));
        return 1;
    }

    void drain() override {
        for (hipStream_t s : h_->streams) (void)hipStreamSynchronize(s);
    }

    uint64_t calls = 0;  // kernel launches and copy calls

  private:
    sllm_ckpt* h_;
    uint8_t* dst_;
    uint32_t max_batch_;
};

// With SLLM_TRACE_FILE set, each streamed load appends its pipeline
// timeline to that file as CSV (load, t_s, event, chunk, slot, thread):
// read_begin / read_end per chunk on its reader thread, moved when the issue
// loop hands the chunk's batch to the GPU, done when the loop sees the
// batch's event complete.  Tracing makes the load wait for its last batches.
const char* trace_path() {
    const char* s = std::getenv("SLLM_TRACE_FILE");
    return s && *s ? s : nullptr;
}

void write_trace(const char* path, std::vector<TraceEvent>& tr) {
    static std::atomic<uint64_t> loads{0};
    const uint64_t id = loads.fetch_add(1);
    std::sort(tr.begin(), tr.end(), [](const TraceEvent& a, const TraceEvent& b) { return a.t < b.t; });
    FILE* f = std::fopen(path, "a");
    if (!f) {
        log_msg(1, "cannot open trace file %s", path);
        return;
    }
    std::fseek(f, 0, SEEK_END);
    if (std::ftell(f) == 0) std::fprintf(f, "load,t_s,event,chunk,slot,thread\n");
    static const char* kNames[] = {"read_begin", "read_end", "moved", "done"};
    for (const TraceEvent& e : tr)
        std::fprintf(f, "%llu,%.7f,%s,%llu,%u,%u\n", (unsigned long long)id, e.t, kNames[e.kind],
                     (unsigned long long)e.chunk, e.slot, e.thread);
    std::fclose(f);
}

int32_t load_streamed(sllm_ckpt* h, uint8_t* dst, hipStream_t user) {
    const uint64_t C = h->chunk, T = h->ix.total;
    h->stats.n_chunks = ceil_div(T, C);
    SLLM_TRY(ensure_streams(h));
    // kernel loads in the file layout move every chunk that is ready in one
    // batched gather, device layouts one scatter per run of consecutive
    // chunks, the copy engines one copy per run of adjacent slots (one chunk
    // per batch with a device layout).  A batch's slots come back together,
    // so a batch holds at most a quarter of the ring: four batches can be on
    // the GPU while readers refill the rest.
    const uint32_t quarter = std::max<uint32_t>(1, (uint32_t)h->slots.size() / 4);
    const uint32_t max_batch = h->engine == SLLM_ENGINE_KERNEL
                                   ? std::min<uint32_t>(h->dev_align ? kScatterBatch : kGatherBatch, quarter)
                                   : h->dev_align ? 1 : std::min<uint32_t>(kGatherBatch, quarter);
    GpuSink sink(h, dst, max_batch);
    SLLM_TRY(reclaim_batches(sink, h->inflight));
    SLLM_TRY(fork_streams(h, user));

    StreamPlan plan;
    plan.chunk = C;
    plan.total = T;
    plan.read_end = h->file.direct ? h->ix.file_bytes : T;
    plan.io_threads = h->io_threads;
    plan.n_slots = (uint32_t)h->slots.size();
    plan.max_batch = max_batch;
    plan.target = std::max<uint64_t>(1, batch_target_bytes() / C);
    plan.keep = h->keep;
    // the first chunks are read in pieces of at least 1 MiB by all readers
    // together (SLLM_SPLIT_CHUNKS of them, default one per reader; 0 reads
    // every chunk whole), aligned for direct reads
    plan.split_chunks = split_chunks(h->io_threads);
    plan.split_min = 1ull << 20;
    plan.split_align = h->file.direct ? std::max<uint64_t>(h->file.dio_align, 4096) : 4096;
    auto read = [h](uint64_t k, uint32_t si, uint64_t off, uint64_t len, uint64_t* bounced) {
        return read_chunk(h->file, h->slots[si].host + off, len, k * h->chunk + off, h->data_path, bounced);
    };
    std::vector<TraceEvent> trace;
    const char* tpath = trace_path();
    if (tpath) plan.trace = &trace;
    StreamStats ss;
    const int32_t st = run_stream(plan, read, sink, h->inflight, &ss);
    h->stats.read_wait_s = ss.wait_s;
    h->stats.bytes_read = ss.bytes_read;
    h->stats.bytes_bounced = ss.bytes_bounced;
    h->stats.n_launches = sink.calls;
    h->stats.reader_busy_s = ss.reader_busy_s;
    h->stats.reader_starved_s = ss.reader_starved_s;
    if (st != SLLM_OK) return st;
    if (tpath) {
        SLLM_TRY(reclaim_batches(sink, h->inflight, &trace, ss.t_start));
        write_trace(tpath, trace);
    }
    SLLM_TRY(join_streams(h, user));
    if (h->keep) adopt_kept(h);
    return SLLM_OK;
}

}  // namespace

extern "C" int32_t sllm_open(const char* dir, const sllm_open_opts* opts, sllm_ckpt** out) try {
    Range range_("sllm_open");
    clear_error();
    const double t0 = now_s();
    if (!dir || !out) return fail(SLLM_E_INVAL, "dir and out must be non-NULL");
    *out = nullptr;
    sllm_open_opts o{};
    if (opts) o = *opts;
    if (o.engine != SLLM_ENGINE_KERNEL && o.engine != SLLM_ENGINE_SDMA) return fail(SLLM_E_INVAL, "unknown engine %u", o.engine);
    if (o.flags & ~(SLLM_OPEN_DIRECT_IO | SLLM_OPEN_TIMING | SLLM_OPEN_INDEX_ONLY | SLLM_OPEN_CACHE))
        return fail(SLLM_E_INVAL, "unknown flags 0x%x", o.flags);
    if ((o.flags & SLLM_OPEN_CACHE) && (!o.pool || (o.flags & SLLM_OPEN_INDEX_ONLY)))
        return fail(SLLM_E_INVAL, "SLLM_OPEN_CACHE needs a pool and a data file");
    if (o.dev_alignment && (!is_pow2(o.dev_alignment) || o.dev_alignment < 16))
        return fail(SLLM_E_INVAL, "device alignment %llu is not a power of two >= 16", (unsigned long long)o.dev_alignment);
    if (o.pool && o.pool->device != o.device)
        return fail(SLLM_E_INVAL, "pool belongs to device %d, not %d", o.pool->device, o.device);

    auto* h = new (std::nothrow) sllm_ckpt;
    if (!h) return fail(SLLM_E_NOMEM, "out of host memory");
    h->dir = dir;
    h->data_path = std::string(dir) + "/" + kDataName;
    h->device = o.device;
    h->io_threads = o.io_threads ? o.io_threads : 4;
    h->n_streams = o.n_streams ? o.n_streams : 2;
    h->ring_slots = o.ring_slots ? o.ring_slots : 2 * h->io_threads;
    h->engine = o.engine;
    h->flags = o.flags;
    h->dev_align = o.dev_alignment;
    auto bail = [&](int32_t st) {
        std::string msg = sllm_last_error();
        release(h);
        return fail(st, "%s", msg.c_str());
    };

    std::string blob;
    int32_t st = read_small_file(std::string(dir) + "/" + kIndexName, &blob);
    if (st == SLLM_OK) st = decode_index(blob.data(), blob.size(), &h->ix);
    if (st != SLLM_OK) return bail(st);
    const bool index_only = (o.flags & SLLM_OPEN_INDEX_ONLY) != 0;
    if (!index_only) st = open_data(h->data_path, (o.flags & SLLM_OPEN_DIRECT_IO) != 0, &h->file);
    if (st != SLLM_OK) return bail(st);
    if (!index_only && h->file.size != h->ix.file_bytes) {
        fail(SLLM_E_FORMAT, "%s is %llu bytes, the index says %llu", h->data_path.c_str(),
             (unsigned long long)h->file.size, (unsigned long long)h->ix.file_bytes);
        return bail(SLLM_E_FORMAT);
    }

    // device layout: the file offsets, or the closed form at A2
    const size_t nt = h->ix.tensors.size();
    h->dev_off.resize(nt);
    if (h->dev_align) {
        std::vector<uint64_t> sizes(nt);
        for (size_t i = 0; i < nt; ++i) sizes[i] = h->ix.tensors[i].nbytes;
        st = plan_layout(sizes.data(), nt, h->dev_align, h->dev_off.data(), &h->dev_total);
        if (st != SLLM_OK) return bail(st);
    } else {
        for (size_t i = 0; i < nt; ++i) h->dev_off[i] = h->ix.tensors[i].offset;
        h->dev_total = h->ix.total;
    }

    if (index_only) {
        h->stats.device_ms = -1;
        h->stats.open_s = now_s() - t0;
        *out = h;
        return SLLM_OK;
    }

    // the chunk pool: a shared one (maybe caching this partition) or a private ring
    if (o.pool) {
        h->pool = o.pool;
        {
            std::lock_guard<std::mutex> g(h->pool->mu);
            ++h->pool->users;
            h->cached = pool_find(h->pool, h->file);
            if (h->cached) ++h->cached->refs;
            h->chunk = h->cached ? h->pool->chunk : (o.chunk_size ? o.chunk_size : h->pool->chunk);
            h->keep = !h->cached && (o.flags & SLLM_OPEN_CACHE);
            if ((h->cached || h->keep) && o.chunk_size && o.chunk_size != h->pool->chunk)
                st = fail(SLLM_E_INVAL, "cached partitions use the pool's chunk size %llu", (unsigned long long)h->pool->chunk);
            else if (h->chunk > h->pool->chunk)
                st = fail(SLLM_E_INVAL, "chunk size %llu exceeds the pool's %llu", (unsigned long long)h->chunk,
                          (unsigned long long)h->pool->chunk);
            else if (h->keep)  // one chunk of the pool per chunk of the partition
                st = pool_take(h->pool, ceil_div(h->ix.total, h->chunk), &h->slot_ids);
            else if (!h->cached)
                st = pool_take(h->pool, h->ring_slots, &h->slot_ids);
        }
        if (st != SLLM_OK) return bail(st);
    } else {
        h->chunk = o.chunk_size ? o.chunk_size : h->ix.chunk_size;
        st = sllm_pool_create(h->chunk, h->ring_slots, h->device, &h->pool);
        if (st != SLLM_OK) return bail(st);
        h->own_pool = true;
        {
            std::lock_guard<std::mutex> g(h->pool->mu);
            ++h->pool->users;
            st = pool_take(h->pool, h->ring_slots, &h->slot_ids);
        }
        if (st != SLLM_OK) return bail(st);
    }
    // direct reads run to the 4 KiB-padded file end, so every read's offset
    // and length must be multiples of the file's direct-I/O alignment
    if (!h->cached && h->file.direct && (h->chunk % h->file.dio_align || h->ix.file_bytes % h->file.dio_align)) {
        fail(SLLM_E_INVAL, "direct reads need chunk size %llu and file size %llu to be multiples of %llu",
             (unsigned long long)h->chunk, (unsigned long long)h->ix.file_bytes, (unsigned long long)h->file.dio_align);
        return bail(SLLM_E_INVAL);
    }

    DeviceGuard guard(h->device);
    if (!guard.ok()) {
        fail(SLLM_E_HIP, "cannot make device %d current", h->device);
        return bail(SLLM_E_HIP);
    }
    auto hip_ok = [&](hipError_t e, const char* what) {
        if (e == hipSuccess) return true;
        fail(SLLM_E_HIP, "%s failed: %s", what, hipGetErrorString(e));
        return false;
    };
    if ((o.flags & SLLM_OPEN_TIMING) &&
        (!hip_ok(hipEventCreate(&h->t0_ev), "hipEventCreate") || !hip_ok(hipEventCreate(&h->t1_ev), "hipEventCreate")))
        return bail(SLLM_E_HIP);
    h->slots.resize(h->slot_ids.size());
    for (size_t i = 0; i < h->slot_ids.size(); ++i) {
        Slot& s = h->slots[i];
        s.id = h->slot_ids[i];
        s.host = h->pool->host[s.id];
        s.mapped = h->pool->mapped[s.id];
        if (!hip_ok(hipEventCreateWithFlags(&s.done, hipEventDisableTiming), "hipEventCreateWithFlags")) return bail(SLLM_E_HIP);
    }
    if (h->keep) {
        st = pool_chunk_table(h->pool, h->slot_ids, &h->keep_table);
        if (st != SLLM_OK) return bail(st);
    }
    if (h->dev_align) {
        std::vector<uint64_t> file_off(nt), sizes(nt);
        for (size_t i = 0; i < nt; ++i) {
            file_off[i] = h->ix.tensors[i].offset;
            sizes[i] = h->ix.tensors[i].nbytes;
        }
        // copy-engine loads stage in HBM: one chunk per stream when streaming,
        // merged runs of up to 64 MiB when the partition is cached
        const uint64_t staging = (h->engine == SLLM_ENGINE_SDMA) ? h->n_streams : 0;
        const uint64_t stage_bytes = h->cached ? std::max<uint64_t>(h->chunk, 64ull << 20) : h->chunk;
        st = device_layout_build(file_off, sizes, h->dev_off, h->ix.total, h->dev_total, h->dev_align, staging,
                                 stage_bytes, &h->layout);
        if (st != SLLM_OK) return bail(st);
    }
    h->stats.io_threads = h->io_threads;
    h->stats.engine = h->engine;
    h->stats.direct_io = h->file.direct ? 1 : 0;
    h->stats.device_ms = -1;
    h->stats.open_s = now_s() - t0;
    *out = h;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" uint64_t sllm_total_bytes(const sllm_ckpt* h) { return h ? h->dev_total : 0; }

extern "C" int32_t sllm_load(sllm_ckpt* h, void* dev_dst, uint64_t dst_bytes, void* stream) try {
    Range range_("sllm_load");
    clear_error();
    if (!h) return fail(SLLM_E_INVAL, "handle is NULL");
    if (h->busy.exchange(true)) return fail(SLLM_E_BUSY, "a load is already running on this handle");
    struct Unbusy {
        std::atomic<bool>* b;
        ~Unbusy() { b->store(false); }
    } unbusy{&h->busy};
    if (h->flags & SLLM_OPEN_INDEX_ONLY) return fail(SLLM_E_INVAL, "the handle was opened for its index only");
    if (!dev_dst && h->dev_total) return fail(SLLM_E_INVAL, "destination is NULL");
    if (reinterpret_cast<uintptr_t>(dev_dst) % 16) return fail(SLLM_E_INVAL, "destination is not 16-byte aligned");
    if (dst_bytes < h->dev_total)
        return fail(SLLM_E_RANGE, "destination holds %llu bytes, the checkpoint needs %llu", (unsigned long long)dst_bytes,
                    (unsigned long long)h->dev_total);
    DeviceGuard guard(h->device);
    if (!guard.ok()) return fail(SLLM_E_HIP, "cannot make device %d current", h->device);
    SLLM_TRY(check_device_range(dev_dst, h->dev_total, h->device, "destination"));
    hipStream_t user = static_cast<hipStream_t>(stream);
    const double t0 = now_s();
    h->stats.bytes_loaded = 0;
    h->stats.bytes_read = 0;
    h->stats.n_chunks = 0;
    h->stats.n_launches = 0;
    h->stats.from_cache = 0;
    h->stats.read_wait_s = 0;
    h->stats.bytes_bounced = 0;
    h->stats.reader_busy_s = 0;
    h->stats.reader_starved_s = 0;
    h->stats.device_ms = -1;
    h->timed = false;
    const bool timing = (h->flags & SLLM_OPEN_TIMING) != 0;
    if (timing) SLLM_HIP(hipEventRecord(h->t0_ev, user));
    int32_t st = SLLM_OK;
    if (h->dev_total) {
        uint8_t* dst = static_cast<uint8_t*>(dev_dst);
        st = h->cached ? load_cached(h, dst, user) : load_streamed(h, dst, user);
    }
    if (st != SLLM_OK) {
        // a load that failed part way may have queued copies or launches
        // before the failing call: let them finish, so that the caller may
        // free the destination as soon as the error is returned (the copy
        // streams are the handle's own, invisible to the caller's allocator)
        for (hipStream_t s : h->streams) (void)hipStreamSynchronize(s);
        (void)hipStreamSynchronize(user);
        return st;
    }
    if (h->dev_total) {
        st = mark_end(h, user);
        if (st != SLLM_OK) {
            (void)hipStreamSynchronize(user);
            return st;
        }
    }
    if (timing) {
        SLLM_HIP(hipEventRecord(h->t1_ev, user));
        h->timed = true;
    }
    h->stats.bytes_loaded = h->dev_total;
    h->stats.load_s = now_s() - t0;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_repack(const sllm_ckpt* h, const void* src_dev, uint64_t src_bytes, void* dst_dev,
                               uint64_t dst_bytes, void* stream) try {
    Range range_("sllm_repack");
    clear_error();
    if (!h) return fail(SLLM_E_INVAL, "handle is NULL");
    if (!h->dev_align) return fail(SLLM_E_INVAL, "the handle was opened without a device alignment");
    if (h->flags & SLLM_OPEN_INDEX_ONLY) return fail(SLLM_E_INVAL, "the handle was opened for its index only");
    if (src_bytes < h->ix.total || dst_bytes < h->dev_total)
        return fail(SLLM_E_RANGE, "repack needs %llu source and %llu destination bytes", (unsigned long long)h->ix.total,
                    (unsigned long long)h->dev_total);
    if ((reinterpret_cast<uintptr_t>(src_dev) | reinterpret_cast<uintptr_t>(dst_dev)) % 16)
        return fail(SLLM_E_INVAL, "buffers must be 16-byte aligned");
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(src_dev), d0 = reinterpret_cast<uintptr_t>(dst_dev);
    if (h->ix.total && h->dev_total && s0 < d0 + h->dev_total && d0 < s0 + h->ix.total)
        return fail(SLLM_E_INVAL, "source and destination overlap");
    if (!h->dev_total) return SLLM_OK;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return fail(SLLM_E_HIP, "cannot make device %d current", h->device);
    SLLM_TRY(check_device_range(src_dev, h->ix.total, h->device, "source"));
    SLLM_TRY(check_device_range(dst_dev, h->dev_total, h->device, "destination"));
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint8_t* dst = static_cast<uint8_t*>(dst_dev);
    SLLM_TRY(launch_scatter_window(h->layout, dst, static_cast<const uint8_t*>(src_dev), 0, h->ix.total,
                                   /*src_is_host=*/false, s));
    return mark_end(h, s);
} SLLM_CATCH_ALL

extern "C" int32_t sllm_repack_noalloc(const sllm_ckpt* h, uint64_t dev_alignment, const void* src_dev,
                                       uint64_t src_bytes, void* dst_dev, uint64_t dst_bytes, void* stream) try {
    clear_error();
    if (!h) return fail(SLLM_E_INVAL, "handle is NULL");
    const uint64_t a2 = dev_alignment ? dev_alignment : h->dev_align;
    if (!a2) return fail(SLLM_E_INVAL, "no device alignment: pass one or open the handle with one");
    if (!is_pow2(a2) || a2 < 16)
        return fail(SLLM_E_INVAL, "device alignment %llu is not a power of two >= 16", (unsigned long long)a2);
    const uint64_t n = h->ix.tensors.size();
    if (n > kNoAllocMaxTensors)
        return fail(SLLM_E_RANGE, "%llu tensors exceed the %llu the allocation-free repack holds", (unsigned long long)n,
                    (unsigned long long)kNoAllocMaxTensors);
    uint64_t t2 = 0;  // T2 = sum align_up(s_i, A2), without a host table
    for (const TensorRec& t : h->ix.tensors) {
        uint64_t padded = 0;
        if (!align_up(t.nbytes, a2, &padded) || !add_ok(t2, padded, &t2))
            return fail(SLLM_E_RANGE, "the device layout overflows 64 bits");
    }
    const uint64_t total = h->ix.total;
    if (src_bytes < total || dst_bytes < t2)
        return fail(SLLM_E_RANGE, "repack needs %llu source and %llu destination bytes", (unsigned long long)total,
                    (unsigned long long)t2);
    if ((reinterpret_cast<uintptr_t>(src_dev) | reinterpret_cast<uintptr_t>(dst_dev)) % 16)
        return fail(SLLM_E_INVAL, "buffers must be 16-byte aligned");
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(src_dev), d0 = reinterpret_cast<uintptr_t>(dst_dev);
    if (total && t2 && s0 < d0 + t2 && d0 < s0 + total) return fail(SLLM_E_INVAL, "source and destination overlap");
    if (!t2) return SLLM_OK;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return fail(SLLM_E_HIP, "cannot make device %d current", h->device);
    SLLM_TRY(check_device_range(src_dev, total, h->device, "source"));
    SLLM_TRY(check_device_range(dst_dev, t2, h->device, "destination"));
    return repack_noalloc(h->ix, h->device, a2, t2, static_cast<const uint8_t*>(src_dev), static_cast<uint8_t*>(dst_dev),
                          static_cast<hipStream_t>(stream));
} SLLM_CATCH_ALL

namespace {

void fill_info(const sllm_ckpt* h, uint32_t i, sllm_tensor_info* out) {
    const TensorRec& t = h->ix.tensors[i];
    std::memset(out, 0, sizeof *out);
    out->name = h->ix.name(i);
    out->dtype = t.dtype;
    out->ndim = t.ndim;
    for (uint32_t d = 0; d < t.ndim; ++d) out->shape[d] = t.shape[d];
    out->offset = h->dev_off[i];
    out->nbytes = t.nbytes;
}

}  // namespace

extern "C" int32_t sllm_tensor_index(const sllm_ckpt* h, sllm_tensor_info* out, uint64_t cap, uint64_t* n_total) try {
    clear_error();
    if (!h) return fail(SLLM_E_INVAL, "handle is NULL");
    if (cap && !out) return fail(SLLM_E_INVAL, "out is NULL");
    const uint64_t n = h->ix.tensors.size();
    if (n_total) *n_total = n;
    for (uint64_t i = 0; i < std::min(cap, n); ++i) fill_info(h, (uint32_t)i, &out[i]);
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_tensor_find(const sllm_ckpt* h, const char* name, sllm_tensor_info* out) try {
    clear_error();
    if (!h || !name || !out) return fail(SLLM_E_INVAL, "handle, name and out must be non-NULL");
    std::call_once(h->by_name_once, [h] {
        h->by_name.reserve(h->ix.tensors.size() * 2);
        for (uint32_t i = 0; i < h->ix.tensors.size(); ++i) h->by_name.emplace(h->ix.name_view(i), i);
    });
    auto it = h->by_name.find(std::string_view(name));
    if (it == h->by_name.end()) return fail(SLLM_E_NOTFOUND, "no tensor named '%s'", name);
    fill_info(h, it->second, out);
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_get_stats(const sllm_ckpt* hc, sllm_stats* out) try {
    clear_error();
    if (!hc || !out) return fail(SLLM_E_INVAL, "handle and out must be non-NULL");
    auto* h = const_cast<sllm_ckpt*>(hc);
    if (h->timed) {
        DeviceGuard guard(h->device);
        float ms = 0;
        SLLM_HIP(hipEventSynchronize(h->t1_ev));
        SLLM_HIP(hipEventElapsedTime(&ms, h->t0_ev, h->t1_ev));
        h->stats.device_ms = ms;
    }
    *out = h->stats;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_close(sllm_ckpt* h) try {
    Range range_("sllm_close");
    clear_error();
    if (!h) return SLLM_OK;
    if (h->busy.load()) return fail(SLLM_E_BUSY, "a load is running on this handle");
    release(h);
    return SLLM_OK;
} SLLM_CATCH_ALL
