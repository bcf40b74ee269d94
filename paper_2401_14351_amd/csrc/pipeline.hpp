// The streamed load's task-queue pipeline (Sec. 4.2, multi-tier loading
// pipeline with intra-tier concurrency): I/O threads read chunks of the
// partition into free pinned slots and queue (chunk, slot) for the next
// tier; an issue loop hands the ready chunks to that tier in batches and
// gives a batch's slots back once the tier reports the batch complete.
//
// Host-only (no HIP): the next tier is a BatchSink.  The loader's sink moves
// batches to the GPU (K1 gather, K1-scatter or copy-engine copies) and
// records one event per batch; the CPU tests plug in a sink that copies on a
// worker thread, so the pipeline's slot recycling runs under ThreadSanitizer
// without a GPU.
#pragma once

#include <cstdint>
#include <deque>
#include <functional>
#include <vector>

namespace sllm {

// Chunk k of the partition, held in ring slot `slot`.
struct ChunkSlot {
    uint64_t chunk;
    uint32_t slot;
};

// The tier after the pinned slots.
class BatchSink {
  public:
    virtual ~BatchSink() = default;
    // Start moving the n chunks of `batch` (sorted by chunk number); `seq`
    // counts the batches of this load.  On success *token names the batch for
    // done().  The slots of the batch must not be refilled before done()
    // reports it complete.
    virtual int32_t move(const ChunkSlot* batch, uint32_t n, uint64_t seq, uint64_t* token) = 0;
    // 1 once the batch's work is complete, 0 while it is not (only when
    // block is false), or a negative status.  With block, wait for it.
    virtual int32_t done(uint64_t token, bool block) = 0;
    // Wait for every piece of work started so far, including that of a
    // move() which failed part-way.
    virtual void drain() = 0;
};

// A batch the sink may still be reading, with the slots it holds.
struct InFlightBatch {
    uint64_t token = 0;
    std::vector<uint32_t> slots;
    std::vector<uint64_t> chunks;  // chunk held by each slot
    uint64_t bytes = 0;  // partition bytes the batch moves
};

// One step of one chunk through the pipeline, for the optional timeline.
struct TraceEvent {
    enum Kind : uint8_t { kReadBegin = 0, kReadEnd = 1, kMoved = 2, kDone = 3 };
    double t;        // seconds since the start of run_stream
    uint64_t chunk;
    uint32_t slot;
    uint32_t thread; // reader index for reads, 0 for the issue loop
    uint8_t kind;
};

struct StreamPlan {
    uint64_t chunk = 0;       // C
    uint64_t total = 0;       // T: chunk k covers [kC, min(kC + C, T))
    uint64_t read_end = 0;    // bytes of the file a chunk read may reach (T, or F for direct reads)
    uint32_t io_threads = 1;  // readers
    uint32_t n_slots = 1;     // ring slots (with keep: one per chunk)
    uint32_t max_batch = 1;   // chunks per move()
    uint64_t target = 1;      // chunks a batch waits to collect while the sink is still busy
    bool keep = false;        // chunk k always uses slot k and slots are never refilled
    // The first split_chunks chunks are read in pieces by all readers
    // together, one chunk after another, so that the next tier gets its first
    // chunk after a fraction of one chunk's read time; later chunks are read
    // whole.  Pieces hold at least split_min bytes and start at multiples of
    // split_align bytes of the chunk (a direct read's alignment).
    uint64_t split_chunks = 0;
    uint64_t split_min = 1;
    uint64_t split_align = 1;
    std::vector<TraceEvent>* trace = nullptr;  // when set, every chunk's steps are appended
};

struct StreamStats {
    double t_start = 0;       // now_s() when run_stream started (origin of the trace)
    uint64_t bytes_read = 0;
    uint64_t bytes_bounced = 0;
    uint64_t batches = 0;
    double wait_s = 0;        // issue loop waiting for readers
    double reader_busy_s = 0;
    double reader_starved_s = 0;
};

// Reads bytes [off, off + len) of chunk k (file offset kC + off) into bytes
// [off, off + len) of slot `slot`; may add to *bounced the bytes it staged
// through a bounce buffer.  A whole chunk is read with off = 0.
using ChunkReader =
    std::function<int32_t(uint64_t k, uint32_t slot, uint64_t off, uint64_t len, uint64_t* bounced)>;

// Wait for every batch still in flight (from an earlier load) and forget it;
// with a trace, append each chunk's kDone at `t` seconds after `t_start`
// (the now_s() value run_stream started at, StreamStats::t_start).
int32_t reclaim_batches(BatchSink& sink, std::deque<InFlightBatch>& inflight,
                        std::vector<TraceEvent>* trace = nullptr, double t_start = 0);

// Stream every chunk of the partition through the ring into the sink.
// Batches still in flight when it returns stay in `inflight` (their slots
// are free again once reclaim_batches has waited for them).  On error the
// readers stop, the sink is drained, `inflight` is cleared and the first
// error is returned with its message.
int32_t run_stream(const StreamPlan& plan, const ChunkReader& read, BatchSink& sink,
                   std::deque<InFlightBatch>& inflight, StreamStats* stats);

}  // namespace sllm
