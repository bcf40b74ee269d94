// The streamed load's task-queue pipeline (Sec. 4.2): readers fill free
// pinned slots and queue them; the issue loop hands ready chunks to the next
// tier in batches and recycles a batch's slots once that tier is done.
#include "pipeline.hpp"

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <mutex>
#include <string>
#include <thread>

#include "common.hpp"
#include "workers.hpp"

namespace sllm {

int32_t reclaim_batches(BatchSink& sink, std::deque<InFlightBatch>& inflight, std::vector<TraceEvent>* trace,
                        double t_start) {
    for (const InFlightBatch& b : inflight) {
        const int32_t st = sink.done(b.token, true);
        if (st < 0) return st;
        if (trace)
            for (size_t j = 0; j < b.slots.size(); ++j)
                trace->push_back({now_s() - t_start, b.chunks[j], b.slots[j], 0, TraceEvent::kDone});
    }
    inflight.clear();
    return SLLM_OK;
}

int32_t run_stream(const StreamPlan& p, const ChunkReader& read, BatchSink& sink, std::deque<InFlightBatch>& inflight,
                   StreamStats* stats) {
    const uint64_t C = p.chunk, T = p.total;
    const uint64_t n = ceil_div(T, C);
    if (p.n_slots == 0 || p.max_batch == 0 || (p.keep && p.n_slots < n))
        return fail(SLLM_E_INVAL, "stream: %u slots and batches of %u for %llu chunks", p.n_slots, p.max_batch,
                    (unsigned long long)n);

    std::mutex mu;
    std::condition_variable cv_free, cv_ready;
    std::deque<uint32_t> free_q;
    std::deque<ChunkSlot> ready_q;
    if (!p.keep)
        for (uint32_t i = 0; i < p.n_slots; ++i) free_q.push_back(i);
    std::atomic<uint64_t> next{0};
    uint32_t reading = 0;  // slots held by readers
    bool stop = false;
    int32_t err = SLLM_OK;
    std::string err_msg;
    uint64_t bytes_read = 0, bytes_bounced = 0;
    std::atomic<uint64_t> busy_ns{0}, starved_ns{0};
    const double t_start = now_s();
    std::mutex trace_mu;
    auto trace = [&](TraceEvent::Kind kind, uint64_t k, uint32_t slot, uint32_t thread) {
        if (!p.trace) return;
        const double t = now_s() - t_start;
        std::lock_guard<std::mutex> g(trace_mu);
        p.trace->push_back({t, k, slot, thread, kind});
    };

    auto set_error = [&](int32_t st) {  // caller holds mu
        if (err == SLLM_OK) {
            err = st;
            err_msg = sllm_last_error();
        }
        stop = true;
        cv_free.notify_all();
        cv_ready.notify_all();
    };

    // The first split_chunks chunks are read in pieces: the reader that
    // takes such a chunk publishes its other pieces, and readers take open
    // pieces before they start a chunk of their own.  Only the newest split
    // chunk can have pieces nobody took yet.
    struct Split {
        uint64_t k = 0, len = 0, piece = 0;
        uint32_t si = 0, pieces = 0, taken = 0, left = 0;
    };
    std::vector<Split> splits;  // split chunks not yet read completely (guarded by mu)
    auto open_split = [&]() -> Split* {
        return !splits.empty() && splits.back().taken < splits.back().pieces ? &splits.back() : nullptr;
    };
    const uint32_t nt = (uint32_t)std::min<uint64_t>(p.io_threads ? p.io_threads : 1, n);
    auto pieces_of = [&](uint64_t k, uint64_t len, uint64_t* piece) -> uint32_t {
        if (k >= p.split_chunks || nt < 2 || p.split_min == 0) return 1;
        const uint64_t want = std::min<uint64_t>(nt, len / p.split_min);
        if (want < 2) return 1;
        const uint64_t a = std::max<uint64_t>(1, p.split_align);
        *piece = ceil_div(ceil_div(len, want), a) * a;
        return (uint32_t)ceil_div(len, *piece);
    };

    // a reader takes an open piece, else a free slot (with keep: slot k) and
    // then the next chunk number, reads it into the slot and queues the
    // chunk once all of it is read.  Slots go to chunks in chunk order, so a
    // chunk the sink waits for is always being read or already queued: a
    // sink that consumes chunks in order cannot be left waiting for a chunk
    // with every slot held by later ones.
    auto reader = [&](uint32_t thread) {
        for (;;) {
            uint64_t k = 0, off = 0, len = 0;
            uint32_t si = 0;
            bool piece = false;
            {
                const double w0 = now_s();
                std::unique_lock<std::mutex> lk(mu);
                if (!p.keep) {
                    cv_free.wait(lk, [&] { return stop || open_split() || next.load() >= n || !free_q.empty(); });
                    starved_ns += (uint64_t)((now_s() - w0) * 1e9);
                }
                if (stop) return;
                if (Split* sp = open_split()) {
                    k = sp->k;
                    si = sp->si;
                    off = (uint64_t)sp->taken * sp->piece;
                    len = std::min(sp->piece, sp->len - off);
                    ++sp->taken;
                    piece = true;
                } else {
                    if (next.load() >= n) return;
                    k = next.fetch_add(1);
                    if (p.keep) {
                        si = (uint32_t)k;
                    } else {
                        si = free_q.front();
                        free_q.pop_front();
                    }
                    const uint64_t chunk_len = std::min(C, p.read_end - k * C);
                    uint64_t piece_len = 0;
                    const uint32_t np = pieces_of(k, chunk_len, &piece_len);
                    len = chunk_len;
                    if (np > 1) {
                        Split sp;
                        sp.k = k;
                        sp.len = chunk_len;
                        sp.piece = piece_len;
                        sp.si = si;
                        sp.pieces = np;
                        sp.taken = 1;
                        sp.left = np;
                        splits.push_back(sp);
                        len = piece_len;
                        piece = true;
                        cv_free.notify_all();  // idle readers take the other pieces
                    }
                    trace(TraceEvent::kReadBegin, k, si, thread);
                }
                ++reading;
            }
            uint64_t bounced = 0;
            const double r0 = now_s();
            range_push("sllm read chunk");
            const int32_t st = read(k, si, off, len, &bounced);
            range_pop();
            busy_ns += (uint64_t)((now_s() - r0) * 1e9);
            std::lock_guard<std::mutex> g(mu);
            --reading;
            if (st != SLLM_OK) {
                if (!p.keep && !piece) free_q.push_back(si);
                set_error(st);
                return;
            }
            bytes_read += len;
            bytes_bounced += bounced;
            if (piece) {
                auto it = std::find_if(splits.begin(), splits.end(), [&](const Split& x) { return x.k == k; });
                if (--it->left > 0) continue;
                splits.erase(it);
            }
            trace(TraceEvent::kReadEnd, k, si, thread);
            ready_q.push_back({k, si});
            cv_ready.notify_one();
        }
    };


    TaskGroup readers;  // idle threads of earlier loads, else new ones
    if (readers.start(nt, reader) != SLLM_OK) {  // could not start every reader: stop the ones that run
        const std::string why = sllm_last_error();
        {
            std::lock_guard<std::mutex> g(mu);
            stop = true;
            cv_free.notify_all();
        }
        readers.wait();
        sink.drain();
        return fail(SLLM_E_NOMEM, "cannot start %u I/O threads: %s", nt, why.c_str());
    }
    // however this function ends (an exception included), stop the readers
    // before `readers` waits for them, so that none stays blocked on a slot
    struct StopReaders {
        std::function<void()> f;
        ~StopReaders() { f(); }
    } stop_readers{[&] {
        std::lock_guard<std::mutex> g(mu);
        stop = true;
        cv_free.notify_all();
    }};

    // give the slots of completed batches back to the readers; with `block`,
    // wait for the oldest batch first
    auto reclaim = [&](bool block) -> int32_t {
        while (!inflight.empty()) {
            const int32_t d = sink.done(inflight.front().token, block);
            block = false;
            if (d < 0) return d;
            if (d == 0) break;
            for (size_t j = 0; j < inflight.front().slots.size(); ++j)
                trace(TraceEvent::kDone, inflight.front().chunks[j], inflight.front().slots[j], 0);
            if (!p.keep) {  // kept slots are not refilled
                std::lock_guard<std::mutex> g(mu);
                for (uint32_t si : inflight.front().slots) free_q.push_back(si);
            }
            cv_free.notify_all();
            inflight.pop_front();
        }
        return SLLM_OK;
    };
    auto queued_bytes = [&] {
        uint64_t b = 0;
        for (const InFlightBatch& f : inflight) b += f.bytes;
        return b;
    };

    // A short batch is held back while the sink still has at least a full
    // batch's bytes queued and readers are filling slots, so that batches
    // carry about `target` chunks instead of whatever arrived last.
    const uint64_t target = std::max<uint64_t>(1, std::min<uint64_t>(p.target, p.max_batch));
    std::vector<ChunkSlot> batch;
    batch.reserve(p.max_batch);
    double wait_s = 0;
    uint64_t moved = 0, seq = 0;
    int32_t rc = SLLM_OK;
    while (moved < n && rc == SLLM_OK) {
        rc = reclaim(false);
        if (rc != SLLM_OK) break;
        batch.clear();
        bool wait_sink = false;
        {
            const double w0 = now_s();
            std::unique_lock<std::mutex> lk(mu);
            // readers are reading, will take an open piece, or will start on
            // a free slot (a chunk of their own when slots are kept)
            const bool readers_busy =
                reading > 0 || open_split() || (next.load() < n && (p.keep || !free_q.empty()));
            if (ready_q.empty() && !stop) {
                if (!readers_busy && !inflight.empty())
                    wait_sink = true;  // every slot is with the sink
                else
                    cv_ready.wait_for(lk, std::chrono::microseconds(200), [&] { return stop || !ready_q.empty(); });
            }
            const uint64_t fill = std::min<uint64_t>(target, n - moved);
            bool hold = false;
            if (!wait_sink && !stop && ready_q.size() < fill && readers_busy && queued_bytes() >= target * C) {
                cv_ready.wait_for(lk, std::chrono::microseconds(50), [&] { return stop || ready_q.size() >= fill; });
                hold = !stop && ready_q.size() < fill;  // still short: reclaim, then look again
            }
            wait_s += now_s() - w0;
            if (stop && ready_q.empty()) break;  // a reader failed
            while (!hold && !ready_q.empty() && batch.size() < p.max_batch) {
                batch.push_back(ready_q.front());
                ready_q.pop_front();
            }
        }
        if (wait_sink) {
            rc = reclaim(true);
            continue;
        }
        if (batch.empty()) continue;
        std::sort(batch.begin(), batch.end(), [](const ChunkSlot& a, const ChunkSlot& b) { return a.chunk < b.chunk; });
        InFlightBatch f;
        range_push("sllm move batch");
        rc = sink.move(batch.data(), (uint32_t)batch.size(), seq, &f.token);
        range_pop();
        // on error part of the batch may be with the sink: its slots are not
        // handed back (the load stops, drains the sink, and the next load
        // starts from a full free list)
        if (rc == SLLM_OK) {
            for (const ChunkSlot& c : batch) {
                f.slots.push_back(c.slot);
                f.chunks.push_back(c.chunk);
                f.bytes += std::min(C, T - c.chunk * C);
                trace(TraceEvent::kMoved, c.chunk, c.slot, 0);
            }
            inflight.push_back(std::move(f));
        }
        ++seq;
        moved += batch.size();
    }
    {
        // after a complete pass every chunk has been read, so no reader waits
        // for a slot; after an error, stop releases the ones that do
        std::lock_guard<std::mutex> g(mu);
        if (rc != SLLM_OK) set_error(rc);
        stop = true;
        cv_free.notify_all();
    }
    readers.wait();
    if (stats) {
        stats->t_start = t_start;
        stats->bytes_read = bytes_read;
        stats->bytes_bounced = bytes_bounced;
        stats->batches = seq;
        stats->wait_s = wait_s;
        stats->reader_busy_s = (double)busy_ns.load() * 1e-9;
        stats->reader_starved_s = (double)starved_ns.load() * 1e-9;
    }
    if (err != SLLM_OK) {
        sink.drain();  // work a failed move() left behind, and every batch in flight
        inflight.clear();
        return fail(err, "%s", err_msg.c_str());
    }
    return SLLM_OK;
}

}  // namespace sllm
