// CPU-only driver for the streamed load's pipeline (csrc/pipeline.cpp), built
// with ThreadSanitizer and with AddressSanitizer by tests/test_sanitize.py.
//
// A CPU sink stands in for the GPU: move() queues a batch for a worker thread
// that, after a random delay, copies each chunk from its ring slot into the
// destination image and marks the batch done.  Readers copy chunks from an
// in-memory "file" with random delays.  Over a few hundred random
// geometries (sizes, chunk sizes, ring sizes, reader counts, batch limits,
// kept slots) and repeated loads it checks that
//   * the destination equals the source bytes [0, T) after every load;
//   * a reader never writes a slot that a batch not yet complete still holds
//     (the slot-recycling rule; ThreadSanitizer checks the same ordering);
//   * an injected read error or move() error is returned with its message,
//     leaves nothing in flight, and the next load on the same sink succeeds;
//   * the optional timeline has every chunk read, moved and done once, in
//     that order, and no slot read again before its previous chunk was done.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <mutex>
#include <random>
#include <string>
#include <thread>
#include <vector>

#include "common.hpp"
#include "pipeline.hpp"
#include "workers.hpp"

using namespace sllm;

namespace {

std::atomic<int> g_violations{0};

void sleep_us(std::mt19937_64& rng, uint32_t max_us) {
    const uint32_t us = (uint32_t)(rng() % (max_us + 1));
    if (us) std::this_thread::sleep_for(std::chrono::microseconds(us));
}

class CpuSink final : public BatchSink {
  public:
    CpuSink(std::vector<uint8_t>& slots, uint64_t stride, uint32_t n_slots, std::vector<uint8_t>& dst, uint64_t C,
            uint64_t T, uint64_t seed)
        : slots_(slots), stride_(stride), dst_(dst), C_(C), T_(T), pending_(n_slots, 0), rng_(seed),
          worker_([this] { run(); }) {}

    ~CpuSink() override {
        {
            std::lock_guard<std::mutex> g(mu_);
            quit_ = true;
        }
        cv_.notify_all();
        worker_.join();
    }

    int32_t move(const ChunkSlot* b, uint32_t n, uint64_t seq, uint64_t* token) override {
        std::lock_guard<std::mutex> g(mu_);
        Job j;
        j.token = ++next_token_;
        for (uint32_t i = 0; i < n; ++i) {
            if (i && b[i].chunk <= b[i - 1].chunk) ++g_violations;  // batches arrive sorted
            if (pending_[b[i].slot]++) ++g_violations;                // a slot in two batches at once
            j.chunks.push_back(b[i]);
        }
        if (fail_seq_ >= 0 && (uint64_t)fail_seq_ == seq) {
            // half the batch was started before the failure: drain() must wait for it
            j.chunks.resize(n / 2);
            for (uint32_t i = n / 2; i < n; ++i) --pending_[b[i].slot];
            q_.push_back(std::move(j));
            cv_.notify_all();
            return fail(SLLM_E_HIP, "injected move failure at batch %llu", (unsigned long long)seq);
        }
        q_.push_back(std::move(j));
        *token = q_.back().token;
        cv_.notify_all();
        return SLLM_OK;
    }

    int32_t done(uint64_t token, bool block) override {
        std::unique_lock<std::mutex> lk(mu_);
        if (block) cv_done_.wait(lk, [&] { return completed_ >= token; });
        return completed_ >= token ? 1 : 0;
    }

    void drain() override {
        std::unique_lock<std::mutex> lk(mu_);
        cv_done_.wait(lk, [&] { return q_.empty() && !busy_; });
    }

    // called by a reader before it writes slot si
    void check_free(uint32_t si) {
        std::lock_guard<std::mutex> g(mu_);
        if (pending_[si]) ++g_violations;
    }

    int fail_seq_ = -1;

  private:
    struct Job {
        uint64_t token = 0;
        std::vector<ChunkSlot> chunks;
    };

    void run() {
        for (;;) {
            Job j;
            {
                std::unique_lock<std::mutex> lk(mu_);
                cv_.wait(lk, [&] { return quit_ || !q_.empty(); });
                if (quit_ && q_.empty()) return;
                j = std::move(q_.front());
                q_.pop_front();
                busy_ = true;
            }
            sleep_us(rng_, 60);
            for (const ChunkSlot& c : j.chunks) {
                const uint64_t off = c.chunk * C_, len = std::min(C_, T_ - off);
                std::memcpy(dst_.data() + off, slots_.data() + (uint64_t)c.slot * stride_, len);
            }
            {
                std::lock_guard<std::mutex> g(mu_);
                for (const ChunkSlot& c : j.chunks) --pending_[c.slot];
                // tokens complete in order (one worker, FIFO); a failed batch
                // never got its token, so the next one may skip it
                if (j.token > completed_) completed_ = j.token;
                busy_ = false;
            }
            cv_done_.notify_all();
        }
    }

    std::vector<uint8_t>& slots_;
    uint64_t stride_;
    std::vector<uint8_t>& dst_;
    uint64_t C_, T_;
    std::vector<int> pending_;
    std::mt19937_64 rng_;
    std::mutex mu_;
    std::condition_variable cv_, cv_done_;
    std::deque<Job> q_;
    uint64_t next_token_ = 0, completed_ = 0;
    bool busy_ = false, quit_ = false;
    std::thread worker_;
};

// The timeline of one clean load: every chunk read, moved and done once, in
// that order, and a slot read again only after the chunk it held was done.
int check_trace(const std::vector<TraceEvent>& tr, uint64_t n, uint32_t n_slots) {
    std::vector<double> t[4];
    for (auto& v : t) v.assign(n, -1);
    std::vector<uint32_t> slot_of(n, 0);
    for (const TraceEvent& e : tr) {
        if (e.chunk >= n || e.kind > 3 || e.slot >= n_slots) return 1;
        if (t[e.kind][e.chunk] >= 0) return 2;  // a step recorded twice
        t[e.kind][e.chunk] = e.t;
        if (e.kind == TraceEvent::kReadBegin) slot_of[e.chunk] = e.slot;
    }
    std::vector<std::vector<std::pair<double, double>>> uses(n_slots);
    for (uint64_t k = 0; k < n; ++k) {
        for (int s = 0; s < 4; ++s)
            if (t[s][k] < 0) return 3;  // a step missing
        if (!(t[0][k] <= t[1][k] && t[1][k] <= t[2][k] && t[2][k] <= t[3][k])) return 4;
        uses[slot_of[k]].push_back({t[0][k], t[3][k]});
    }
    for (auto& u : uses) {
        std::sort(u.begin(), u.end());
        for (size_t i = 1; i < u.size(); ++i)
            if (u[i].first < u[i - 1].second) return 5;  // refilled before its chunk was done
    }
    return 0;
}

struct Case {
    uint64_t T, C;
    uint32_t slots, threads, max_batch;
    uint64_t target;
    bool keep;
    uint64_t split_chunks = 0, split_min = 1, split_align = 1;  // leading chunks read in pieces
    uint64_t tail = 0;  // reads reach tail bytes past T (a direct read's padded end)
};

// A piece must lie inside its chunk and start at a multiple of the alignment.
void check_piece(const Case& cs, uint64_t k, uint64_t off, uint64_t len) {
    const uint64_t chunk_len = std::min(cs.C, cs.T + cs.tail - k * cs.C);
    if (off + len > chunk_len || (off % cs.split_align) != 0 || (off && k >= cs.split_chunks)) ++g_violations;
}

// One sink, several loads: clean ones, then (optionally) one with an
// injected error, then a clean one again.
int run_case(const Case& cs, uint64_t seed, int inject) {
    std::mt19937_64 rng(seed);
    const uint64_t n = ceil_div(cs.T, cs.C);
    std::vector<uint8_t> file(cs.T + cs.tail, 0);  // zero past T, as a padded file
    for (uint64_t i = 0; i < cs.T; ++i) file[i] = (uint8_t)rng();
    const uint32_t n_slots = cs.keep ? (uint32_t)std::max<uint64_t>(n, 1) : cs.slots;
    std::vector<uint8_t> slots((uint64_t)n_slots * cs.C);
    std::vector<uint8_t> dst(cs.T);
    CpuSink sink(slots, cs.C, n_slots, dst, cs.C, cs.T, seed ^ 0x5bd1e995);
    std::deque<InFlightBatch> inflight;
    std::atomic<int64_t> fail_read_at{-1};
    std::mutex rng_mu;
    ChunkReader read = [&](uint64_t k, uint32_t si, uint64_t off, uint64_t len, uint64_t* bounced) -> int32_t {
        uint32_t delay;
        {
            std::lock_guard<std::mutex> g(rng_mu);
            delay = (uint32_t)(rng() % 40);
        }
        if (delay) std::this_thread::sleep_for(std::chrono::microseconds(delay));
        if ((int64_t)k == fail_read_at.load()) return fail(SLLM_E_IO, "injected read error at chunk %llu", (unsigned long long)k);
        if (cs.keep && si != k) ++g_violations;
        check_piece(cs, k, off, len);
        sink.check_free(si);
        std::memcpy(slots.data() + (uint64_t)si * cs.C + off, file.data() + k * cs.C + off, len);
        *bounced += len & 1;
        return SLLM_OK;
    };
    StreamPlan plan;
    plan.chunk = cs.C;
    plan.total = cs.T;
    plan.read_end = cs.T + cs.tail;
    plan.io_threads = cs.threads;
    plan.n_slots = n_slots;
    plan.max_batch = cs.max_batch;
    plan.target = cs.target;
    plan.keep = cs.keep;
    plan.split_chunks = cs.split_chunks;
    plan.split_min = cs.split_min;
    plan.split_align = cs.split_align;
    for (int load = 0; load < 4; ++load) {
        const bool faulty = inject && load == 2 && n > 0;
        if (faulty) {
            if (inject == 1)
                fail_read_at = (int64_t)(rng() % n);
            else
                sink.fail_seq_ = (int)(rng() % std::max<uint64_t>(1, n / std::max<uint32_t>(1, cs.max_batch)));
        }
        std::fill(dst.begin(), dst.end(), 0xEE);
        int32_t st = reclaim_batches(sink, inflight);
        if (st != SLLM_OK) {
            std::printf("reclaim failed: %s\n", sllm_last_error());
            return 1;
        }
        std::vector<TraceEvent> trace;
        plan.trace = faulty || load % 2 ? nullptr : &trace;
        StreamStats ss;
        st = run_stream(plan, read, sink, inflight, &ss);
        if (faulty) {
            fail_read_at = -1;
            sink.fail_seq_ = -1;
            const int32_t want = inject == 1 ? SLLM_E_IO : SLLM_E_HIP;
            // a move() failure at a batch past the last one never fires
            if (st == SLLM_OK && inject == 2) {
                (void)reclaim_batches(sink, inflight);
                continue;
            }
            if (st != want || !std::strstr(sllm_last_error(), "injected") || !inflight.empty()) {
                std::printf("injected error %d: got status %d (%s), %zu batches in flight\n", inject, st,
                            sllm_last_error(), inflight.size());
                return 1;
            }
            continue;
        }
        if (st != SLLM_OK) {
            std::printf("load %d failed: %d %s\n", load, st, sllm_last_error());
            return 1;
        }
        st = reclaim_batches(sink, inflight, plan.trace, ss.t_start);  // the GPU path's stream join
        if (st != SLLM_OK || !inflight.empty()) return 1;
        if (plan.trace) {
            const int bad = check_trace(trace, n, n_slots);
            if (bad) {
                std::printf("load %d: timeline check %d failed (%zu events)\n", load, bad, trace.size());
                return 1;
            }
        }
        const uint64_t want_read = std::min(cs.T + cs.tail, n * cs.C);
        if (ss.bytes_read != want_read) {
            std::printf("read %llu bytes of %llu\n", (unsigned long long)ss.bytes_read, (unsigned long long)want_read);
            return 1;
        }
        if (cs.T && std::memcmp(dst.data(), file.data(), cs.T) != 0) {
            uint64_t bad = 0;
            while (dst[bad] == file[bad]) ++bad;
            std::printf("load %d: image differs at byte %llu\n", load, (unsigned long long)bad);
            return 1;
        }
    }
    return 0;
}

// A sink that consumes chunks strictly in chunk order: its worker waits
// (bounded) for chunk k to be moved before it copies chunk k and marks it
// done.  With slots handed to chunks out of order, every slot could end up
// holding a later chunk while the worker waits for an earlier one; the
// bounded wait then reports it.
class InOrderSink final : public BatchSink {
  public:
    InOrderSink(std::vector<uint8_t>& slots, uint64_t stride, uint32_t n_slots, std::vector<uint8_t>& dst, uint64_t C,
                uint64_t T)
        : slots_(slots), stride_(stride), dst_(dst), C_(C), T_(T), n_(ceil_div(T, C)), slot_of_(n_, 0),
          done_(n_, 0), pending_(n_slots, 0), worker_([this] { run(); }) {}

    ~InOrderSink() override {
        drain();
        worker_.join();
    }

    int32_t move(const ChunkSlot* b, uint32_t n, uint64_t, uint64_t* token) override {
        std::lock_guard<std::mutex> g(mu_);
        for (uint32_t i = 0; i < n; ++i) {
            if (slot_of_[b[i].chunk] || pending_[b[i].slot]++) ++g_violations;
            slot_of_[b[i].chunk] = b[i].slot + 1;
        }
        *token = b[0].chunk;
        cv_.notify_all();
        return SLLM_OK;
    }

    int32_t done(uint64_t k, bool block) override {
        std::unique_lock<std::mutex> lk(mu_);
        if (block) cv_done_.wait(lk, [&] { return done_[k] || finished_; });
        if (done_[k]) return 1;
        if (finished_) return fail(SLLM_E_IO, "in-order sink stopped before chunk %llu", (unsigned long long)k);
        return 0;
    }

    void drain() override {
        std::unique_lock<std::mutex> lk(mu_);
        abort_ = true;
        cv_.notify_all();
        cv_done_.wait(lk, [&] { return finished_; });
    }

    void check_free(uint32_t si) {
        std::lock_guard<std::mutex> g(mu_);
        if (pending_[si]) ++g_violations;
    }

    bool timed_out() {
        std::lock_guard<std::mutex> g(mu_);
        return timed_out_;
    }

  private:
    void run() {
        for (uint64_t k = 0; k < n_; ++k) {
            uint32_t slot;
            {
                std::unique_lock<std::mutex> lk(mu_);
                const bool ok = cv_.wait_for(lk, std::chrono::seconds(5), [&] { return abort_ || slot_of_[k] != 0; });
                if (!ok) timed_out_ = true;
                if (!ok || abort_) break;
                slot = slot_of_[k] - 1;
            }
            const uint64_t off = k * C_, len = std::min(C_, T_ - off);
            std::memcpy(dst_.data() + off, slots_.data() + (uint64_t)slot * stride_, len);
            {
                std::lock_guard<std::mutex> g(mu_);
                --pending_[slot];
                done_[k] = 1;
            }
            cv_done_.notify_all();
        }
        {
            std::lock_guard<std::mutex> g(mu_);
            finished_ = true;
        }
        cv_done_.notify_all();
    }

    std::vector<uint8_t>& slots_;
    uint64_t stride_;
    std::vector<uint8_t>& dst_;
    uint64_t C_, T_, n_;
    std::vector<uint32_t> slot_of_;
    std::vector<uint8_t> done_;
    std::vector<int> pending_;
    std::mutex mu_;
    std::condition_variable cv_, cv_done_;
    bool abort_ = false, finished_ = false, timed_out_ = false;
    std::thread worker_;
};

// Several loads through an in-order sink (a fresh one per load), with one
// chunk per batch.
int run_in_order_case(const Case& cs, uint64_t seed) {
    std::mt19937_64 rng(seed);
    const uint64_t n = ceil_div(cs.T, cs.C);
    if (n == 0) return 0;
    std::vector<uint8_t> file(cs.T);
    for (auto& b : file) b = (uint8_t)rng();
    std::vector<uint8_t> slots((uint64_t)cs.slots * cs.C);
    std::vector<uint8_t> dst(cs.T);
    std::mutex rng_mu;
    for (int load = 0; load < 3; ++load) {
        std::fill(dst.begin(), dst.end(), 0xEE);
        InOrderSink sink(slots, cs.C, cs.slots, dst, cs.C, cs.T);
        ChunkReader read = [&](uint64_t k, uint32_t si, uint64_t off, uint64_t len, uint64_t*) -> int32_t {
            uint32_t delay;
            {
                std::lock_guard<std::mutex> g(rng_mu);
                delay = (uint32_t)(rng() % 200);
            }
            if (delay) std::this_thread::sleep_for(std::chrono::microseconds(delay));
            check_piece(cs, k, off, len);
            sink.check_free(si);
            std::memcpy(slots.data() + (uint64_t)si * cs.C + off, file.data() + k * cs.C + off, len);
            return SLLM_OK;
        };
        StreamPlan plan;
        plan.chunk = cs.C;
        plan.total = cs.T;
        plan.read_end = cs.T;
        plan.io_threads = cs.threads;
        plan.n_slots = cs.slots;
        plan.max_batch = 1;
        plan.target = 1;
        plan.split_chunks = cs.split_chunks;
        plan.split_min = cs.split_min;
        plan.split_align = cs.split_align;
        std::deque<InFlightBatch> inflight;
        StreamStats ss;
        int32_t st = run_stream(plan, read, sink, inflight, &ss);
        if (st == SLLM_OK) st = reclaim_batches(sink, inflight);
        if (st != SLLM_OK || sink.timed_out()) {
            std::printf("in-order load %d: status %d (%s), timed out %d\n", load, st, sllm_last_error(),
                        (int)sink.timed_out());
            return 1;
        }
        if (std::memcmp(dst.data(), file.data(), cs.T) != 0) {
            std::printf("in-order load %d: image differs\n", load);
            return 1;
        }
    }
    return 0;
}

}  // namespace

// Two cases in three read some leading chunks (sometimes all) in pieces.
void random_split(Case& cs, std::mt19937_64& rng) {
    if (rng() % 3 == 0) return;
    cs.split_chunks = rng() % 4 == 0 ? 1000000 : rng() % 6;
    cs.split_min = 1 + rng() % 4;
    const uint64_t aligns[] = {1, 2, 4, 8};
    cs.split_align = aligns[rng() % 4];
}

// Task groups started from several threads at once, as concurrent loads
// start their readers: every task runs exactly once, on a thread of its own
// (all of a group's tasks run at the same time: each waits for the others),
// and the idle list never exceeds its bound.
int check_task_groups(int rounds) {
    std::atomic<int> bad{0};
    auto client = [&](uint64_t seed) {
        std::mt19937_64 rng(seed);
        for (int r = 0; r < rounds; ++r) {
            const uint32_t n = 1 + (uint32_t)(rng() % 24);
            std::vector<std::atomic<int>> ran(n);
            for (auto& x : ran) x = 0;
            std::mutex mu;
            std::condition_variable cv;
            uint32_t arrived = 0;
            TaskGroup g;
            const int32_t st = g.start(n, [&](uint32_t i) {
                ran[i].fetch_add(1);
                std::unique_lock<std::mutex> lk(mu);
                if (++arrived == n) cv.notify_all();
                // a barrier: only threads of their own can all get past it
                if (!cv.wait_for(lk, std::chrono::seconds(20), [&] { return arrived == n; })) bad.fetch_add(1);
            });
            g.wait();
            if (st != SLLM_OK || g.started() != n) bad.fetch_add(1);
            for (auto& x : ran)
                if (x.load() != 1) bad.fetch_add(1);
            if (idle_workers() > kMaxIdleWorkers) bad.fetch_add(1);
        }
    };
    std::vector<std::thread> clients;
    for (uint64_t c = 0; c < 4; ++c) clients.emplace_back(client, 77 + c);
    for (auto& t : clients) t.join();
    if (bad.load()) std::printf("task groups: %d failures\n", bad.load());
    return bad.load() ? 1 : 0;
}

int main(int argc, char** argv) {
    const int n_cases = argc > 1 ? std::atoi(argv[1]) : 300;
    std::mt19937_64 rng(20240114351ull);
    if (check_task_groups(n_cases) != 0) return 1;
    const uint64_t Cs[] = {1, 7, 16, 64, 100, 4096};
    int failures = 0;
    for (int i = 0; i < n_cases; ++i) {
        Case cs;
        cs.C = Cs[rng() % 6];
        cs.T = rng() % 4 == 0 ? rng() % (3 * cs.C + 1) : rng() % (60 * cs.C + 1);
        cs.slots = 1 + (uint32_t)(rng() % 6);
        cs.threads = 1 + (uint32_t)(rng() % 4);
        cs.max_batch = rng() % 3 == 0 ? 1 : 1 + (uint32_t)(rng() % 8);
        cs.target = 1 + rng() % 4;
        cs.keep = rng() % 5 == 0;
        random_split(cs, rng);
        cs.tail = rng() % 4 == 0 ? rng() % (cs.C + 1) : 0;
        const int inject = (int)(i % 3);  // none, read error, move error
        if (run_case(cs, rng(), inject) != 0) {
            std::printf("case %d failed: T=%llu C=%llu slots=%u threads=%u max_batch=%u target=%llu keep=%d inject=%d "
                        "split=%llu/%llu/%llu tail=%llu\n",
                        i, (unsigned long long)cs.T, (unsigned long long)cs.C, cs.slots, cs.threads, cs.max_batch,
                        (unsigned long long)cs.target, (int)cs.keep, inject, (unsigned long long)cs.split_chunks,
                        (unsigned long long)cs.split_min, (unsigned long long)cs.split_align,
                        (unsigned long long)cs.tail);
            ++failures;
            if (failures > 5) break;
        }
    }
    // in-order sinks: small rings, more readers than slots, slow random reads
    for (int i = 0; i < n_cases / 3 && failures <= 5; ++i) {
        Case cs{};
        cs.C = Cs[rng() % 6];
        cs.T = 1 + rng() % (40 * cs.C);
        cs.slots = 1 + (uint32_t)(rng() % 4);
        cs.threads = 1 + (uint32_t)(rng() % 6);
        random_split(cs, rng);
        if (run_in_order_case(cs, rng()) != 0) {
            std::printf("in-order case %d failed: T=%llu C=%llu slots=%u threads=%u split=%llu/%llu/%llu\n", i,
                        (unsigned long long)cs.T, (unsigned long long)cs.C, cs.slots, cs.threads,
                        (unsigned long long)cs.split_chunks, (unsigned long long)cs.split_min,
                        (unsigned long long)cs.split_align);
            ++failures;
        }
    }
    if (g_violations.load()) {
        std::printf("%d slot-recycling violations\n", g_violations.load());
        return 1;
    }
    if (failures) return 1;
    std::printf("ok %d cases\n", n_cases);
    return 0;
}
