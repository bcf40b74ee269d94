// Loading-time estimator of Sec. 6: q + n / b per server, with b the
// slowest tier's bandwidth and b refined from measured loads.  Host-only.
#include <algorithm>
#include <cmath>
#include <deque>
#include <mutex>

#include "common.hpp"

struct sllm_estimator {
    double bw[2] = {0, 0};  // bytes/s: [0] DRAM -> HBM, [1] storage -> DRAM
    double weight = 0.5;
    struct Task {
        uint64_t id;
        uint64_t bytes;
        uint32_t tiers;
        double cost_s;  // n / b when it was queued
    };
    std::deque<Task> queue;
    uint64_t next_id = 1;
    mutable std::mutex mu;
};

using namespace sllm;

namespace {

bool tiers_ok(uint32_t tiers) { return tiers && !(tiers & ~(SLLM_TIER_DRAM | SLLM_TIER_STORAGE)); }

// index of the slowest tier the load crosses
int slowest(const sllm_estimator* e, uint32_t tiers) {
    const bool dram = tiers & SLLM_TIER_DRAM, storage = tiers & SLLM_TIER_STORAGE;
    if (dram && storage) return e->bw[1] < e->bw[0] ? 1 : 0;
    return storage ? 1 : 0;
}

double queued_s(const sllm_estimator* e) {
    double q = 0;
    for (const auto& t : e->queue) q += t.cost_s;
    return q;
}

}  // namespace

extern "C" int32_t sllm_estimator_create(double dram_bps, double storage_bps, double weight, sllm_estimator** out) try {
    clear_error();
    if (!out) return fail(SLLM_E_INVAL, "out is NULL");
    *out = nullptr;
    if (!(dram_bps > 0) || !(storage_bps > 0) || !std::isfinite(dram_bps) || !std::isfinite(storage_bps))
        return fail(SLLM_E_INVAL, "bandwidths must be positive");
    if (!(weight > 0 && weight <= 1)) return fail(SLLM_E_INVAL, "weight must be in (0, 1]");
    auto* e = new (std::nothrow) sllm_estimator;
    if (!e) return fail(SLLM_E_NOMEM, "out of host memory");
    e->bw[0] = dram_bps;
    e->bw[1] = storage_bps;
    e->weight = weight;
    *out = e;
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" void sllm_estimator_destroy(sllm_estimator* e) { delete e; }

extern "C" int32_t sllm_estimator_query(const sllm_estimator* e, uint64_t bytes, uint32_t tiers, double* eta_s) try {
    clear_error();
    if (!e || !eta_s) return fail(SLLM_E_INVAL, "estimator and eta_s must be non-NULL");
    if (!tiers_ok(tiers)) return fail(SLLM_E_INVAL, "unknown tiers 0x%x", tiers);
    std::lock_guard<std::mutex> g(e->mu);
    *eta_s = queued_s(e) + (double)bytes / e->bw[slowest(e, tiers)];
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_estimator_enqueue(sllm_estimator* e, uint64_t bytes, uint32_t tiers, uint64_t* task,
                                          double* eta_s) try {
    clear_error();
    if (!e || !task || !eta_s) return fail(SLLM_E_INVAL, "estimator, task and eta_s must be non-NULL");
    if (!tiers_ok(tiers)) return fail(SLLM_E_INVAL, "unknown tiers 0x%x", tiers);
    std::lock_guard<std::mutex> g(e->mu);
    const double cost = (double)bytes / e->bw[slowest(e, tiers)];
    *eta_s = queued_s(e) + cost;
    *task = e->next_id++;
    e->queue.push_back({*task, bytes, tiers, cost});
    return SLLM_OK;
} SLLM_CATCH_ALL

extern "C" int32_t sllm_estimator_complete(sllm_estimator* e, uint64_t task, double seconds) try {
    clear_error();
    if (!e) return fail(SLLM_E_INVAL, "estimator is NULL");
    if (!(seconds > 0) || !std::isfinite(seconds)) return fail(SLLM_E_INVAL, "seconds must be positive");
    std::lock_guard<std::mutex> g(e->mu);
    for (auto it = e->queue.begin(); it != e->queue.end(); ++it) {
        if (it->id != task) continue;
        const int k = slowest(e, it->tiers);
        const double sample = (double)it->bytes / seconds;
        if (it->bytes) e->bw[k] = (1 - e->weight) * e->bw[k] + e->weight * sample;
        e->queue.erase(it);
        return SLLM_OK;
    }
    return fail(SLLM_E_NOTFOUND, "no queued task %llu", (unsigned long long)task);
} SLLM_CATCH_ALL

extern "C" int32_t sllm_estimator_complete_load(sllm_estimator* e, uint64_t task, const sllm_ckpt* h) try {
    clear_error();
    if (!e || !h) return fail(SLLM_E_INVAL, "estimator and handle must be non-NULL");
    sllm_stats st{};
    SLLM_TRY(sllm_get_stats(h, &st));
    if (st.bytes_loaded == 0) return fail(SLLM_E_INVAL, "the handle has not loaded anything");
    // the host-side call covers the reads; with timing the device events
    // cover the copies or kernels that finish after it returns
    const double seconds = st.open_s + std::max(st.load_s, st.device_ms >= 0 ? st.device_ms * 1e-3 : 0.0);
    return sllm_estimator_complete(e, task, seconds);
} SLLM_CATCH_ALL

extern "C" int32_t sllm_estimator_bandwidth(const sllm_estimator* e, uint32_t tier, double* bps) try {
    clear_error();
    if (!e || !bps) return fail(SLLM_E_INVAL, "estimator and out must be non-NULL");
    if (tier != SLLM_TIER_DRAM && tier != SLLM_TIER_STORAGE) return fail(SLLM_E_INVAL, "unknown tier %u", tier);
    std::lock_guard<std::mutex> g(e->mu);
    *bps = e->bw[tier == SLLM_TIER_DRAM ? 0 : 1];
    return SLLM_OK;
} SLLM_CATCH_ALL
