// dstd_profile.hip -- opt-in per-kernel timing of the library's launches.
//
// When enabled, every kernel launch of the library is bracketed by two
// hipEvents recorded on the launch stream; dstd_profile_collect() waits for
// the pending events and folds them into per-kernel totals. Disabled (the
// default) it costs one atomic load per launch. Not for use while a stream
// is being captured into a graph.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/dstd_lif.h"
#include "dstd_profile.h"

namespace dstd {
namespace {

struct Pending { const char *name; hipEvent_t a, b; };
struct Entry { std::string name; int64_t launches; double ms; };

std::atomic<int> g_on{0};
std::mutex g_mu;
std::vector<Pending> g_pending;
std::vector<Entry> g_entries;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

ProfScope::ProfScope(const char *name, hipStream_t st) : name_(name), st_(st) {
    if (!g_on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_mu);
    a_ = take_event();
    b_ = take_event();
    if (a_ && b_) hipEventRecord(a_, st_);
}

ProfScope::~ProfScope() {
    if (!a_ || !b_) return;
    hipEventRecord(b_, st_);
    std::lock_guard<std::mutex> lk(g_mu);
    g_pending.push_back({name_, a_, b_});
}

}  // namespace dstd

using namespace dstd;

extern "C" {

int32_t dstd_profile_enable(int32_t on) {
    int prev = g_on.exchange(on ? 1 : 0);
    return prev;
}

dstd_status dstd_profile_collect(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    for (auto &p : g_pending) {
        float ms = 0.f;
        if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
            bool found = false;
            for (auto &e : g_entries)
                if (e.name == p.name) {
                    e.launches += 1;
                    e.ms += ms;
                    found = true;
                    break;
                }
            if (!found) g_entries.push_back({p.name, 1, static_cast<double>(ms)});
        }
        g_pool.push_back(p.a);
        g_pool.push_back(p.b);
    }
    g_pending.clear();
    return DSTD_OK;
}

int32_t dstd_profile_count(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    return static_cast<int32_t>(g_entries.size());
}

dstd_status dstd_profile_entry(int32_t idx, const char **name, int64_t *launches, double *total_ms) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (idx < 0 || idx >= static_cast<int32_t>(g_entries.size())) return DSTD_ERR_PARAM;
    if (!name || !launches || !total_ms) return DSTD_ERR_NULL;
    *name = g_entries[idx].name.c_str();
    *launches = g_entries[idx].launches;
    *total_ms = g_entries[idx].ms;
    return DSTD_OK;
}

void dstd_profile_reset(void) {
    dstd_profile_collect();
    std::lock_guard<std::mutex> lk(g_mu);
    g_entries.clear();
}

}  // extern "C"
