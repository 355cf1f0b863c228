// Per-kernel timing with HIP events (diagnostics).  While enabled, each
// kernel launch of encode/rank is bracketed by two events recorded on the
// call's stream; reading synchronises them and sums durations per name.
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "upr_profile.h"

namespace upr {

namespace {

struct Record {
    std::string name;
    hipEvent_t start, stop;
};

struct Profiler {
    std::mutex mu;
    bool enabled = false;
    std::vector<Record> live;          // recorded, not yet read
    std::vector<hipEvent_t> pool;      // reusable events
};

Profiler& prof() {
    static Profiler p;
    return p;
}

hipEvent_t take_event(Profiler& p) {
    if (!p.pool.empty()) {
        hipEvent_t e = p.pool.back();
        p.pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

ProfScope::ProfScope(const char* name, hipStream_t s) : stream_(s) {
    Profiler& p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    if (!p.enabled) return;
    hipEvent_t a = take_event(p), b = take_event(p);
    if (!a || !b) return;
    if (hipEventRecord(a, s) != hipSuccess) return;
    p.live.push_back(Record{name, a, b});
    index_ = (int64_t)p.live.size() - 1;
}

ProfScope::~ProfScope() {
    if (index_ < 0) return;
    Profiler& p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    if (index_ < (int64_t)p.live.size()) (void)hipEventRecord(p.live[index_].stop, stream_);
}

}  // namespace upr

extern "C" {

upr_status upr_profile_enable(int32_t enable) {
    upr::Profiler& p = upr::prof();
    std::lock_guard<std::mutex> lk(p.mu);
    for (auto& r : p.live) {
        (void)hipEventSynchronize(r.stop);
        p.pool.push_back(r.start);
        p.pool.push_back(r.stop);
    }
    p.live.clear();
    p.enabled = enable != 0;
    return UPR_OK;
}

int32_t upr_profile_read(upr_kernel_stat* out, int32_t max_entries) {
    upr::Profiler& p = upr::prof();
    std::lock_guard<std::mutex> lk(p.mu);
    std::vector<upr_kernel_stat> agg;
    for (auto& r : p.live) {
        float ms = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess) continue;
        if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) continue;
        upr_kernel_stat* hit = nullptr;
        for (auto& a : agg)
            if (std::strncmp(a.name, r.name.c_str(), sizeof(a.name)) == 0) hit = &a;
        if (!hit) {
            agg.push_back(upr_kernel_stat{});
            hit = &agg.back();
            std::strncpy(hit->name, r.name.c_str(), sizeof(hit->name) - 1);
        }
        hit->launches += 1;
        hit->total_ms += ms;
    }
    const int32_t n = (int32_t)agg.size();
    for (int32_t i = 0; i < n && i < max_entries && out; ++i) out[i] = agg[i];
    return n;
}

}  // extern "C"
