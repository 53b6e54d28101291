// timing.cpp -- opt-in per-kernel timing with hipEvents recorded on the launch
// stream around each kernel (measurement support; off by default, and no
// events are created while it is off).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdio>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"
#include "ssm_adjoint.h"

namespace ssmk {
namespace {

struct Rec {
    const char* name;
    hipEvent_t a;
    hipEvent_t b;
};

std::atomic<bool> g_on{false};
std::mutex g_mu;
std::vector<Rec> g_recs;

}  // namespace

bool timing_enabled() { return g_on.load(std::memory_order_relaxed); }

TimedScope::TimedScope(const char* name, hipStream_t s) : on_(timing_enabled()), s_(s) {
    if (!on_) return;
    Rec r{name, nullptr, nullptr};
    if (hipEventCreate(&r.a) != hipSuccess || hipEventCreate(&r.b) != hipSuccess) {
        on_ = false;
        return;
    }
    (void)hipEventRecord(r.a, s_);
    std::lock_guard<std::mutex> lk(g_mu);
    idx_ = g_recs.size();
    g_recs.push_back(r);
}

TimedScope::~TimedScope() {
    if (!on_) return;
    std::lock_guard<std::mutex> lk(g_mu);
    (void)hipEventRecord(g_recs[idx_].b, s_);
}

}  // namespace ssmk

extern "C" {

ssm_status ssm_timing_enable(int32_t on) {
    ssmk::g_on.store(on != 0);
    return SSM_OK;
}

ssm_status ssm_timing_summary(char* buf, size_t len) {
    if (!buf || len == 0) return SSM_ERR_NULL;
    std::vector<ssmk::Rec> recs;
    {
        std::lock_guard<std::mutex> lk(ssmk::g_mu);
        recs.swap(ssmk::g_recs);
    }
    std::map<std::string, std::pair<long long, double>> agg;
    ssm_status st = SSM_OK;
    for (auto& r : recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess)
            st = SSM_ERR_HIP;
        auto& e = agg[r.name];
        e.first += 1;
        e.second += ms;
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
    }
    std::string out;
    char line[256];
    for (auto& kv : agg) {
        std::snprintf(line, sizeof line, "%s %lld %.6f\n", kv.first.c_str(), kv.second.first, kv.second.second);
        out += line;
    }
    std::snprintf(buf, len, "%s", out.c_str());
    return out.size() + 1 > len ? SSM_ERR_SHAPE : st;
}

}  // extern "C"
