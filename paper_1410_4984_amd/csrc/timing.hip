// Optional per-kernel timing for benchmarks: while enabled, every kernel launch
// of the library is bracketed by two HIP events recorded on the launch stream.
// gpps_timing_collect() waits for the recorded events, sums the elapsed times
// per kernel name and releases the events.  Disabled (the default), the scopes
// cost one relaxed atomic load.
#include <hip/hip_runtime.h>

#include <atomic>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

namespace gpps {
namespace {

struct Rec {
    const char *name;
    hipEvent_t start, stop;
};

std::atomic<int> g_enabled{0};
std::mutex g_mu;
std::vector<Rec> g_recs;
std::vector<std::string> g_names;   // storage behind the pointers handed out by collect
bool g_failed = false;

}  // namespace

TimedScope::TimedScope(hipStream_t st, const char *name) : st_(st), name_(name) {
    if (!g_enabled.load(std::memory_order_relaxed)) return;
    if (hipEventCreate(&start_) != hipSuccess) { g_failed = true; return; }
    if (hipEventCreate(&stop_) != hipSuccess) {
        (void)hipEventDestroy(start_);
        g_failed = true;
        return;
    }
    if (hipEventRecord(start_, st_) != hipSuccess) g_failed = true;
    active_ = true;
}

TimedScope::~TimedScope() {
    if (!active_) return;
    if (hipEventRecord(stop_, st_) != hipSuccess) g_failed = true;
    std::lock_guard<std::mutex> lk(g_mu);
    g_recs.push_back(Rec{name_, start_, stop_});
}

}  // namespace gpps

extern "C" {

gpps_status gpps_timing_enable(int on) {
    gpps::g_enabled.store(on ? 1 : 0);
    return GPPS_OK;
}

int gpps_timing_collect(int max_entries, const char **names, double *total_ms,
                        int64_t *launches) {
    using namespace gpps;
    std::lock_guard<std::mutex> lk(g_mu);
    std::map<std::string, std::pair<double, int64_t>> acc;
    bool ok = !g_failed;
    for (const Rec &r : g_recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess ||
            hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
            ok = false;
        auto &a = acc[r.name];
        a.first += ms;
        a.second += 1;
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.stop);
    }
    g_recs.clear();
    g_failed = false;
    if (!ok) return -1;
    g_names.clear();
    for (auto &kv : acc) g_names.push_back(kv.first);
    int n = 0;
    for (auto &kv : acc) {
        if (n >= max_entries) break;
        if (names) names[n] = g_names[n].c_str();
        if (total_ms) total_ms[n] = kv.second.first;
        if (launches) launches[n] = kv.second.second;
        ++n;
    }
    return n;
}

}  // extern "C"
