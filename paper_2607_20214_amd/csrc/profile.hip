// profile.hip -- opt-in per-kernel timing with HIP events.
//
// When enabled (elsaa_profile_enable(1)), every kernel launch of the library
// is bracketed by two events recorded on the launch stream; the elapsed times
// are summed per kernel name when elsaa_profile_get() collects them.  When
// disabled (the default) a launch costs one relaxed atomic load.
#include <atomic>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "elsaa.h"
#include "internal.hpp"

namespace elsaa {

namespace {

struct Pending {
    const char* name;
    hipEvent_t start, stop;
};

struct Stat {
    double ms = 0.0;
    int64_t launches = 0;
};

std::atomic<int> g_on{0};
std::mutex g_mu;
std::vector<hipEvent_t> g_pool;
std::vector<Pending> g_pending;
std::map<std::string, Stat> g_stats;
thread_local Pending t_open{nullptr, nullptr, nullptr};

hipEvent_t take_event()
{
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Collect finished pending launches (blocks until each has completed).
void drain()
{
    for (auto& p : g_pending) {
        float ms = 0.f;
        if (hipEventSynchronize(p.stop) == hipSuccess && hipEventElapsedTime(&ms, p.start, p.stop) == hipSuccess) {
            Stat& s = g_stats[p.name];
            s.ms += ms;
            s.launches += 1;
        }
        g_pool.push_back(p.start);
        g_pool.push_back(p.stop);
    }
    g_pending.clear();
}

}  // namespace

ProfScope::ProfScope(const char* name, hipStream_t st) : stream_(st), active_(false)
{
    if (!g_on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_mu);
    hipEvent_t a = take_event(), b = take_event();
    if (!a || !b) return;
    if (hipEventRecord(a, st) != hipSuccess) return;
    t_open = Pending{name, a, b};
    active_ = true;
}

ProfScope::~ProfScope()
{
    if (!active_) return;
    std::lock_guard<std::mutex> lk(g_mu);
    if (hipEventRecord(t_open.stop, stream_) == hipSuccess) g_pending.push_back(t_open);
    t_open = Pending{nullptr, nullptr, nullptr};
}

}  // namespace elsaa

using namespace elsaa;

extern "C" {

int elsaa_profile_enable(int on)
{
    std::lock_guard<std::mutex> lk(g_mu);
    drain();
    if (on) g_stats.clear();
    g_on.store(on ? 1 : 0);
    return ELSAA_OK;
}

int elsaa_profile_count(void)
{
    std::lock_guard<std::mutex> lk(g_mu);
    drain();
    return (int)g_stats.size();
}

int elsaa_profile_get(int index, char* name, size_t name_len, double* total_ms, int64_t* launches)
{
    std::lock_guard<std::mutex> lk(g_mu);
    drain();
    if (index < 0 || index >= (int)g_stats.size() || !name || name_len == 0 || !total_ms || !launches)
        return ELSAA_ERR_INVALID_ARG;
    auto it = g_stats.begin();
    std::advance(it, index);
    snprintf(name, name_len, "%s", it->first.c_str());
    *total_ms = it->second.ms;
    *launches = it->second.launches;
    return ELSAA_OK;
}

}  // extern "C"
