// Error state, version and the optional per-kernel timing of the library.
#include "common.h"

#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

namespace acsc {
namespace {
thread_local char g_err[512] = {0};

// Per-kernel timing: each launch made while timing is on is bracketed by two
// HIP events recorded on the launch stream; durations are read back (after
// the events complete) when the counters are queried.
struct Pending {
    const char *tag;
    hipEvent_t start, stop;
};
struct Totals {
    int64_t launches = 0;
    double ms = 0.0;
};
std::mutex g_mu;
bool g_on = false;
std::string g_only;   // time only the launches of this kernel name (empty: all)
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
std::map<std::string, Totals> g_totals;

hipEvent_t take_event()
{
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess)
        return nullptr;
    return e;
}

// Fold completed events into the totals (waits for them).  g_mu held.
int drain_locked()
{
    int rc = ACSC_OK;
    for (const Pending &p : g_pending) {
        float ms = 0.f;
        if (hipEventSynchronize(p.stop) != hipSuccess || hipEventElapsedTime(&ms, p.start, p.stop) != hipSuccess)
            rc = ACSC_EHIP;
        Totals &t = g_totals[p.tag];
        t.launches += 1;
        t.ms += ms;
        g_pool.push_back(p.start);
        g_pool.push_back(p.stop);
    }
    g_pending.clear();
    return rc;
}
}  // namespace

int set_error(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_err[0] = '\0'; }

bool stats_on() { return g_on; }

void *stats_begin(hipStream_t st, const char *tag)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_on || (!g_only.empty() && g_only != tag))
        return nullptr;
    if (g_pending.size() >= 8192)
        drain_locked();
    Pending p{tag, take_event(), take_event()};
    if (!p.start || !p.stop || hipEventRecord(p.start, st) != hipSuccess)
        return nullptr;
    g_pending.push_back(p);
    return reinterpret_cast<void *>(static_cast<uintptr_t>(g_pending.size()));
}

// Timing assumes one launching thread between stats_begin and stats_end.
void stats_end(hipStream_t st, void *token)
{
    if (!token)
        return;
    std::lock_guard<std::mutex> lk(g_mu);
    const size_t i = static_cast<size_t>(reinterpret_cast<uintptr_t>(token)) - 1;
    if (i < g_pending.size())
        hipEventRecord(g_pending[i].stop, st);
}

}  // namespace acsc

extern "C" const char *acsc_last_error(void) { return acsc::g_err; }

extern "C" int acsc_version(void) { return 1; }

extern "C" int acsc_stats_enable(int on)
{
    acsc::clear_error();
    std::lock_guard<std::mutex> lk(acsc::g_mu);
    int rc = acsc::drain_locked();
    acsc::g_totals.clear();
    acsc::g_on = on != 0;
    if (rc)
        return acsc::set_error(rc, "an event of a timed launch failed");
    return ACSC_OK;
}

extern "C" int acsc_stats_only(const char *tag)
{
    acsc::clear_error();
    const size_t len = tag ? std::strlen(tag) : 0;
    if (len >= 64)
        return acsc::set_error(ACSC_EINVAL, "kernel name of %zu characters", len);
    std::lock_guard<std::mutex> lk(acsc::g_mu);
    acsc::g_only.assign(tag ? tag : "");
    return ACSC_OK;
}

extern "C" int acsc_stats_read(int index, char *name, size_t name_len, int64_t *launches, double *total_ms)
{
    acsc::clear_error();
    std::lock_guard<std::mutex> lk(acsc::g_mu);
    int rc = acsc::drain_locked();
    if (rc)
        return acsc::set_error(rc, "an event of a timed launch failed");
    if (index < 0 || index >= static_cast<int>(acsc::g_totals.size()))
        return acsc::set_error(ACSC_EINVAL, "no kernel name with index %d", index);
    auto it = acsc::g_totals.begin();
    std::advance(it, index);
    if (name && name_len) {
        std::strncpy(name, it->first.c_str(), name_len - 1);
        name[name_len - 1] = '\0';
    }
    if (launches)
        *launches = it->second.launches;
    if (total_ms)
        *total_ms = it->second.ms;
    return ACSC_OK;
}
