// Optional per-launch timing (mpq_timing_enable / mpq_timing_only /
// mpq_timing_read): while it is on, every kernel launch of the library (or
// of the one kernel mpq_timing_only names) is bracketed by two events
// recorded on the stream the kernel is launched on, so a kernel that runs on
// one of the library's own streams is timed there.  Off by default; then a
// LaunchTimer does nothing.
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "internal.hpp"
#include "mpq.h"

namespace mpq {

namespace {

struct Record {
    std::string name;
    hipEvent_t start, stop;
};

constexpr size_t kTimingEventPool = 1024;
std::atomic<bool> g_on{false};
std::mutex g_mu;
std::string g_only;               // record only this kernel ("" = every kernel)
std::vector<Record> g_records;
std::vector<hipEvent_t> g_free;   // events for reuse

hipEvent_t take_event()
{
    if (!g_free.empty()) {
        hipEvent_t e = g_free.back();
        g_free.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

LaunchTimer::LaunchTimer(hipStream_t s, const char *name) : s_(s), start_(nullptr)
{
    if (!g_on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_only.empty() && g_only != name) return;
    start_ = take_event();
    if (start_ && hipEventRecord(start_, s) != hipSuccess) {
        g_free.push_back(start_);
        start_ = nullptr;
    }
    name_ = name;
}

LaunchTimer::~LaunchTimer()
{
    if (!start_) return;
    std::lock_guard<std::mutex> lk(g_mu);
    hipEvent_t stop = take_event();
    if (stop && hipEventRecord(stop, s_) == hipSuccess) {
        g_records.push_back(Record{name_, start_, stop});
    } else {
        g_free.push_back(start_);
        if (stop) g_free.push_back(stop);
    }
}

}  // namespace mpq

extern "C" {

int mpq_timing_enable(int on)
{
    std::lock_guard<std::mutex> lk(mpq::g_mu);
    for (auto &r : mpq::g_records) {
        mpq::g_free.push_back(r.start);
        mpq::g_free.push_back(r.stop);
    }
    mpq::g_records.clear();
    // events are created here, not at the launches, so that recording adds
    // no event creation to the enqueue of a timed call
    while (on && mpq::g_free.size() < mpq::kTimingEventPool) {
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) break;
        mpq::g_free.push_back(e);
    }
    mpq::g_on.store(on != 0);
    return MPQ_OK;
}

int mpq_timing_only(const char *name)
{
    if (name && strlen(name) >= sizeof(((mpq_kernel_time *)nullptr)->name)) return MPQ_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lk(mpq::g_mu);
    mpq::g_only = name ? name : "";
    return MPQ_OK;
}

int mpq_timing_read(mpq_kernel_time *out, int cap)
{
    if (cap < 0 || (cap > 0 && !out)) return MPQ_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lk(mpq::g_mu);
    const int n = (int)mpq::g_records.size();
    for (int i = 0; i < n && i < cap; ++i) {
        const auto &r = mpq::g_records[i];
        float ms = -1.0f;
        if (hipEventSynchronize(r.stop) != hipSuccess ||
            hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
            ms = -1.0f;
        snprintf(out[i].name, sizeof out[i].name, "%s", r.name.c_str());
        out[i].ms = ms;
    }
    return n;
}

}  // extern "C"
