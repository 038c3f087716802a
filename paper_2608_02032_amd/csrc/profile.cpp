// profile.cpp -- optional kernel timing with HIP events (dart_profile_* in
// dart.h).  Off by default; when on, every launch (or only the launches of the
// kernel named by the filter) is bracketed by two events recorded on the
// launch stream, and flush() turns them into per-kernel totals.  The totals
// are shared by all threads under one mutex; the event opened by prof_begin
// belongs to the launching thread, so concurrent launches from several
// threads pair their own events.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "dart.h"
#include "dart_internal.hpp"

namespace {

struct Entry {
    std::string name;
    double ms = 0.0;
    int64_t launches = 0;
};
struct Pending {
    int entry;
    hipEvent_t start, stop;
};

std::mutex g_mu;
std::atomic<bool> g_on{false};
std::string g_filter;  // empty: every kernel
std::vector<Entry> g_entries;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_free;
thread_local int g_open_entry = -1;
thread_local hipEvent_t g_open_start = nullptr;

hipEvent_t take_event() {
    if (!g_free.empty()) {
        hipEvent_t e = g_free.back();
        g_free.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

int entry_for(const char* name) {
    for (size_t i = 0; i < g_entries.size(); ++i)
        if (g_entries[i].name == name) return (int)i;
    g_entries.push_back(Entry{name, 0.0, 0});
    return (int)g_entries.size() - 1;
}

}  // namespace

namespace dart {

void prof_begin(const char* kernel, hipStream_t st) {
    if (!g_on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_filter.empty() && g_filter != kernel) return;
    hipEvent_t e = take_event();
    if (!e) return;
    (void)hipEventRecord(e, st);
    g_open_entry = entry_for(kernel);
    g_open_start = e;
}

void prof_end(hipStream_t st) {
    if (!g_on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_open_start) return;
    hipEvent_t e = take_event();
    if (!e) return;
    (void)hipEventRecord(e, st);
    g_pending.push_back(Pending{g_open_entry, g_open_start, e});
    g_open_start = nullptr;
    g_open_entry = -1;
}

}  // namespace dart

extern "C" {

dart_status dart_profile_enable(int enable) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_on.store(enable != 0);
    return DART_OK;
}

dart_status dart_profile_filter(const char* kernel) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_filter = kernel ? kernel : "";
    return DART_OK;
}

dart_status dart_profile_flush(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    dart_status st = DART_OK;
    for (const Pending& p : g_pending) {
        float ms = 0.f;
        if (hipEventSynchronize(p.stop) != hipSuccess ||
            hipEventElapsedTime(&ms, p.start, p.stop) != hipSuccess) {
            st = DART_ERR_HIP;
        } else {
            g_entries[p.entry].ms += ms;
            g_entries[p.entry].launches += 1;
        }
        g_free.push_back(p.start);
        g_free.push_back(p.stop);
    }
    g_pending.clear();
    return st;
}

int dart_profile_count(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    return (int)g_entries.size();
}

const char* dart_profile_name(int index) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (index < 0 || index >= (int)g_entries.size()) return nullptr;
    return g_entries[index].name.c_str();
}

double dart_profile_total_ms(int index) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (index < 0 || index >= (int)g_entries.size()) return 0.0;
    return g_entries[index].ms;
}

int64_t dart_profile_launches(int index) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (index < 0 || index >= (int)g_entries.size()) return 0;
    return g_entries[index].launches;
}

void dart_profile_reset(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    for (const Pending& p : g_pending) {
        (void)hipEventSynchronize(p.stop);
        g_free.push_back(p.start);
        g_free.push_back(p.stop);
    }
    g_pending.clear();
    for (hipEvent_t e : g_free) (void)hipEventDestroy(e);
    g_free.clear();
    g_entries.clear();
    g_filter.clear();
}

}  // extern "C"
