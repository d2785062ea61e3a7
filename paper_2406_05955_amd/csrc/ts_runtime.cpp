// Error capture and per-kernel event timing (see ts_runtime.h).
#include "ts_runtime.h"

#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

namespace ts {

namespace {
thread_local char g_last_error[256] = "";

struct ProfRecord {
    std::string kernel;
    hipEvent_t start = nullptr, stop = nullptr;
};

std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRecord> g_prof;   // events recorded since the last reset
std::vector<hipEvent_t> g_pool;   // created events available for reuse

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

// Both events of a record, or neither (a half-made pair goes back to the pool).
bool take_pair(ProfRecord &r) {
    r.start = take_event();
    r.stop = take_event();
    if (r.start && r.stop) return true;
    if (r.start) g_pool.push_back(r.start);
    if (r.stop) g_pool.push_back(r.stop);
    return false;
}
}  // namespace

void set_last_error(const char *where, hipError_t e) {
    std::snprintf(g_last_error, sizeof g_last_error, "%s: %s", where, hipGetErrorString(e));
}

void set_last_message(const char *msg) { std::snprintf(g_last_error, sizeof g_last_error, "%s", msg); }

ts_status check_launch(const char *where) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_last_error(where, e);
        return TS_ERR_HIP;
    }
    return TS_OK;
}

bool prof_events(const char *kernel, hipEvent_t *start, hipEvent_t *stop) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof_on) return false;
    ProfRecord r;
    r.kernel = kernel;
    if (!take_pair(r)) return false;
    g_prof.push_back(r);
    *start = r.start;
    *stop = r.stop;
    return true;
}

ProfScope::ProfScope(const char *kernel, hipStream_t stream) : stream_(stream) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof_on) return;
    ProfRecord r;
    r.kernel = kernel;
    if (!take_pair(r)) return;
    if (hipEventRecord(r.start, stream) != hipSuccess) {
        g_pool.push_back(r.start);
        g_pool.push_back(r.stop);
        return;
    }
    g_prof.push_back(r);
    slot_ = (int)g_prof.size() - 1;
}

ProfScope::~ProfScope() {
    if (slot_ < 0) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (slot_ < (int)g_prof.size()) (void)hipEventRecord(g_prof[slot_].stop, stream_);
}

}  // namespace ts

extern "C" {

const char *ts_last_error(void) { return ts::g_last_error; }

void ts_prof_enable(int on) {
    std::lock_guard<std::mutex> lk(ts::g_prof_mu);
    ts::g_prof_on = on != 0;
}

void ts_prof_reset(void) {
    std::lock_guard<std::mutex> lk(ts::g_prof_mu);
    for (auto &r : ts::g_prof) {
        (void)hipEventSynchronize(r.stop);
        ts::g_pool.push_back(r.start);
        ts::g_pool.push_back(r.stop);
    }
    ts::g_prof.clear();
}

ts_status ts_prof_read(const char *kernel, long *launches, double *total_ms) {
    if (!kernel || !launches || !total_ms) return TS_ERR_NULL;
    std::lock_guard<std::mutex> lk(ts::g_prof_mu);
    long n = 0;
    double ms = 0.0;
    for (auto &r : ts::g_prof) {
        if (r.kernel != kernel) continue;
        hipError_t e = hipEventSynchronize(r.stop);
        if (e != hipSuccess) {
            ts::set_last_error("ts_prof_read", e);
            return TS_ERR_HIP;
        }
        float t = 0.f;
        e = hipEventElapsedTime(&t, r.start, r.stop);
        if (e != hipSuccess) {
            ts::set_last_error("ts_prof_read", e);
            return TS_ERR_HIP;
        }
        ++n;
        ms += t;
    }
    *launches = n;
    *total_ms = ms;
    return TS_OK;
}

}  // extern "C"
