// Optional per-kernel timing: when enabled, every kernel the library launches
// is bracketed by two HIP events recorded on its stream.  Reading the totals
// waits for those events and sums the elapsed times per kernel name.
#include <hip/hip_runtime.h>

#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"

namespace ordermoe {
namespace {

struct Pending {
    std::string name;
    hipEvent_t a, b;
};
struct Total {
    double ms = 0.0;
    int64_t launches = 0;
};

std::mutex g_mu;
bool g_on = false;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
std::map<std::string, Total> g_totals;

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

// moves finished launches into the totals; waits for them if `wait`
int drain(bool wait) {
    std::vector<Pending> keep;
    for (auto& p : g_pending) {
        if (!wait && hipEventQuery(p.b) == hipErrorNotReady) { keep.push_back(p); continue; }
        hipError_t e = hipEventSynchronize(p.b);
        if (e != hipSuccess) return (int)e;
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, p.a, p.b);
        if (e != hipSuccess) return (int)e;
        Total& t = g_totals[p.name];
        t.ms += ms;
        t.launches += 1;
        g_pool.push_back(p.a);
        g_pool.push_back(p.b);
    }
    g_pending.swap(keep);
    return 0;
}

}  // namespace

KernelTimer::KernelTimer(const char* name, void* stream) : name_(name), stream_(stream) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_on) return;
    if (g_pending.size() > 4096) drain(false);
    start_ = take_event();
    if (start_) hipEventRecord((hipEvent_t)start_, (hipStream_t)stream_);
}

KernelTimer::~KernelTimer() {
    if (!start_) return;
    std::lock_guard<std::mutex> lk(g_mu);
    hipEvent_t b = take_event();
    if (!b) return;
    hipEventRecord(b, (hipStream_t)stream_);
    g_pending.push_back({name_, (hipEvent_t)start_, b});
}

}  // namespace ordermoe

using namespace ordermoe;

extern "C" int ordermoe_timing_enable(int32_t on) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_on = on != 0;
    clear_error();
    return ORDERMOE_OK;
}

extern "C" int ordermoe_timing_read(int32_t max_entries, char* names, double* total_ms,
                                    int64_t* launches, int32_t* n_entries, int32_t reset) {
    if (max_entries < 0 || !n_entries || (max_entries > 0 && (!names || !total_ms || !launches)))
        return fail(ORDERMOE_EINVAL, "timing_read: bad arguments");
    std::lock_guard<std::mutex> lk(g_mu);
    const int e = drain(true);
    if (e) return fail(ORDERMOE_EHIP, std::string("timing_read: ") + hipGetErrorString((hipError_t)e));
    int i = 0;
    for (auto& kv : g_totals) {
        if (i >= max_entries) break;
        std::memset(names + (size_t)i * ORDERMOE_TIMING_NAME, 0, ORDERMOE_TIMING_NAME);
        std::strncpy(names + (size_t)i * ORDERMOE_TIMING_NAME, kv.first.c_str(), ORDERMOE_TIMING_NAME - 1);
        total_ms[i] = kv.second.ms;
        launches[i] = kv.second.launches;
        ++i;
    }
    *n_entries = (int32_t)g_totals.size();
    if (reset) g_totals.clear();
    clear_error();
    return ORDERMOE_OK;
}
