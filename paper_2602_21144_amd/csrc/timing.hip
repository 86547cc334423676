// Per-kernel device timing for measurement runs: when enabled, each kernel the library
// launches on the calling thread gets a start/stop event pair bound to its own dispatch
// (hipExtLaunchKernel), so the elapsed time is the kernel's execution alone, not the
// time it waited in the queue. Events come from a pool that is reused across
// collections, so the launch path creates no events once the pool is warm.
#include <cstring>
#include <string>
#include <vector>

#include "common.h"

namespace ssm {
namespace {

struct Rec {
    const char* name;
    hipEvent_t a, b;
};

thread_local bool g_on = false;
thread_local std::string g_only;  // when non-empty, only launches with this name are timed
thread_local int g_stride = 1;    // time every g_stride-th launch of each name
thread_local std::vector<std::pair<std::string, int64_t>> g_seen;  // launches per name while enabled

// true for the launches of `name` to time: every g_stride-th one (the first included)
bool sampled(const char* name) {
    if (g_stride <= 1) return true;
    for (auto& kv : g_seen)
        if (kv.first == name) return kv.second++ % g_stride == 0;
    g_seen.emplace_back(name, 1);
    return true;
}
thread_local std::vector<Rec> g_recs;
thread_local std::vector<hipEvent_t> g_pool;

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

thread_local const char* g_cur = nullptr;  // name of the active timer, null when not timing

}  // namespace

KernelTimer::KernelTimer(const char* name, hipStream_t s) : prev_(g_cur) {
    g_cur = nullptr;
    if (!g_on) return;
    if (!g_only.empty() && g_only != name) return;
    if (!sampled(name)) return;
    // nothing is timed inside graph capture: captured launches carry no timestamps
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
        (void)hipGetLastError();
        return;
    }
    g_cur = name;
}

KernelTimer::~KernelTimer() { g_cur = prev_; }

bool launch_timed_events(hipEvent_t* start, hipEvent_t* stop) {
    if (!g_cur) return false;
    hipEvent_t a = take_event();
    hipEvent_t b = a ? take_event() : nullptr;
    if (!b) {
        if (a) g_pool.push_back(a);
        return false;
    }
    g_recs.push_back({g_cur, a, b});
    *start = a;
    *stop = b;
    return true;
}

}  // namespace ssm

extern "C" {

int ssm_timing_enable(int32_t on, const char* only) {
    if (on < 0) return SSM_E_INVAL;
    ssm::g_on = on != 0;
    ssm::g_only = only ? only : "";
    ssm::g_stride = on > 1 ? on : 1;
    ssm::g_seen.clear();
    return SSM_OK;
}

int ssm_timing_collect(ssm_kernel_time_t* out, int32_t max, int32_t* count) {
    using namespace ssm;
    if (!count || max < 0 || (max > 0 && !out)) return SSM_E_INVAL;
    std::vector<ssm_kernel_time_t> acc;
    int rc = SSM_OK;
    for (const Rec& r : g_recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) rc = SSM_E_HIP;
        ssm_kernel_time_t* slot = nullptr;
        for (auto& k : acc)
            if (std::strncmp(k.name, r.name, sizeof k.name) == 0) slot = &k;
        if (!slot) {
            acc.push_back({});
            slot = &acc.back();
            std::strncpy(slot->name, r.name, sizeof slot->name - 1);
        }
        slot->launches += 1;
        slot->total_ms += ms;
        g_pool.push_back(r.a);
        g_pool.push_back(r.b);
    }
    g_recs.clear();
    const int n = (int)acc.size() < max ? (int)acc.size() : max;
    for (int i = 0; i < n; ++i) out[i] = acc[i];
    *count = n;
    return rc;
}

}  // extern "C"
