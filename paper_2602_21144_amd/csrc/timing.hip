// Per-kernel device timing for measurement runs: when enabled, each kernel the library
// launches on the calling thread is bracketed by a pair of HIP events on its stream.
// Events come from a pool that is reused across collections, so the launch path does
// no event creation once the pool is warm.
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

}  // namespace

KernelTimer::KernelTimer(const char* name, hipStream_t s) : name_(name), s_(s), a_(nullptr) {
    if (!g_on) return;
    if (!g_only.empty() && g_only != name) return;
    // no timing inside graph capture: event records there are not timestamps
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s_, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
        (void)hipGetLastError();
        return;
    }
    a_ = take_event();
    if (a_ && hipEventRecord(a_, s_) != hipSuccess) {
        g_pool.push_back(a_);
        a_ = nullptr;
    }
}

KernelTimer::~KernelTimer() {
    if (!a_) return;
    hipEvent_t b = take_event();
    if (!b || hipEventRecord(b, s_) != hipSuccess) {
        g_pool.push_back(a_);
        if (b) g_pool.push_back(b);
        return;
    }
    g_recs.push_back({name_, a_, b});
}

}  // namespace ssm

extern "C" {

int ssm_timing_enable(int32_t on, const char* only) {
    ssm::g_on = on != 0;
    ssm::g_only = only ? only : "";
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
