// Stage timing (see oc_timer_* in oc.h): each kernel launched while a timer
// is attached gets a pair of the timer's HIP events, which the runtime
// stamps when the kernel starts and when it ends (oc_launch.h).  The
// attached timer and the current stage are thread-local.
#include "../../include/oc.h"
#include "oc_internal.h"

#include <string>
#include <vector>

struct oc_timer {
    struct Rec { int stage; hipEvent_t a, b; };
    std::vector<std::string> names;
    std::vector<double> total_ms;
    std::vector<long long> launches;
    std::vector<Rec> recs;   // event pool; the first `used` hold pending records
    size_t used = 0;
    bool failed = false;
};

namespace {
thread_local oc_timer *g_timer = nullptr;

int stage_index(oc_timer *t, const char *name) {
    for (size_t i = 0; i < t->names.size(); ++i)
        if (t->names[i] == name) return (int)i;
    t->names.emplace_back(name);
    t->total_ms.push_back(0.0);
    t->launches.push_back(0);
    return (int)t->names.size() - 1;
}
}  // namespace

namespace oc {

// A StageScope names the stage of the launches made inside it.
thread_local int g_stage = -1;

StageScope::StageScope(hipStream_t, const char *name) : prev(g_stage) {
    oc_timer *t = g_timer;
    if (t && !t->failed) g_stage = stage_index(t, name);
}

StageScope::~StageScope() { g_stage = prev; }

bool timed_launch_events(hipStream_t, hipEvent_t *start, hipEvent_t *stop) {
    oc_timer *t = g_timer;
    if (!t || t->failed || g_stage < 0) return false;
    if (t->used == t->recs.size()) {
        oc_timer::Rec r{0, nullptr, nullptr};
        // timing-only events: no system-scope fence when they are stamped
        // (that fence writes back and invalidates the caches, which would
        // lengthen the measured kernel and slow the next one)
        if (hipEventCreateWithFlags(&r.a, hipEventDisableSystemFence) != hipSuccess ||
            hipEventCreateWithFlags(&r.b, hipEventDisableSystemFence) != hipSuccess) {
            t->failed = true;
            return false;
        }
        t->recs.push_back(r);
    }
    oc_timer::Rec &r = t->recs[t->used++];
    r.stage = g_stage;
    *start = r.a;
    *stop = r.b;
    return true;
}

}  // namespace oc

extern "C" {

oc_status oc_timer_create(oc_timer **out) {
    if (!out) return OC_ERR_INVALID_ARG;
    *out = new oc_timer();
    return OC_OK;
}

void oc_timer_destroy(oc_timer *t) {
    if (!t) return;
    if (g_timer == t) g_timer = nullptr;
    for (auto &r : t->recs) {
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
    }
    delete t;
}

oc_status oc_timer_use(oc_timer *t) {
    g_timer = t;
    return OC_OK;
}

oc_status oc_timer_collect(oc_timer *t) {
    if (!t) return OC_ERR_INVALID_ARG;
    for (size_t i = 0; i < t->used; ++i) {
        oc_timer::Rec &r = t->recs[i];
        if (hipEventSynchronize(r.b) != hipSuccess) return OC_ERR_HIP;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return OC_ERR_HIP;
        t->total_ms[r.stage] += ms;
        t->launches[r.stage] += 1;
    }
    t->used = 0;
    return t->failed ? OC_ERR_HIP : OC_OK;
}

oc_status oc_timer_reset(oc_timer *t) {
    if (!t) return OC_ERR_INVALID_ARG;
    for (size_t i = 0; i < t->names.size(); ++i) {
        t->total_ms[i] = 0.0;
        t->launches[i] = 0;
    }
    t->used = 0;
    t->failed = false;
    return OC_OK;
}

int32_t oc_timer_stage_count(const oc_timer *t) { return t ? (int32_t)t->names.size() : 0; }

oc_status oc_timer_stage(const oc_timer *t, int32_t i, const char **name, double *total_ms, int64_t *launches) {
    if (!t || i < 0 || (size_t)i >= t->names.size()) return OC_ERR_INVALID_ARG;
    if (name) *name = t->names[i].c_str();
    if (total_ms) *total_ms = t->total_ms[i];
    if (launches) *launches = t->launches[i];
    return OC_OK;
}

}  // extern "C"
