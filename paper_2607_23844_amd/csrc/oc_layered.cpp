// Layered Cache schedule proposal (§3.4, Alg. 1), host side: which layer /
// timestep pairs reuse cached features under a target speed-up.  Each
// candidate pair (l, t) is scored w = Q[l,t] / L[l,t] (quality lost per unit
// of latency saved); candidates are taken from the lowest score up, each as
// (l, t, N), until the saved latency reaches (1 - 1/s_r) times the summed
// latency of all candidates.  Candidates are enumerated layer-major, equal
// scores keep that order (stable sort) and every sum runs in that order, so
// the result is fully determined by the inputs.
#include "../../include/oc.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <numeric>
#include <vector>

namespace oc {
oc_status record_error(oc_status s, const char *msg);   // oc_api.cpp
}

extern "C" oc_status oc_layered_schedule(int32_t n_layers, int32_t n_steps, const double *latency,
                                         const double *quality, const uint8_t *mask, double target_speedup,
                                         int32_t interval, oc_cache_entry *out, int32_t capacity, int32_t *n_out,
                                         double *saved_out, double *budget_out) {
    if (n_layers < 0 || n_steps < 0 || (long long)n_layers * n_steps > (1LL << 30))
        return oc::record_error(OC_ERR_SHAPE, "n_layers and n_steps must be >= 0 (and their product < 2^30)");
    if (!latency || !quality || !n_out || (!out && capacity > 0))
        return oc::record_error(OC_ERR_INVALID_ARG, "NULL pointer");
    if (!(target_speedup >= 1.0)) return oc::record_error(OC_ERR_INVALID_ARG, "target speed-up must be >= 1");
    if (interval < 1) return oc::record_error(OC_ERR_INVALID_ARG, "cache interval must be >= 1");
    const int n = n_layers * n_steps;
    std::vector<int> P;                       // candidate pairs, layer-major
    P.reserve(n);
    for (int i = 0; i < n; ++i) {
        if (mask && !mask[i]) continue;
        if (!(latency[i] > 0.0) || !std::isfinite(latency[i]) || !std::isfinite(quality[i]))
            return oc::record_error(OC_ERR_INVALID_ARG,
                                    "every candidate needs a finite latency > 0 and a finite quality loss");
        P.push_back(i);
    }
    std::vector<double> w(P.size());
    for (size_t i = 0; i < P.size(); ++i) w[i] = quality[P[i]] / latency[P[i]];
    std::vector<int> order(P.size());
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return w[a] < w[b]; });
    double total = 0.0;
    for (int i : P) total += latency[i];
    const double budget = (1.0 - 1.0 / target_speedup) * total;
    double saved = 0.0;
    int k = 0;
    for (size_t j = 0; j < order.size() && saved < budget; ++j) {
        const int i = P[order[j]];
        if (k >= capacity) return oc::record_error(OC_ERR_INVALID_ARG, "output capacity too small");
        out[k].layer = i / n_steps;
        out[k].step = i % n_steps;
        out[k].interval = interval;
        ++k;
        saved += latency[i];
    }
    *n_out = k;
    if (saved_out) *saved_out = saved;
    if (budget_out) *budget_out = budget;
    return oc::record_error(OC_OK, "");
}
