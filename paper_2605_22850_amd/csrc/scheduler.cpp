// Per-request bandwidth under a shared cap (Section 3.6; the baselines of the
// multi-tenant evaluation).  Request i moves s_i bytes per layer and has a
// compute window of c_i seconds per layer; its zero-stall rate is
// r*_i = s_i / c_i (eq. (4)).
//
// Stall-opt (eqs. (5)-(6)) minimises sum_i s_i / r_i under sum_i r_i = B and
// r_i <= cap_i.  Its solution is r_i = min(cap_i, k * sqrt(s_i)) for the one
// k that spends the budget, and sum_i min(cap_i, k sqrt(s_i)) is piecewise
// linear in k with a breakpoint at each cap_i / sqrt(s_i): sorting the
// breakpoints and sweeping them gives k exactly.  Calibrated Stall-opt
// (eq. (7)) is the same with caps r*_i + delta.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "common.hpp"

namespace oc {

// Capped water-filling: rates r_i = min(cap_i, k sqrt(s_i)), sum = B (or the
// caps, when they fit in B).
void water_fill(int n, const double *s, const double *cap, double B, double *r) {
    double cap_sum = 0.0;
    for (int i = 0; i < n; ++i) cap_sum += cap[i];
    if (cap_sum <= B) {
        for (int i = 0; i < n; ++i) r[i] = cap[i];
        return;
    }
    std::vector<int> order(n);
    std::iota(order.begin(), order.end(), 0);
    std::vector<double> w(n), brk(n);
    for (int i = 0; i < n; ++i) {
        w[i] = std::sqrt(s[i]);
        brk[i] = cap[i] / w[i];
    }
    std::sort(order.begin(), order.end(), [&](int a, int b) { return brk[a] < brk[b]; });
    // the first m requests of `order` are capped; the rest share k
    double capped = 0.0, wfree = 0.0;
    for (int i = 0; i < n; ++i) wfree += w[i];
    double k = 0.0;
    for (int m = 0; m < n; ++m) {
        k = (B - capped) / wfree;
        if (k <= brk[order[m]]) break;   // request order[m] stays below its cap: done
        capped += cap[order[m]];
        wfree -= w[order[m]];
    }
    for (int i = 0; i < n; ++i) r[i] = std::min(cap[i], k * w[i]);
}

}  // namespace oc

using oc::fail;

int oc_bandwidth_allocate(int32_t policy, int32_t n, const double *layer_bytes, const double *layer_compute_s,
                          double budget_bytes_per_s, double margin_bytes_per_s, double *rates_out) {
    oc::clear_error();
    if (n < 1 || !layer_bytes || !rates_out) return fail(OC_EINVAL, "need n >= 1 requests and non-NULL arrays");
    if (!(budget_bytes_per_s > 0.0) || !std::isfinite(budget_bytes_per_s))
        return fail(OC_EINVAL, "budget must be positive and finite");
    if (!(margin_bytes_per_s >= 0.0) || !std::isfinite(margin_bytes_per_s))
        return fail(OC_EINVAL, "margin must be >= 0 and finite");
    for (int i = 0; i < n; ++i)
        if (!(layer_bytes[i] > 0.0) || !std::isfinite(layer_bytes[i]))
            return fail(OC_EINVAL, "layer_bytes must be positive and finite");
    const bool needs_c = policy == OC_ALLOC_BW_PROP || policy == OC_ALLOC_STALL_OPT || policy == OC_ALLOC_CAL_STALL_OPT;
    if (needs_c) {
        if (!layer_compute_s) return fail(OC_EINVAL, "this policy needs the per-layer compute windows");
        for (int i = 0; i < n; ++i)
            if (!(layer_compute_s[i] > 0.0) || !std::isfinite(layer_compute_s[i]))
                return fail(OC_EINVAL, "layer_compute_s must be positive and finite");
    }
    const double B = budget_bytes_per_s;
    std::vector<double> v(n);
    switch (policy) {
        case OC_ALLOC_EQUAL:
            for (int i = 0; i < n; ++i) rates_out[i] = B / n;
            return OC_OK;
        case OC_ALLOC_KV_PROP: {
            double tot = 0.0;
            for (int i = 0; i < n; ++i) tot += layer_bytes[i];
            for (int i = 0; i < n; ++i) rates_out[i] = B * layer_bytes[i] / tot;
            return OC_OK;
        }
        case OC_ALLOC_BW_PROP: {
            double tot = 0.0;
            for (int i = 0; i < n; ++i) tot += (v[i] = layer_bytes[i] / layer_compute_s[i]);
            for (int i = 0; i < n; ++i) rates_out[i] = B * v[i] / tot;
            return OC_OK;
        }
        case OC_ALLOC_STALL_OPT:
        case OC_ALLOC_CAL_STALL_OPT: {
            const double d = policy == OC_ALLOC_CAL_STALL_OPT ? margin_bytes_per_s : 0.0;
            for (int i = 0; i < n; ++i) v[i] = layer_bytes[i] / layer_compute_s[i] + d;
            oc::water_fill(n, layer_bytes, v.data(), B, rates_out);
            return OC_OK;
        }
        default:
            return fail(OC_EINVAL, "unknown allocation policy");
    }
}
