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
using oc::guarded;

static int bandwidth_allocate_body(int32_t policy, int32_t n, const double *layer_bytes, const double *layer_compute_s,
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

int oc_bandwidth_allocate(int32_t policy, int32_t n, const double *layer_bytes, const double *layer_compute_s,
                          double budget_bytes_per_s, double margin_bytes_per_s, double *rates_out) {
    return guarded([&] {
        return bandwidth_allocate_body(policy, n, layer_bytes, layer_compute_s, budget_bytes_per_s,
                                       margin_bytes_per_s, rates_out);
    });
}

// Scheduling epochs (Section 3.6): the rates of oc_bandwidth_allocate for
// requests that arrive over time.  At each epoch boundary the requests that
// have arrived and wait are admitted together and share the budget that the
// requests in flight do not hold, under the policy; a request keeps its rate
// until its payloads are delivered (its last byte at admission + L s_i / r_i),
// and the rate it then releases is handed out at the next boundary, never to
// a request already in flight.  Boundaries are the multiples of epoch_s, or
// with epoch_s == 0 every arrival and every completion.
static int epoch_schedule_body(int32_t policy, int32_t n, const double *layer_bytes, const double *layer_compute_s,
                               int32_t num_layers, const double *arrival_s, double budget_bytes_per_s,
                               double margin_bytes_per_s, double epoch_s, double *rates_out, double *admit_s_out) {
    oc::clear_error();
    if (n < 1 || !layer_bytes || !arrival_s || !rates_out || !admit_s_out)
        return fail(OC_EINVAL, "need n >= 1 requests and non-NULL arrays");
    if (num_layers < 1) return fail(OC_EINVAL, "num_layers must be >= 1");
    if (!(epoch_s >= 0.0) || !std::isfinite(epoch_s)) return fail(OC_EINVAL, "epoch_s must be >= 0 and finite");
    for (int i = 0; i < n; ++i)
        if (!(arrival_s[i] >= 0.0) || !std::isfinite(arrival_s[i]))
            return fail(OC_EINVAL, "arrival_s must be >= 0 and finite");
    // the per-call checks of oc_bandwidth_allocate, on all requests at once
    {
        std::vector<double> probe(n);
        const int rc = oc_bandwidth_allocate(policy, n, layer_bytes, layer_compute_s, budget_bytes_per_s,
                                             margin_bytes_per_s, probe.data());
        if (rc) return rc;
    }
    const double B = budget_bytes_per_s;
    const double tiny = 1e-9 * B;                 // a budget residue admits nobody
    std::vector<char> admitted(n, 0);
    std::vector<double> finish(n, 0.0);
    int left = n;
    double t = 0.0;
    for (bool first = true; left > 0; first = false) {
        if (!first) {
            // the next event after t: an arrival or the end of a delivery
            double nx = INFINITY;
            for (int i = 0; i < n; ++i) {
                if (!admitted[i] && arrival_s[i] > t) nx = std::min(nx, arrival_s[i]);
                if (admitted[i] && finish[i] > t) nx = std::min(nx, finish[i]);
            }
            if (!std::isfinite(nx)) return fail(OC_EINVAL, "epoch schedule: requests wait with nothing in flight");
            t = nx;
        }
        if (epoch_s > 0.0) {      // the first boundary at or after the event
            double bnd = std::ceil(t / epoch_s) * epoch_s;
            if (bnd < t) bnd += epoch_s;
            t = bnd;
        }
        double held = 0.0;
        std::vector<int32_t> waiting;
        for (int i = 0; i < n; ++i) {
            if (admitted[i] && finish[i] > t) held += rates_out[i];
            if (!admitted[i] && arrival_s[i] <= t) waiting.push_back(i);
        }
        const double free_bw = B - held;
        if (waiting.empty() || free_bw <= tiny) continue;
        const int m = (int)waiting.size();
        std::vector<double> s(m), c(m), r(m);
        for (int k = 0; k < m; ++k) {
            s[k] = layer_bytes[waiting[k]];
            c[k] = layer_compute_s ? layer_compute_s[waiting[k]] : 0.0;
        }
        const int rc = oc_bandwidth_allocate(policy, m, s.data(), layer_compute_s ? c.data() : nullptr, free_bw,
                                             margin_bytes_per_s, r.data());
        if (rc) return rc;
        for (int k = 0; k < m; ++k) {
            const int i = waiting[k];
            admitted[i] = 1;
            rates_out[i] = r[k];
            admit_s_out[i] = t;
            finish[i] = t + num_layers * layer_bytes[i] / r[k];
            --left;
        }
    }
    return OC_OK;
}

int oc_epoch_schedule(int32_t policy, int32_t n, const double *layer_bytes, const double *layer_compute_s,
                      int32_t num_layers, const double *arrival_s, double budget_bytes_per_s,
                      double margin_bytes_per_s, double epoch_s, double *rates_out, double *admit_s_out) {
    return guarded([&] {
        return epoch_schedule_body(policy, n, layer_bytes, layer_compute_s, num_layers, arrival_s, budget_bytes_per_s,
                                   margin_bytes_per_s, epoch_s, rates_out, admit_s_out);
    });
}
