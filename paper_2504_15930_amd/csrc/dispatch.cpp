// Skewness-aware dispatching (include/sl_dispatch.h): Algorithm 2 with
// Equation 2, on the host.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "sl_dispatch.h"

namespace {

bool valid_profile(const sl_ptl_profile *p)
{
    if (!p || p->points < 1 || !p->batch || !p->seconds)
        return false;
    for (int k = 0; k < p->points; ++k)
        if (p->batch[k] < 1 || (k > 0 && p->batch[k] <= p->batch[k - 1]))
            return false;
    return true;
}

// PTL(batch): linear between profiled points, first value below them, last
// segment continued beyond them.
double ptl_at(const sl_ptl_profile &p, int batch)
{
    const int32_t *x = p.batch;
    const double *y = p.seconds;
    if (batch <= x[0] || p.points == 1)
        return y[0];
    for (int k = 1; k < p.points; ++k)
        if (batch <= x[k])
            return y[k - 1] + (y[k] - y[k - 1]) * (double)(batch - x[k - 1]) / (double)(x[k] - x[k - 1]);
    const int k = p.points - 1;
    return y[k] + (y[k] - y[k - 1]) * (double)(batch - x[k]) / (double)(x[k] - x[k - 1]);
}

double equation2(const sl_ptl_profile &p, double l_avg, int m, int max_batch)
{
    if (m == 0)
        return 0.0;
    const int bs = std::min(m, max_batch);
    const int rounds = (m + bs - 1) / bs;
    return ptl_at(p, bs) * l_avg * rounds;
}

int percentile_lower(std::vector<int32_t> v, double q)
{
    std::sort(v.begin(), v.end());
    return v[(size_t)std::floor(q * (double)(v.size() - 1))];
}

}  // namespace

extern "C" {

sl_status sl_generation_latency(const sl_ptl_profile *ptl, double l_avg, int32_t m, int32_t max_batch,
                                double *latency)
{
    if (!ptl || !latency)
        return SL_ERR_NULL;
    if (!valid_profile(ptl) || m < 0 || max_batch < 1)
        return SL_ERR_SHAPE;
    *latency = equation2(*ptl, l_avg, m, max_batch);
    return SL_OK;
}

sl_status sl_dispatch_plan(const int32_t *est_len, int32_t num_prompts, double alpha,
                           const int32_t *length_samples, int32_t num_samples, int32_t num_instances,
                           const sl_ptl_profile *ptl, int32_t max_batch, int32_t combine_max,
                           int32_t *n_long, int32_t *n_regular, double *latency, int32_t *instance_of)
{
    if (!est_len || !length_samples || !ptl || !n_long || !n_regular || !latency)
        return SL_ERR_NULL;
    if (num_prompts < 1 || num_samples < 1 || num_instances < 1 || max_batch < 1 || !(alpha >= 0.0) ||
        alpha > 1.0 || !valid_profile(ptl))
        return SL_ERR_SHAPE;
    // Sort by estimate, longest first, ties in prompt order; mark the long tail.
    std::vector<int32_t> order(num_prompts);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [est_len](int a, int b) { return est_len[a] > est_len[b]; });
    const int n_tail = (int)std::floor(alpha * (double)num_prompts);
    const int n_reg = num_prompts - n_tail;
    const std::vector<int32_t> dist(length_samples, length_samples + num_samples);
    const double l_alpha = percentile_lower(dist, 0.9);
    const double l_r = percentile_lower(dist, 0.5);
    int best_l = -1;
    double best = 0.0;
    for (int nl = 0; nl <= num_instances; ++nl) {
        const int nr = num_instances - nl;
        if ((n_tail > 0 && nl == 0) || (n_reg > 0 && nr == 0))
            continue;
        const double lat_l = equation2(*ptl, l_alpha, nl ? (n_tail + nl - 1) / nl : 0, max_batch);
        const double lat_r = equation2(*ptl, l_r, nr ? (n_reg + nr - 1) / nr : 0, max_batch);
        const double total = combine_max ? std::max(lat_l, lat_r) : lat_l + lat_r;
        if (best_l < 0 || total < best) {
            best = total;
            best_l = nl;
        }
    }
    if (best_l < 0)
        return SL_ERR_SHAPE;
    *n_long = best_l;
    *n_regular = num_instances - best_l;
    *latency = best;
    if (instance_of) {
        for (int k = 0; k < n_tail; ++k)
            instance_of[order[k]] = k % best_l;
        for (int k = 0; k < n_reg; ++k)
            instance_of[order[n_tail + k]] = best_l + k % (num_instances - best_l);
    }
    return SL_OK;
}

}  // extern "C"
