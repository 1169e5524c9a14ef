/*
 * libsl skewness-aware dispatching: how many generation instances serve the
 * long-tail samples of a batch, and which instance receives each prompt.
 *
 * StreamRL Section 5.3, "Skewness-aware Scheduling" (Algorithm 2 with Equation 2). The prompts are sorted
 * by estimated output length, longest first, and the first
 * floor(alpha * num_prompts) of them are long-tail samples, the rest regular.
 * The P90 and P50 of a sample of output lengths stand for the average output
 * length of the long-tail and regular groups. For every split
 * num_instances = N_l + N_r, each group's latency is estimated with
 *
 *     Latency = PTL(BS) * L_avg * ceil(M / BS),  BS = min(M, max_batch),
 *
 * M being the prompts one instance of the group receives
 * (ceil(group size / its instances)) and PTL(BS) the per-token decode latency
 * at batch size BS, interpolated linearly in a profile measured beforehand
 * (below the first point: the first value; beyond the last: the last segment
 * continued). The split with the smallest combination of the two latencies is
 * chosen (N_l ascending, first minimum kept); a group with samples needs at
 * least one instance. Within each group the prompts, in sorted order, are
 * dealt round-robin to its instances: long-tail instances are 0 .. N_l - 1,
 * regular ones N_l .. N - 1.
 *
 * Combining the groups: Algorithm 2 adds the two latencies (combine_max = 0);
 * since the groups run on disjoint instances at the same time, their maximum
 * is the wall time of the generation stage (combine_max = 1).
 *
 * Percentiles are lower-rank: element floor(q * (n - 1)) of the sorted sample.
 * Ties in the estimate keep prompt order. Host memory only; no GPU work.
 */
#ifndef SL_DISPATCH_H
#define SL_DISPATCH_H

#include "sl.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sl_ptl_profile {
    int32_t points;          /* >= 1 */
    const int32_t *batch;    /* [points] strictly ascending batch sizes, >= 1 */
    const double *seconds;   /* [points] per-token decode latency at each batch size */
} sl_ptl_profile;

/*
 * Equation 2 for one instance receiving m prompts of average output length
 * l_avg; 0 for m == 0. Errors: SL_ERR_NULL, SL_ERR_SHAPE (m < 0, max_batch < 1,
 * a bad profile).
 */
sl_status sl_generation_latency(const sl_ptl_profile *ptl, double l_avg, int32_t m, int32_t max_batch,
                                double *latency);

/*
 * Algorithm 2.
 *   est_len         [num_prompts] estimated output lengths (host)
 *   alpha           long-tail fraction in [0, 1]
 *   length_samples  [num_samples] output lengths of recent samples (host), num_samples >= 1
 *   num_instances   N >= 1
 *   ptl, max_batch  as for sl_generation_latency
 *   n_long, n_regular  receive N_l, N_r
 *   latency         receives the chosen split's estimate
 *   instance_of     [num_prompts] receives each prompt's instance (may be NULL)
 * Errors: SL_ERR_NULL, SL_ERR_SHAPE (sizes, alpha, profile, or no split gives
 * both non-empty groups an instance).
 */
sl_status sl_dispatch_plan(const int32_t *est_len, int32_t num_prompts, double alpha,
                           const int32_t *length_samples, int32_t num_samples, int32_t num_instances,
                           const sl_ptl_profile *ptl, int32_t max_batch, int32_t combine_max,
                           int32_t *n_long, int32_t *n_regular, double *latency, int32_t *instance_of);

#ifdef __cplusplus
}
#endif

#endif /* SL_DISPATCH_H */
