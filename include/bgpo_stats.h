/*
 * bgpo_stats.h - statistics of repeated gradient estimates (libbgpo).
 *
 * For the gradient standard deviation and bias against the Monte-Carlo
 * sample size n_t (Section 4 "Effect of Increasing MC Sample Sizes",
 * Figure grad_time left and middle): the gradient of a batch is computed
 * several times with independent Monte-Carlo samples, the spread of every
 * parameter's gradient across the repeats is measured, and the mean of the
 * repeats is compared with a reference gradient computed with a large n_t.
 *
 * Conventions as in bgpo.h: device pointers owned by the caller, work
 * enqueued on `stream`, negative bgpo_status on host-detectable errors,
 * nothing allocated.  All float arrays are 16-byte aligned.
 */
#ifndef BGPO_STATS_H_
#define BGPO_STATS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Fold the count-th estimate g (count = number of estimates folded in so far,
 * 0 for the first) into per-element running moments (Welford's update):
 *   delta = g - mean;  mean += delta / (count + 1);  m2 += delta * (g - mean)
 * g, mean, m2: float [n]; mean and m2 are zero before the first update. */
int bgpo_moments_update(const float* g, float* mean, float* m2, int64_t n, int32_t count,
                        void* stream);

/* Bytes of device workspace bgpo_moments_summary needs (8-byte aligned). */
size_t bgpo_moments_workspace_size(void);

/* Summary over all n elements after `count` estimates (count >= 1), float64,
 * reduced in a fixed order (deterministic):
 *   out[0] = mean_i sqrt(m2_i / (count - 1))     mean per-element sample std
 *                                                 (0 for count == 1)
 *   out[1] = mean_i |mean_i - ref_i|              mean absolute bias
 *   out[2] = mean_i |ref_i|                       scale of the reference
 * ref may be NULL (out[1] = out[2] = 0).  out: device double [3]. */
int bgpo_moments_summary(const float* mean, const float* m2, const float* ref, int64_t n,
                         int32_t count, double* out, void* workspace, size_t ws_bytes,
                         void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BGPO_STATS_H_ */
