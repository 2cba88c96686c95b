/*
 * kvshot_metrics.h -- C ABI of the drafting metrics on MI355X (gfx950).
 *
 * Operation (KVShot, arXiv 2604.26412, Sec. 3.1, "Metrics"; retention as in
 * the Sec. 3.2 tables): from per-verification accepted draft lengths a_i
 * (values outside [0, K] are clamped into it), with K draft steps,
 *     c_k     = #{ i : a_i >= k }                 k = 0 .. K
 *     alpha_k = c_{k+1} / c_k  (0 when c_k = 0)   k = 0 .. K - 1
 *     MAT     = 1 + sum_{k=0}^{K-1} prod_{j=0}^{k} alpha_j
 *     retention = alpha_r / alpha_0               (r = retention_step)
 * alpha_k is the acceptance rate of draft step k among verifications whose
 * earlier steps were all accepted, so MAT = 1 + the mean accepted length.
 *
 * Conventions as in kvshot_draft_attn.h: device pointers unless marked (host);
 * the caller owns every array until the work queued on `stream` has finished;
 * argument errors are returned before anything is queued.  The call needs no
 * handle and allocates nothing; counts are exact (64-bit integer atomics, any
 * order) and the float64 results are deterministic.
 */
#ifndef KVSHOT_METRICS_H
#define KVSHOT_METRICS_H

#include <stdint.h>

#include "kvshot_draft_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* accepted   int32 [n], n >= 0 (NULL allowed when n == 0)
 * K          draft steps, 1 <= K <= 255
 * counts     int64 [K + 1]: c_0 .. c_K (written; also the histogram's scratch)
 * alpha      float64 [K]: alpha_0 .. alpha_{K-1}
 * mat        float64 [1]
 * retention  nullable float64 [1]: alpha_{retention_step} / alpha_0 (0 when alpha_0 = 0);
 *            0 <= retention_step < K
 * Every device pointer must be 8-byte aligned (accepted: 4-byte). */
kvshot_status kvshot_acceptance_stats(const int32_t* accepted, int64_t n, int32_t K, int64_t* counts, double* alpha,
                                      double* mat, double* retention, int32_t retention_step, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVSHOT_METRICS_H */
