/*
 * SLO-constrained EC-aware chunk scheduling (SPEAR, arXiv 2606.11244, §4.3).
 *
 * Host-only C ABI, part of libspear.so. The scheduler estimates the latency
 * of one serving iteration from per-module latency tables measured offline
 * at a sparse grid of token counts M: the 4-bit-only table l_W4(M) for a
 * module without an EC, the W4+EC table l_EC(M) for a module the selection
 * S compensates, linearly interpolated for unseen M, and summed over the
 * model's layers. Given d decode tokens already scheduled, it picks the
 * largest prefill chunk c in [c_min, c_max] with
 *
 *     T_S(d) + T_S(c) <= T_SLO,
 *
 * by binary search, which is valid because T_S is nondecreasing in M.
 *
 * Conventions: all pointers are host pointers owned by the caller and only
 * read during the call; latencies are microseconds (double); nothing is
 * allocated, and every function is thread-safe and free of side effects.
 * Errors are negative spear_status_t codes (see spear.h) returned before
 * anything is computed.
 */
#ifndef SPEAR_SCHED_H
#define SPEAR_SCHED_H

#include <stdint.h>

#include "spear.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Latency table of one module type (one linear layer shape): n >= 1 token
 * counts M[0] < M[1] < ... (each >= 1) with the measured latency of the
 * 4-bit-only call and of the W4+EC call at each.
 *
 * Evaluation at token count m (the readings this library takes where §4.3
 * is silent):
 *   m <= 0           -> 0 (no call is made);
 *   0 < m <= M[0]    -> the first entry (a kernel's latency floor);
 *   M[i] < m < M[i+1]-> linear interpolation between the two entries;
 *   m > M[n-1]       -> linear extrapolation along the last segment (the
 *                       last entry when n == 1);
 * and every table is read as its running maximum over M (measured tables
 * carry timing noise; the estimate must be nondecreasing for the search).
 * Latencies must be finite and >= 0. */
typedef struct {
  int32_t n;
  const int64_t* M;      /* [n] token counts, strictly increasing, >= 1 */
  const double* lat_w4;  /* [n] microseconds, 4-bit-only call            */
  const double* lat_ec;  /* [n] microseconds, W4+EC call                  */
} spear_lut_t;

/* One iteration of a model: `layers` x `modules` linear calls, call (l, m)
 * using table luts[m], with the EC table when selection[l * modules + m] is
 * nonzero (the selection S) and the 4-bit table otherwise; plus, when
 * `extra` is not NULL, one evaluation of extra->lat_w4 per layer for the
 * iteration's other work (attention, norms), profiled separately. */
typedef struct {
  int32_t layers;               /* >= 1 */
  int32_t modules;              /* >= 1 */
  const spear_lut_t* luts;      /* [modules] */
  const uint8_t* selection;     /* [layers * modules], 0 or 1 */
  const spear_lut_t* extra;     /* or NULL */
} spear_model_lat_t;

/* T_S(m): the estimated iteration latency in microseconds at token count m.
 * SPEAR_E_NULL for a missing pointer, SPEAR_E_SHAPE for a malformed model or
 * table (sizes, order, negative or non-finite latencies). */
spear_status_t spear_sched_latency(const spear_model_lat_t* model, int64_t m, double* out_us);

/* The largest chunk c in [c_min, c_max] with T_S(d) + T_S(c) <= t_slo_us,
 * in *out_c; 0 when even c_min does not fit (no prefill chunk this
 * iteration). Requires 1 <= c_min <= c_max and d >= 0 (SPEAR_E_SHAPE
 * otherwise). */
spear_status_t spear_sched_chunk(const spear_model_lat_t* model, int64_t d, double t_slo_us,
                                 int64_t c_min, int64_t c_max, int64_t* out_c);

#ifdef __cplusplus
}
#endif

#endif /* SPEAR_SCHED_H */
