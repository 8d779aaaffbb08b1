/*
 * Plain fp64 CPU oracle for batched iteration-period detection.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * bench's CPU-baseline leg load this library.  It shares no code, header,
 * constant or helper with the GPU library and includes nothing from it.
 *
 * What it computes (paper Sec. 4.1.2, Algorithms 1 and 2, read as below):
 *
 *   For one window with C channels x_c[0..N-1] (fp32 samples, converted
 *   exactly to fp64) and channel weights w_c > 0:
 *
 *   reference   mean_c = (sum_i x_c[i]) / N
 *               var_c  = (sum_i (x_c[i] - mean_c)^2) / N
 *               R      = 2 * (sum_c w_c * var_c)
 *
 *   score       D_c(T) = sum_{i=0}^{N-T-1} (x_c[i] - x_c[i+T])^2
 *               S(T)   = sum_c w_c * (D_c(T) / (N - T))
 *     S(T) is the mean squared point-wise difference between the trace and
 *     itself shifted by one candidate period T: the Euclidean distance between
 *     corresponding points of adjacent sub-curves of length T (Sec. 4.1.2,
 *     Algorithm 2), taken over all N-T overlapping pairs.
 *
 *   selection   (Algorithm 1: peak finding, relative-height candidate filter,
 *               choice of the candidate, local search around it)
 *     peaks     interior local minima Tmin < T < Tmax with
 *               S(T) < S(T-1) and S(T) <= S(T+1)
 *     S_pk      smallest S over the peaks (none -> APERIODIC)
 *     thr       R - c_lag * (R - S_pk)
 *     cands     peaks with S(T) < thr          (none -> APERIODIC)
 *     T_c       smallest candidate (the fundamental)
 *     window    T_low = max(Tmin, ceil (T_c (N-1) / (N-1+T_c)))
 *               T_up  = min(Tmax, floor(T_c (N-1) / (N-1-T_c)))
 *     T_sel     smallest T in [T_low, T_up] attaining the minimum of S
 *     err       S(T_sel) / R;  APERIODIC if err >= err_max, else PERIODIC
 *     R == 0    CONSTANT, period 0, every score 0
 *
 * Every sum above runs in ascending index order, one addition at a time, in
 * fp64 with no fused multiply-add (the library is built with contraction off).
 */
#ifndef ORACLE_PD_H
#define ORACLE_PD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_PERIODIC = 0, ORACLE_APERIODIC = 1, ORACLE_CONSTANT = 2 };

typedef struct {
    int64_t num_windows;
    int32_t num_channels;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t tmin;
    int32_t tmax;
    double c_lag;
    double err_max;
    const float* channel_weights;   /* C weights, or NULL for all 1 */
} oracle_pd_params;

typedef struct {
    int32_t period;
    int32_t verdict;
    double err;
    int32_t n_candidates;
    int32_t t_cand;
    int32_t t_low;
    int32_t t_up;
    int32_t n_peaks;
    double r;
    double s_pk;
} oracle_pd_out;

/* R of one window; x points at channel 0 of the window. */
double oracle_pd_reference(const float* x, int32_t num_channels, int64_t channel_stride,
                           int64_t n, const float* channel_weights);

/* S(T) of one window at one lag. */
double oracle_pd_score(const float* x, int32_t num_channels, int64_t channel_stride,
                       int64_t n, int64_t t, const float* channel_weights);

/* Selection rule on one window's scores s[0..L-1] (s[j] = S(tmin + j)). */
void oracle_pd_select(const double* s, int64_t n, int32_t tmin, int32_t tmax, double r,
                      double c_lag, double err_max, oracle_pd_out* out);

/* Whole batch: scores [B][L] (may be NULL) and one result per window.
 * Returns 0, or -1 on invalid parameters. */
int oracle_pd_detect(const oracle_pd_params* p, const float* x, double* scores,
                     oracle_pd_out* out);

/* Scores only, for a subset: for k in [0, count), scores_out[k] = S(t[k]) of window w[k]. */
int oracle_pd_score_list(const oracle_pd_params* p, const float* x, const int64_t* w,
                         const int32_t* t, int64_t count, double* scores_out);

/* Number of threads the parallel loops use. */
int oracle_pd_threads(void);

#ifdef __cplusplus
}
#endif
#endif
