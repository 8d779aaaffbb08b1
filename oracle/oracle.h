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
 *   (with params.centred = 1 every S below is the mean-removed S_c instead;
 *   see oracle_pd_score_centred)
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
    int32_t centred;                /* 1: the mean-removed score S_c below instead of S */
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

/* Mean-removed score S_c(T) of one window at one lag (Sec. 4.1.2, Algorithm 2
 * with one group per sample: every value is taken relative to the mean of its
 * own sub-curve before corresponding points of adjacent sub-curves are compared):
 *
 *   Num_T = floor(N / T) whole sub-curves; K = Num_T - 1 adjacent pairs
 *   mu_i  = (sum_{j<T} x_c[iT + j]) / T
 *   D_c   = sum_{i<K} sum_{j<T} ((x_c[iT+j] - mu_i) - (x_c[(i+1)T+j] - mu_{i+1}))^2
 *   S_c(T) = sum_c w_c * (D_c / (K T))
 *
 * Unlike S it is unchanged by adding a linear ramp to a channel, so a drifting
 * periodic trace still scores exactly zero at its period.  Each mean is a
 * sequential sum divided by T, recomputed for every pair that uses it. */
double oracle_pd_score_centred(const float* x, int32_t num_channels, int64_t channel_stride,
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

/* Algorithm 3 (Sec. 4.1.3): rolling detection over suffix windows.
 *
 *   T_init  = period of the whole window (the rule above); if it is not
 *             PERIODIC the result carries its verdict, period 0 and no windows.
 *   D       = N - 1 (the sampling duration in samples, T_s = 1)
 *   D < c_measure * T_init: too short; period T_init, next = c_measure T_init - D
 *   suffix k = 0 .. J-1 starts at s_k = s_0 + k step T_init,
 *       s_0 = max(0, D - (2 + c_eval * step) * T_init),
 *       J = the number of k with D - s_k >= c_measure T_init;
 *       it holds x[floor(s_k) .. N-1] (N_j = N - floor(s_k) samples) and is
 *       scored on the lags [tmin, min(tmax, N_j / 2)] by the same rule -> T_j, err_j
 *   the suffixes with a PERIODIC verdict form T and Err (none -> APERIODIC)
 *   period  = T_k with err_k = min Err (first such k)
 *   diff    = |max T - min T| / mean T
 *   next    = -1 (stable) if diff < diff_threshold,
 *             else ceil(D / max T) * max T - D
 */
#define ORACLE_ROLLING_MAX 32

typedef struct {
    double c_measure;       /* 2 in the paper */
    double step;            /* 0.5 */
    double c_eval;          /* 6.5 */
    double diff_threshold;  /* not given by the paper */
} oracle_pd_rolling_params;

typedef struct {
    int32_t period;
    int32_t verdict;
    int32_t stable;
    int32_t n_windows;
    int32_t t_init;
    int32_t best;                       /* index of the selected suffix window, -1 if none */
    double smpdur_next;
    double diff;
    double err;
    int64_t starts[ORACLE_ROLLING_MAX];  /* suffix start sample */
    int32_t periods[ORACLE_ROLLING_MAX]; /* T_j (0: no period) */
    int32_t verdicts[ORACLE_ROLLING_MAX];
    double errs[ORACLE_ROLLING_MAX];
} oracle_pd_rolling_out;

/* The suffix-window schedule alone: for a window of n samples and T_init,
 * writes the start sample of every suffix window and returns their number, or
 * returns 0 and sets *short_next to c_measure T_init - D when the window is too
 * short (otherwise *short_next = 0); -1 if more than `cap` windows. */
int32_t oracle_pd_rolling_schedule(int64_t n, int32_t t_init, const oracle_pd_rolling_params* rp,
                                   int64_t* starts, int32_t cap, double* short_next);

/* One result per window of the batch; returns 0, or -1 on invalid parameters
 * (including a schedule longer than ORACLE_ROLLING_MAX windows). */
int oracle_pd_rolling(const oracle_pd_params* p, const oracle_pd_rolling_params* rp,
                      const float* x, oracle_pd_rolling_out* out);

/* Algorithm 2 (Sec. 4.1.2): feature sequence similarity error Err_T.
 *
 *   sub-curves  Smp_i = x[(i-1) T .. i T - 1], i = 1 .. Num_T = floor(N / T)
 *   for each adjacent pair (Smp_i, Smp_{i+1}), per channel:
 *     groups    a 1-D Gaussian mixture of num_groups components fitted to the
 *               values of Smp_i by em_iters EM iterations (fp64), then every
 *               sample assigned to its most responsible component (ties: the
 *               lower index).  Initialisation: means evenly spaced at
 *               min + (k + 1/2) (max - min) / G, variances ((max - min) / G)^2,
 *               weights 1/G; variances never drop below 1e-6 ((max - min)/G)^2;
 *               a component that loses all responsibility keeps its
 *               parameters.  A constant Smp_i is a single group.
 *     RelVal    group mean minus sub-curve mean, on Smp_i and on Smp_{i+1}
 *               with the same sample indices
 *     grperr    SMAPE(a, b) = |a - b| / ((|a| + |b|) / 2), 0 / 0 := 0
 *     err_i     mean of grperr over groups weighted by group size
 *   Err_T      mean over the Num_T - 1 pairs, then weighted sum over channels
 *              (weights w_c / sum w_c); -1 when Num_T < 2.
 */
typedef struct {
    int32_t num_groups;     /* NumG; the paper leaves it open */
    int32_t em_iters;       /* EM iterations */
} oracle_pd_similarity_params;

/* err_out[k] = Err_T of window w[k] at lag t[k]; returns 0 or -1. */
int oracle_pd_similarity(const oracle_pd_params* p, const oracle_pd_similarity_params* sp,
                         const float* x, const int64_t* w, const int32_t* t, int64_t count,
                         double* err_out);

/* Number of threads the parallel loops use. */
int oracle_pd_threads(void);

#ifdef __cplusplus
}
#endif
#endif
