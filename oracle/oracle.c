/*
 * Plain fp64 CPU oracle for batched iteration-period detection.
 * TEST INFRASTRUCTURE ONLY; see oracle.h for the definitions it follows
 * (paper Sec. 4.1.2, Algorithms 1 and 2).
 *
 * Built with gcc -O2 -fopenmp -ffp-contract=off: no fused multiply-add, no
 * reassociation.  Threads only run independent sums side by side (one lag or
 * one window each); no single sum is ever split, so results do not depend on
 * the thread count.
 */
#include "oracle.h"

#include <math.h>
#include <stddef.h>
#include <stdlib.h>
#include <omp.h>

static double weight_of(const float* w, int32_t c) { return w ? (double)w[c] : 1.0; }

double oracle_pd_reference(const float* x, int32_t num_channels, int64_t channel_stride,
                           int64_t n, const float* channel_weights) {
    /* Population variance per channel, two passes, then R = 2 * sum_c w_c var_c. */
    double acc = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* xc = x + (int64_t)c * channel_stride;
        double sum = 0.0;
        for (int64_t i = 0; i < n; ++i) sum += (double)xc[i];
        double mean = sum / (double)n;
        double sq = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            double d = (double)xc[i] - mean;
            sq += d * d;
        }
        double var = sq / (double)n;
        acc += weight_of(channel_weights, c) * var;
    }
    return 2.0 * acc;
}

double oracle_pd_score(const float* x, int32_t num_channels, int64_t channel_stride,
                       int64_t n, int64_t t, const float* channel_weights) {
    /* S(T): per channel, the mean over the N-T pairs (i, i+T) of the squared
     * difference; channels are combined as a weighted sum (composite feature). */
    double s = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* xc = x + (int64_t)c * channel_stride;
        double dsum = 0.0;
        for (int64_t i = 0; i < n - t; ++i) {
            double d = (double)xc[i] - (double)xc[i + t];
            dsum += d * d;
        }
        s += weight_of(channel_weights, c) * (dsum / (double)(n - t));
    }
    return s;
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }   /* a >= 0, b > 0 */

void oracle_pd_select(const double* s, int64_t n, int32_t tmin, int32_t tmax, double r,
                      double c_lag, double err_max, oracle_pd_out* out) {
    out->period = 0;
    out->verdict = ORACLE_APERIODIC;
    out->err = 0.0;
    out->n_candidates = 0;
    out->t_cand = 0;
    out->t_low = 0;
    out->t_up = 0;
    out->n_peaks = 0;
    out->r = r;
    out->s_pk = 0.0;
    if (r == 0.0) {
        out->verdict = ORACLE_CONSTANT;
        return;
    }
    /* Peaks: interior local minima, strict on the left and non-strict on the
     * right, so a flat bottom contributes its first lag. */
    int have_peak = 0;
    double s_pk = 0.0;
    for (int32_t t = tmin + 1; t < tmax; ++t) {
        double v = s[t - tmin];
        if (v < s[t - 1 - tmin] && v <= s[t + 1 - tmin]) {
            out->n_peaks++;
            if (!have_peak || v < s_pk) s_pk = v;
            have_peak = 1;
        }
    }
    if (!have_peak) return;
    out->s_pk = s_pk;
    /* Relative-height filter: keep peaks whose height 1 - S/R exceeds c_lag
     * times the highest peak's height. */
    double thr = r - c_lag * (r - s_pk);
    int32_t t_c = 0;
    for (int32_t t = tmin + 1; t < tmax; ++t) {
        double v = s[t - tmin];
        if (v < s[t - 1 - tmin] && v <= s[t + 1 - tmin] && v < thr) {
            out->n_candidates++;
            if (t_c == 0) t_c = t;
        }
    }
    if (t_c == 0) return;
    out->t_cand = t_c;
    /* Local search over the periods of the neighbouring Fourier bins of T_c:
     * D/(k+1) .. D/(k-1) with D = N-1 and T_c = D/k, at a step of one sample. */
    int64_t d = n - 1;
    int64_t lo = ceil_div((int64_t)t_c * d, d + t_c);
    int64_t hi = ((int64_t)t_c * d) / (d - t_c);
    if (lo < tmin) lo = tmin;
    if (hi > tmax) hi = tmax;
    out->t_low = (int32_t)lo;
    out->t_up = (int32_t)hi;
    int64_t best = lo;
    for (int64_t t = lo + 1; t <= hi; ++t)
        if (s[t - tmin] < s[best - tmin]) best = t;
    out->period = (int32_t)best;
    out->err = s[best - tmin] / r;
    out->verdict = (out->err >= err_max) ? ORACLE_APERIODIC : ORACLE_PERIODIC;
}

static int check_params(const oracle_pd_params* p) {
    if (!p) return -1;
    if (p->num_windows < 1 || p->num_channels < 1 || p->n < 4) return -1;
    if (p->tmin < 1 || p->tmin + 2 > p->tmax || (int64_t)p->tmax > p->n / 2) return -1;
    if (p->channel_stride < p->n && p->num_channels > 1) return -1;
    if (p->window_stride < 1 && p->num_windows > 1) return -1;
    if (!(p->c_lag > 0.0 && p->c_lag < 1.0)) return -1;
    if (p->channel_weights)
        for (int32_t c = 0; c < p->num_channels; ++c)
            if (!(p->channel_weights[c] > 0.0f)) return -1;
    return 0;
}

int oracle_pd_detect(const oracle_pd_params* p, const float* x, double* scores,
                     oracle_pd_out* out) {
    if (check_params(p) || !x || !out) return -1;
    const int64_t L = (int64_t)p->tmax - p->tmin + 1;
    double* s_local = NULL;
    for (int64_t b = 0; b < p->num_windows; ++b) {
        const float* xw = x + b * p->window_stride;
        double* sw = scores ? scores + b * L : NULL;
        double r = oracle_pd_reference(xw, p->num_channels, p->channel_stride, p->n,
                                       p->channel_weights);
        if (!sw) {
            if (!s_local) {
                s_local = (double*)malloc((size_t)L * sizeof(double));
                if (!s_local) return -1;
            }
            sw = s_local;
        }
#pragma omp parallel for schedule(dynamic, 16)
        for (int64_t j = 0; j < L; ++j)
            sw[j] = oracle_pd_score(xw, p->num_channels, p->channel_stride, p->n, p->tmin + j,
                                    p->channel_weights);
        oracle_pd_select(sw, p->n, p->tmin, p->tmax, r, p->c_lag, p->err_max, &out[b]);
    }
    free(s_local);
    return 0;
}

int oracle_pd_score_list(const oracle_pd_params* p, const float* x, const int64_t* w,
                         const int32_t* t, int64_t count, double* scores_out) {
    if (check_params(p) || !x || (count > 0 && (!w || !t || !scores_out))) return -1;
    for (int64_t k = 0; k < count; ++k)
        if (w[k] < 0 || w[k] >= p->num_windows || t[k] < 0 || (int64_t)t[k] >= p->n) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t k = 0; k < count; ++k)
        scores_out[k] = oracle_pd_score(x + w[k] * p->window_stride, p->num_channels,
                                        p->channel_stride, p->n, t[k], p->channel_weights);
    return 0;
}

int oracle_pd_threads(void) { return omp_get_max_threads(); }
