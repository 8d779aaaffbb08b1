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
#include <string.h>
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

double oracle_pd_score_centred(const float* x, int32_t num_channels, int64_t channel_stride,
                               int64_t n, int64_t t, const float* channel_weights) {
    /* Algorithm 2's relative values with one group per sample: whole
     * sub-curves of T samples, each pair of neighbours compared point by point
     * after removing each sub-curve's own mean. */
    double s = 0.0;
    const int64_t pairs = n / t - 1;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* xc = x + (int64_t)c * channel_stride;
        double dsum = 0.0;
        for (int64_t i = 0; i < pairs; ++i) {
            const float* a = xc + i * t;
            const float* b = a + t;
            double sa = 0.0, sb = 0.0;
            for (int64_t j = 0; j < t; ++j) sa += (double)a[j];
            for (int64_t j = 0; j < t; ++j) sb += (double)b[j];
            const double mu_a = sa / (double)t, mu_b = sb / (double)t;
            for (int64_t j = 0; j < t; ++j) {
                const double d = ((double)a[j] - mu_a) - ((double)b[j] - mu_b);
                dsum += d * d;
            }
        }
        s += weight_of(channel_weights, c) * (dsum / (double)(pairs * t));
    }
    return s;
}

static double score_of(const oracle_pd_params* p, const float* xw, int64_t n, int64_t t) {
    return p->centred
               ? oracle_pd_score_centred(xw, p->num_channels, p->channel_stride, n, t,
                                         p->channel_weights)
               : oracle_pd_score(xw, p->num_channels, p->channel_stride, n, t,
                                 p->channel_weights);
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
        for (int64_t j = 0; j < L; ++j) sw[j] = score_of(p, xw, p->n, p->tmin + j);
        oracle_pd_select(sw, p->n, p->tmin, p->tmax, r, p->c_lag, p->err_max, &out[b]);
    }
    free(s_local);
    return 0;
}

int oracle_pd_score_list(const oracle_pd_params* p, const float* x, const int64_t* w,
                         const int32_t* t, int64_t count, double* scores_out) {
    if (check_params(p) || !x || (count > 0 && (!w || !t || !scores_out))) return -1;
    for (int64_t k = 0; k < count; ++k)
        if (w[k] < 0 || w[k] >= p->num_windows || t[k] < 0 || (int64_t)t[k] >= p->n ||
            (p->centred && (t[k] < 1 || 2 * (int64_t)t[k] > p->n)))
            return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t k = 0; k < count; ++k)
        scores_out[k] = score_of(p, x + w[k] * p->window_stride, p->n, t[k]);
    return 0;
}

/* The rule on one window of n samples (channels at channel_stride), lags
 * [tmin, tmax]; scores in the caller's buffer of tmax - tmin + 1 doubles. */
static void detect_one(const oracle_pd_params* p, const float* xw, int64_t n, int32_t tmax,
                       double* s, oracle_pd_out* o) {
    const int64_t L = (int64_t)tmax - p->tmin + 1;
    double r = oracle_pd_reference(xw, p->num_channels, p->channel_stride, n, p->channel_weights);
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t j = 0; j < L; ++j) s[j] = score_of(p, xw, n, p->tmin + j);
    oracle_pd_select(s, n, p->tmin, tmax, r, p->c_lag, p->err_max, o);
}

int32_t oracle_pd_rolling_schedule(int64_t n, int32_t t_init, const oracle_pd_rolling_params* rp,
                                   int64_t* starts, int32_t cap, double* short_next) {
    /* Algorithm 3 (Sec. 4.1.3) measures suffixes of the trace that start
     * (2 + c_eval step) periods before its end and then every step periods
     * later, as long as at least c_measure periods remain.  With u = step T,
     * s_k = s_0 + k u for s_0 = max(0, D - (2 + c_eval step) T), the suffix k
     * exists iff D - s_k >= c_measure T, i.e. k <= (D - s_0 - c_measure T) / u:
     * J = floor of that, plus one, suffixes.  The rounded quotient is checked
     * against the condition itself on both sides of J. */
    const double t = (double)t_init;
    const double dur = (double)(n - 1);
    const double need = rp->c_measure * t;
    *short_next = 0.0;
    if (dur < need) {
        *short_next = need - dur;
        return 0;
    }
    double s0 = dur - (2.0 + rp->c_eval * rp->step) * t;
    if (s0 < 0.0) s0 = 0.0;
    const double u = rp->step * t;
    if (dur - s0 < need) return 0;
    double jq = floor((dur - s0 - need) / u);
    if (jq > (double)cap) return -1;
    int64_t j = (int64_t)jq + 1;
    while (j > 1 && !(dur - (s0 + (double)(j - 1) * u) >= need)) --j;
    while (dur - (s0 + (double)j * u) >= need) {
        ++j;
        if (j > cap) return -1;
    }
    if (j > cap) return -1;
    for (int64_t k = 0; k < j; ++k) starts[k] = (int64_t)floor(s0 + (double)k * u);
    return (int32_t)j;
}

int oracle_pd_rolling(const oracle_pd_params* p, const oracle_pd_rolling_params* rp,
                      const float* x, oracle_pd_rolling_out* out) {
    if (check_params(p) || !rp || !x || !out) return -1;
    if (!(rp->c_measure > 0.0) || !(rp->step > 0.0) || !(rp->c_eval >= 0.0)) return -1;
    const int64_t L = (int64_t)p->tmax - p->tmin + 1;
    double* s = (double*)malloc((size_t)L * sizeof(double));
    if (!s) return -1;
    int rc = 0;
    for (int64_t b = 0; b < p->num_windows && rc == 0; ++b) {
        const float* xw = x + b * p->window_stride;
        oracle_pd_rolling_out* o = &out[b];
        memset(o, 0, sizeof(*o));
        o->best = -1;
        oracle_pd_out first;
        detect_one(p, xw, p->n, p->tmax, s, &first);
        o->t_init = first.period;
        if (first.verdict != ORACLE_PERIODIC) {
            o->verdict = first.verdict;
            continue;
        }
        const double dur = (double)(p->n - 1);
        double short_next;
        const int32_t j = oracle_pd_rolling_schedule(p->n, first.period, rp, o->starts,
                                                     ORACLE_ROLLING_MAX, &short_next);
        if (j < 0) {
            rc = -1;
            break;
        }
        if (j == 0) {   /* too short for a rolling evaluation (or no suffix fits) */
            o->verdict = ORACLE_PERIODIC;
            o->period = first.period;
            o->err = first.err;
            o->smpdur_next = short_next;
            continue;
        }
        for (int32_t k = 0; k < j; ++k) {
            const int64_t start = o->starts[k];
            const int64_t nj = p->n - start;
            int32_t tmax_j = p->tmax;
            if ((int64_t)tmax_j > nj / 2) tmax_j = (int32_t)(nj / 2);
            if (tmax_j >= p->tmin + 2) {
                oracle_pd_out sub;
                detect_one(p, xw + start, nj, tmax_j, s, &sub);
                o->verdicts[k] = sub.verdict;
                o->periods[k] = sub.verdict == ORACLE_PERIODIC ? sub.period : 0;
                o->errs[k] = sub.err;
            } else {
                o->verdicts[k] = ORACLE_APERIODIC;
            }
        }
        o->n_windows = j;
        /* best window, spread and next sampling duration over the periodic suffixes */
        int32_t cnt = 0, tmin_p = 0, tmax_p = 0;
        double sum = 0.0;
        for (int32_t k = 0; k < j; ++k) {
            if (o->verdicts[k] != ORACLE_PERIODIC) continue;
            if (o->best < 0 || o->errs[k] < o->errs[o->best]) o->best = k;
            if (cnt == 0 || o->periods[k] < tmin_p) tmin_p = o->periods[k];
            if (cnt == 0 || o->periods[k] > tmax_p) tmax_p = o->periods[k];
            sum += (double)o->periods[k];
            ++cnt;
        }
        if (cnt == 0) {
            o->verdict = ORACLE_APERIODIC;
            continue;
        }
        o->verdict = ORACLE_PERIODIC;
        o->period = o->periods[o->best];
        o->err = o->errs[o->best];
        o->diff = fabs(((double)tmax_p - (double)tmin_p) / (sum / (double)cnt));
        if (o->diff < rp->diff_threshold) {
            o->stable = 1;
            o->smpdur_next = -1.0;
        } else {
            o->smpdur_next = ceil(dur / (double)tmax_p) * (double)tmax_p - dur;
        }
    }
    free(s);
    return rc;
}

/* SMAPE of two relative group values; 0 / 0 := 0. */
static double smape(double a, double b) {
    const double den = (fabs(a) + fabs(b)) / 2.0;
    if (den == 0.0) return 0.0;
    return fabs(a - b) / den;
}

/* Hard group index of every sample of v[0..m-1] (1-D GMM, EM, see oracle.h). */
static void gmm_groups(const double* v, int64_t m, int32_t g, int32_t iters, int32_t* group,
                       double* resp /* m * g scratch */) {
    double lo = v[0], hi = v[0];
    for (int64_t i = 1; i < m; ++i) {
        if (v[i] < lo) lo = v[i];
        if (v[i] > hi) hi = v[i];
    }
    if (hi == lo) {
        for (int64_t i = 0; i < m; ++i) group[i] = 0;
        return;
    }
    double mu[64], var[64], pi[64];
    const double width = (hi - lo) / (double)g;
    const double floor_var = 1e-6 * width * width;
    for (int32_t k = 0; k < g; ++k) {
        mu[k] = lo + ((double)k + 0.5) * width;
        var[k] = width * width;
        pi[k] = 1.0 / (double)g;
    }
    const double two_pi = 6.283185307179586;
    for (int32_t it = 0; it < iters; ++it) {
        /* E step: responsibilities from log densities, normalised per sample */
        for (int64_t i = 0; i < m; ++i) {
            double* r = resp + i * g;
            double best = -INFINITY;
            for (int32_t k = 0; k < g; ++k) {
                const double d = v[i] - mu[k];
                r[k] = log(pi[k]) - 0.5 * log(two_pi * var[k]) - d * d / (2.0 * var[k]);
                if (r[k] > best) best = r[k];
            }
            double sum = 0.0;
            for (int32_t k = 0; k < g; ++k) {
                r[k] = exp(r[k] - best);
                sum += r[k];
            }
            for (int32_t k = 0; k < g; ++k) r[k] /= sum;
        }
        /* M step */
        for (int32_t k = 0; k < g; ++k) {
            double nk = 0.0, s1 = 0.0;
            for (int64_t i = 0; i < m; ++i) {
                nk += resp[i * g + k];
                s1 += resp[i * g + k] * v[i];
            }
            if (!(nk > 0.0)) continue;
            const double mk = s1 / nk;
            double s2 = 0.0;
            for (int64_t i = 0; i < m; ++i) {
                const double d = v[i] - mk;
                s2 += resp[i * g + k] * d * d;
            }
            mu[k] = mk;
            var[k] = s2 / nk;
            if (var[k] < floor_var) var[k] = floor_var;
            pi[k] = nk / (double)m;
        }
    }
    /* hard assignment: the most responsible component (lower index on ties) */
    for (int64_t i = 0; i < m; ++i) {
        int32_t arg = 0;
        double best = -INFINITY;
        for (int32_t k = 0; k < g; ++k) {
            const double d = v[i] - mu[k];
            const double lk = log(pi[k]) - 0.5 * log(two_pi * var[k]) - d * d / (2.0 * var[k]);
            if (lk > best) {
                best = lk;
                arg = k;
            }
        }
        group[i] = arg;
    }
}

/* Err_T of one channel of one window (Algorithm 2). */
static double similarity_one(const float* xc, int64_t n, int64_t t, int32_t g, int32_t iters) {
    const int64_t num_t = n / t;
    if (num_t < 2) return -1.0;
    double* a = (double*)malloc((size_t)t * sizeof(double));
    double* b = (double*)malloc((size_t)t * sizeof(double));
    int32_t* grp = (int32_t*)malloc((size_t)t * sizeof(int32_t));
    double* resp = (double*)malloc((size_t)t * (size_t)g * sizeof(double));
    if (!a || !b || !grp || !resp) {
        free(a); free(b); free(grp); free(resp);
        return -2.0;
    }
    double total = 0.0;
    for (int64_t i = 0; i + 1 < num_t; ++i) {
        double mean_prev = 0.0, mean_back = 0.0;
        for (int64_t j = 0; j < t; ++j) {
            a[j] = (double)xc[i * t + j];
            b[j] = (double)xc[(i + 1) * t + j];
            mean_prev += a[j];
            mean_back += b[j];
        }
        mean_prev /= (double)t;
        mean_back /= (double)t;
        gmm_groups(a, t, g, iters, grp, resp);
        double err = 0.0;
        for (int32_t k = 0; k < g; ++k) {
            double sa = 0.0, sb = 0.0;
            int64_t cnt = 0;
            for (int64_t j = 0; j < t; ++j) {
                if (grp[j] != k) continue;
                sa += a[j];
                sb += b[j];
                ++cnt;
            }
            if (cnt == 0) continue;
            const double rel_prev = sa / (double)cnt - mean_prev;
            const double rel_back = sb / (double)cnt - mean_back;
            err += (double)cnt * smape(rel_prev, rel_back);
        }
        total += err / (double)t;
    }
    free(a); free(b); free(grp); free(resp);
    return total / (double)(num_t - 1);
}

int oracle_pd_similarity(const oracle_pd_params* p, const oracle_pd_similarity_params* sp,
                         const float* x, const int64_t* w, const int32_t* t, int64_t count,
                         double* err_out) {
    if (check_params(p) || !sp || !x || (count > 0 && (!w || !t || !err_out))) return -1;
    if (sp->num_groups < 1 || sp->num_groups > 64 || sp->em_iters < 0) return -1;
    for (int64_t k = 0; k < count; ++k)
        if (w[k] < 0 || w[k] >= p->num_windows || t[k] < 1 || (int64_t)t[k] > p->n) return -1;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t k = 0; k < count; ++k) {
        const float* xw = x + w[k] * p->window_stride;
        double wsum = 0.0, acc = 0.0;
        int undefined = 0;
        for (int32_t c = 0; c < p->num_channels; ++c) {
            const double e = similarity_one(xw + (int64_t)c * p->channel_stride, p->n, t[k],
                                            sp->num_groups, sp->em_iters);
            if (e == -2.0) bad = 1;
            if (e < 0.0) undefined = 1;
            const double wc = weight_of(p->channel_weights, c);
            acc += wc * e;
            wsum += wc;
        }
        err_out[k] = undefined ? -1.0 : acc / wsum;
    }
    return bad ? -1 : 0;
}

int oracle_pd_threads(void) { return omp_get_max_threads(); }
