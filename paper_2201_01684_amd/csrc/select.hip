// Period selection per window (Algorithm 1 of Sec. 4.1.2, in the lag domain),
// with exact re-decision of every comparison the score error bound leaves open.
//
// Rule (one workgroup per window):
//   R      = 2 * sum_c w_c * Var_c; R == 0 -> CONSTANT
//   peaks  = { Tmin < T < Tmax : S(T) < S(T-1) and S(T) <= S(T+1) }
//            (Algorithm 1's "find peaks": interior local minima of the score;
//            strict on the left so a flat bottom contributes its first lag)
//   S_pk   = min S over peaks; thr = R - c_lag * (R - S_pk)
//            (candidate filter "peak > c_peak * max peak" on the height 1 - S/R)
//   T_c    = smallest peak with S(T) < thr (the fundamental; the spectrum of a
//            periodic signal has no component at multiples of its period)
//   window = [max(Tmin, ceil(T_c D / (D + T_c))), min(Tmax, floor(T_c D / (D - T_c)))],
//            D = N - 1: the periods of the two neighbouring Fourier bins of
//            T_c = D / k, i.e. Algorithm 1's local search at a one-sample step
//   period = smallest T in the window attaining min S; err = S(period) / R
//
// Each score comes from the score kernels with a relative error bound
// (kScoreRelBound), so it is handled as the interval [v(1-e), v(1+e)] that
// contains the value a plain sequential fp64 evaluation gives.  A comparison
// the intervals decide is final.  Otherwise the lags involved (and R, when the
// threshold or err is involved) are recomputed here as plain sequential fp64
// sums in ascending index order with no fused multiply-add, which makes them
// exact points, and the rule runs again.  The number of passes is bounded; if
// the bound is reached the last pass decides on the unwidened values and the
// window is flagged GPOEO_PD_UNRESOLVED.
#include "internal.h"
#include "gpoeo_pd.h"

namespace gpoeo {
namespace {

constexpr int kThreads = 256;
constexpr int kNeedCap = 512;
constexpr int kMaxPasses = 24;

struct SelectArgs {
    const float* x;
    const double* var;       // [B][C]
    double* s64;             // [B][L], overwritten in place by exact re-scores
    uint32_t* bits;          // [B][bitmap_words], 1 = exact value in s64
    gpoeo_pd_result* results;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t num_channels;
    int32_t tmin, tmax, lags, words;
    double c_lag, err_max;
    uint32_t flags;
};

enum Tri : int { kNo = 0, kYes = 1, kUnk = 2 };

struct Iv {
    double lo, hi, v;
    bool exact;
};

__device__ __forceinline__ Tri lt(const Iv& a, const Iv& b) {
    if (a.hi < b.lo) return kYes;
    if (a.lo >= b.hi) return kNo;
    return kUnk;
}
__device__ __forceinline__ Tri le(const Iv& a, const Iv& b) {
    if (a.hi <= b.lo) return kYes;
    if (a.lo > b.hi) return kNo;
    return kUnk;
}

// Plain sequential fp64 evaluation of S(T), ascending i, no contraction.
__device__ double exact_score(const float* __restrict__ xw, int32_t num_channels,
                              int64_t channel_stride, int64_t n, int64_t t, const Weights& w) {
#pragma clang fp contract(off)
    double s = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* __restrict__ xc = xw + (int64_t)c * channel_stride;
        double dsum = 0.0;
        const int64_t m = n - t;
        int64_t i = 0;
        for (; i + 4 <= m; i += 4) {
            const float a0 = xc[i], a1 = xc[i + 1], a2 = xc[i + 2], a3 = xc[i + 3];
            const float b0 = xc[i + t], b1 = xc[i + t + 1], b2 = xc[i + t + 2],
                        b3 = xc[i + t + 3];
            double d;
            d = (double)a0 - (double)b0; dsum = dsum + d * d;
            d = (double)a1 - (double)b1; dsum = dsum + d * d;
            d = (double)a2 - (double)b2; dsum = dsum + d * d;
            d = (double)a3 - (double)b3; dsum = dsum + d * d;
        }
        for (; i < m; ++i) {
            const double d = (double)xc[i] - (double)xc[i + t];
            dsum = dsum + d * d;
        }
        s = s + (double)w.w[c] * (dsum / (double)m);
    }
    return s;
}

// Plain sequential fp64 evaluation of R = 2 * sum_c w_c * Var_c (two passes).
__device__ double exact_reference(const float* __restrict__ xw, int32_t num_channels,
                                  int64_t channel_stride, int64_t n, const Weights& w) {
#pragma clang fp contract(off)
    double acc = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* __restrict__ xc = xw + (int64_t)c * channel_stride;
        double sum = 0.0;
        for (int64_t i = 0; i < n; ++i) sum = sum + (double)xc[i];
        const double mean = sum / (double)n;
        double sq = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            const double d = (double)xc[i] - mean;
            sq = sq + d * d;
        }
        acc = acc + (double)w.w[c] * (sq / (double)n);
    }
    return 2.0 * acc;
}

struct Shared {
    double red_d[kThreads];
    double red_d2[kThreads];
    int64_t red_i[kThreads];
    int64_t red_j[kThreads];
    int32_t need[kNeedCap];
    int need_count;
    int need_r;
    int need_pk;
    int rescored;
    double r_lo, r_hi, r_v;
    int r_exact;
};

__device__ double block_min_d(double v, double* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] = fmin(red[threadIdx.x], red[threadIdx.x + w]);
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}

__device__ int64_t block_sum_i(int64_t v, int64_t* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    const int64_t r = red[0];
    __syncthreads();
    return r;
}

__device__ int64_t block_min_i(int64_t v, int64_t* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] = min(red[threadIdx.x], red[threadIdx.x + w]);
        __syncthreads();
    }
    const int64_t r = red[0];
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a, Weights w) {
    __shared__ Shared sh;
    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int32_t tmin = a.tmin, tmax = a.tmax;
    double* __restrict__ s = a.s64 + b * (int64_t)a.lags;
    uint32_t* __restrict__ bits = a.bits + b * (int64_t)a.words;
    const float* __restrict__ xw = a.x + b * a.window_stride;
    gpoeo_pd_result* res = a.results + b;

    for (int32_t k = tid; k < a.words; k += kThreads) bits[k] = 0u;
    if (tid == 0) {
        double acc = 0.0;
        for (int32_t c = 0; c < a.num_channels; ++c)
            acc += (double)w.w[c] * a.var[b * a.num_channels + c];
        sh.r_v = 2.0 * acc;
        sh.r_exact = 0;
        sh.rescored = 0;
    }
    __syncthreads();
    const double r_approx = sh.r_v;
    if (r_approx == 0.0) {   // every weighted channel constant (exact: see window_stats)
        if (tid == 0) {
            gpoeo_pd_result o = {};
            o.verdict = GPOEO_PD_CONSTANT;
            *res = o;
        }
        return;
    }

    const bool rescue = (a.flags & GPOEO_PD_NO_RESCUE) == 0;
    bool unresolved = false;
    const double c_lag = a.c_lag;

    for (int pass = 0;; ++pass) {
        const bool last = !rescue || pass == kMaxPasses;
        if (rescue && pass == kMaxPasses) unresolved = true;
        const double tau = last ? 0.0 : kScoreRelBound;
        const double tau_r = last ? 0.0 : kRefRelBound;
        if (tid == 0) {
            sh.need_count = 0;
            sh.need_r = 0;
            sh.need_pk = 0;
            if (sh.r_exact) {
                sh.r_lo = sh.r_hi = sh.r_v;
            } else {
                sh.r_lo = r_approx * (1.0 - tau_r);
                sh.r_hi = r_approx * (1.0 + tau_r);
                sh.r_v = r_approx;
            }
        }
        __syncthreads();
        const double r_lo = sh.r_lo, r_hi = sh.r_hi, r_v = sh.r_v;

        auto iv = [&](int64_t t) -> Iv {
            const int64_t j = t - tmin;
            const double v = s[j];
            const bool ex = (bits[j >> 5] >> (j & 31)) & 1u;
            Iv r;
            r.v = v;
            r.exact = ex;
            if (ex) {
                r.lo = r.hi = v;
            } else {
                r.lo = v * (1.0 - tau);
                r.hi = v * (1.0 + tau);
            }
            return r;
        };
        auto push = [&](int64_t t, const Iv& z) {
            if (z.exact || last) return;
            const int k = atomicAdd(&sh.need_count, 1);
            if (k < kNeedCap) sh.need[k] = (int32_t)t;
        };
        // peak status of T: kYes / kNo / kUnk (and pushes the lags of an open test)
        auto peak = [&](int64_t t, Iv& z, bool do_push) -> Tri {
            const Iv m = iv(t - 1);
            z = iv(t);
            const Iv p = iv(t + 1);
            const Tri t1 = lt(z, m), t2 = le(z, p);
            if (t1 == kNo || t2 == kNo) return kNo;
            if (t1 == kYes && t2 == kYes) return kYes;
            if (do_push) {
                push(t - 1, m);
                push(t, z);
                push(t + 1, p);
            }
            return kUnk;
        };

        gpoeo_pd_result o = {};
        bool done = false;
        do {
            // 1. peaks.  An open local-minimum test only matters for a lag that
            // could be a candidate (S < thr) or the smallest peak; thr is at most
            // thr(R_hi, min hi over decided peaks), so open tests of lags whose
            // lower bound lies above that (and above the smallest decided peak)
            // are left open.
            int64_t npk = 0, unk = 0;
            double pk_lo = INFINITY, pk_hi = INFINITY, unk_lo = INFINITY;
            for (int64_t t = tmin + 1 + tid; t < tmax; t += kThreads) {
                Iv z;
                const Tri q = peak(t, z, false);
                if (q == kYes) {
                    ++npk;
                    pk_lo = fmin(pk_lo, z.lo);
                    pk_hi = fmin(pk_hi, z.hi);
                } else if (q == kUnk) {
                    ++unk;
                    unk_lo = fmin(unk_lo, z.lo);
                }
            }
            unk = block_sum_i(unk, sh.red_i);
            npk = block_sum_i(npk, sh.red_j);
            pk_lo = block_min_d(pk_lo, sh.red_d);
            pk_hi = block_min_d(pk_hi, sh.red_d2);
            unk_lo = block_min_d(unk_lo, sh.red_d);
            if (unk > 0) {
                const double pad = 4.0 * 2.220446049250313e-16 * r_hi;
                const double cut =
                    npk > 0 ? fmax(r_hi - c_lag * (r_hi - pk_hi) + pad, pk_hi) : INFINITY;
                if (unk_lo < cut) {
                    for (int64_t t = tmin + 1 + tid; t < tmax; t += kThreads) {
                        Iv z;
                        if (peak(t, z, false) == kUnk && z.lo < cut) peak(t, z, true);
                    }
                    break;
                }
            }
            if (npk == 0) {
                o.verdict = GPOEO_PD_APERIODIC;
                done = true;
                break;
            }
            // 2. threshold and candidates
            double thr_lo, thr_hi;
            if (pk_lo == pk_hi && r_lo == r_hi) {
                thr_lo = thr_hi = r_v - c_lag * (r_v - pk_lo);
            } else {
                const double pad = 4.0 * 2.220446049250313e-16 * r_hi;
                thr_lo = r_lo - c_lag * (r_lo - pk_lo) - pad;
                thr_hi = r_hi - c_lag * (r_hi - pk_hi) + pad;
            }
            Iv thr;
            thr.lo = thr_lo;
            thr.hi = thr_hi;
            thr.v = 0.5 * (thr_lo + thr_hi);
            thr.exact = thr_lo == thr_hi;
            int64_t ncand = 0, tc = INT64_MAX;
            unk = 0;
            for (int64_t t = tmin + 1 + tid; t < tmax; t += kThreads) {
                Iv z;
                if (peak(t, z, false) != kYes) continue;
                const Tri q = lt(z, thr);
                if (q == kYes) {
                    ++ncand;
                    tc = min(tc, t);
                } else if (q == kUnk) {
                    ++unk;
                    push(t, z);
                }
            }
            unk = block_sum_i(unk, sh.red_i);
            ncand = block_sum_i(ncand, sh.red_j);
            tc = block_min_i(tc, sh.red_i);
            if (unk > 0) {
                // the threshold itself must become exact: R and every peak that
                // can be the smallest one
                if (r_lo != r_hi && tid == 0) sh.need_r = 1;
                if (pk_lo != pk_hi) {
                    for (int64_t t = tmin + 1 + tid; t < tmax; t += kThreads) {
                        Iv z;
                        if (peak(t, z, false) == kYes && z.lo <= pk_hi) push(t, z);
                    }
                }
                break;
            }
            o.n_candidates = (int32_t)ncand;
            if (ncand == 0) {
                o.verdict = GPOEO_PD_APERIODIC;
                done = true;
                break;
            }
            o.t_cand = (int32_t)tc;
            // 3. local search window
            const int64_t d = a.n - 1;
            int64_t lo = (tc * d + (d + tc) - 1) / (d + tc);
            int64_t hi = (tc * d) / (d - tc);
            lo = max(lo, (int64_t)tmin);
            hi = min(hi, (int64_t)tmax);
            o.t_low = (int32_t)lo;
            o.t_up = (int32_t)hi;
            double m_hi = INFINITY;
            for (int64_t t = lo + tid; t <= hi; t += kThreads) m_hi = fmin(m_hi, iv(t).hi);
            m_hi = block_min_d(m_hi, sh.red_d);
            int64_t ncont = 0, nopen = 0, tbest = INT64_MAX;
            for (int64_t t = lo + tid; t <= hi; t += kThreads) {
                const Iv z = iv(t);
                if (z.lo <= m_hi) {
                    ++ncont;
                    if (!z.exact) ++nopen;
                    tbest = min(tbest, t);
                }
            }
            ncont = block_sum_i(ncont, sh.red_i);
            nopen = block_sum_i(nopen, sh.red_j);
            tbest = block_min_i(tbest, sh.red_i);
            if (ncont > 1 && nopen > 0 && !last) {
                for (int64_t t = lo + tid; t <= hi; t += kThreads) {
                    const Iv z = iv(t);
                    if (z.lo <= m_hi) push(t, z);
                }
                break;
            }
            // One contender is the strict argmin; several exact contenders all
            // equal m_hi, so the smallest lag wins the tie.
            o.period = (int32_t)tbest;
            const Iv z = iv(tbest);
            // 4. err and verdict
            bool aper;
            if ((z.exact && r_lo == r_hi) || last) {
                const double e = z.v / r_v;
                aper = e >= a.err_max;
                o.err = (float)e;
            } else {
                const double e_lo = z.lo / r_hi * (1.0 - 4.0 * 2.220446049250313e-16);
                const double e_hi = z.hi / r_lo * (1.0 + 4.0 * 2.220446049250313e-16);
                if (e_lo >= a.err_max) {
                    aper = true;
                } else if (e_hi < a.err_max) {
                    aper = false;
                } else {
                    if (tid == 0) {
                        push(tbest, z);
                        sh.need_r = 1;
                    }
                    break;
                }
                o.err = (float)(z.v / r_v);
            }
            o.verdict = aper ? GPOEO_PD_APERIODIC : GPOEO_PD_PERIODIC;
            done = true;
        } while (false);

        __syncthreads();
        if (done) {
            if (tid == 0) {
                o.n_rescored = sh.rescored;
                o.flags = unresolved ? GPOEO_PD_UNRESOLVED : 0u;
                *res = o;
            }
            return;
        }
        // Re-score the open lags (and R) as exact points, then run the rule again.
        const int cnt = min(sh.need_count, kNeedCap);
        for (int k = tid; k < cnt; k += kThreads) {
            const int64_t t = sh.need[k];
            const int64_t j = t - tmin;
            if ((bits[j >> 5] >> (j & 31)) & 1u) continue;
            const double v = exact_score(xw, a.num_channels, a.channel_stride, a.n, t, w);
            s[j] = v;
            __threadfence_block();
            const uint32_t old = atomicOr(&bits[j >> 5], 1u << (j & 31));
            if (!((old >> (j & 31)) & 1u)) atomicAdd(&sh.rescored, 1);
        }
        if (sh.need_r && tid == kThreads - 1 && !sh.r_exact) {
            sh.r_v = exact_reference(xw, a.num_channels, a.channel_stride, a.n, w);
            sh.r_exact = 1;
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_select(const Plan& p, const Weights& w, const float* x, const double* var,
                         double* s64, uint32_t* bits, void* results, hipStream_t s) {
    SelectArgs a;
    a.x = x;
    a.var = var;
    a.s64 = s64;
    a.bits = bits;
    a.results = static_cast<gpoeo_pd_result*>(results);
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    a.tmin = p.tmin;
    a.tmax = p.tmax;
    a.lags = p.lags;
    a.words = p.bitmap_words;
    a.c_lag = p.c_lag;
    a.err_max = p.err_max;
    a.flags = p.flags;
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)p.num_windows), dim3(kThreads), 0, s, a, w);
    return hipGetLastError();
}

}  // namespace gpoeo
