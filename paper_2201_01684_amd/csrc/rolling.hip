// Rolling detection (Algorithm 3, Sec. 4.1.3): the schedule of suffix windows
// and the combination of their selections.
//
// The pipeline (launched from api.cpp on one stream):
//   1. the rule on every whole window (the first pass gives T_init);
//   2. rolling_schedule_kernel: per window, Algorithm 3's suffix windows as a
//      window table (offset, length, largest lag), with empty slots;
//   3. the rule on every suffix window of the table (one batch);
//   4. rolling_combine_kernel: per window, the suffix with the smallest err
//      (decided on bounded errs, re-evaluated exactly when the bounds overlap),
//      the relative period spread and the next sampling duration.
// Schedule and combination use the same fp64 expressions as the definition
// (this file is compiled with -ffp-contract=off).
#include "internal.h"
#include "exact.h"
#include "gpoeo_pd.h"

namespace gpoeo {
namespace {

__global__ void rolling_schedule_kernel(const gpoeo_pd_result* __restrict__ res_a,
                                        int64_t num_windows, int64_t n, int64_t window_stride,
                                        int32_t tmin, int32_t tmax, RollingConfig rc,
                                        int64_t* __restrict__ tab_off, int64_t* __restrict__ tab_n,
                                        int32_t* __restrict__ tab_tmax,
                                        RollState* __restrict__ state) {
    const int64_t b = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (b >= num_windows) return;
    const gpoeo_pd_result o = res_a[b];
    RollState st;
    st.err_a = (double)o.err;
    st.short_next = 0.0;
    st.t_init = o.period;
    st.verdict_a = o.verdict;
    st.count = 0;
    st.flags = o.flags & GPOEO_PD_UNRESOLVED;
    const int64_t base = b * (int64_t)rc.jmax;
    for (int32_t j = 0; j < rc.jmax; ++j) {   // empty slots unless filled below
        tab_off[base + j] = b * window_stride;
        tab_n[base + j] = 0;
        tab_tmax[base + j] = tmin;
    }
    if (o.verdict == GPOEO_PD_PERIODIC) {
        const double t = (double)o.period;
        const double dur = (double)(n - 1);
        if (dur < rc.c_measure * t) {
            st.short_next = rc.c_measure * t - dur;
        } else {
            double t_start = dur - (2.0 + rc.c_eval * rc.step) * t;
            if (t_start < 0.0) t_start = 0.0;
            int32_t j = 0;
            while ((dur - t_start) / t >= rc.c_measure) {
                if (j == rc.jmax) {   // cannot happen for the validated parameters
                    st.flags |= GPOEO_PD_UNRESOLVED;
                    break;
                }
                const int64_t start = (int64_t)floor(t_start);
                const int64_t nj = n - start;
                tab_off[base + j] = b * window_stride + start;
                tab_n[base + j] = nj;
                tab_tmax[base + j] = (int32_t)min((int64_t)tmax, nj / 2);
                ++j;
                t_start += rc.step * t;
            }
            st.count = j;
        }
    }
    state[b] = st;
}

// One wavefront per window; lane j handles suffix window j.
__global__ __launch_bounds__(kWave) void rolling_combine_kernel(RollingCombineArgs a, Weights w) {
    const int lane = threadIdx.x;
    const int64_t b = blockIdx.x;
    const RollState st = a.state[b];
    gpoeo_pd_rolling_result* out = a.out + b;
    __shared__ int32_t per_t[GPOEO_PD_ROLLING_MAX];
    __shared__ int32_t per_v[GPOEO_PD_ROLLING_MAX];
    __shared__ double per_e[GPOEO_PD_ROLLING_MAX];
    __shared__ uint32_t per_f[GPOEO_PD_ROLLING_MAX];

    if (st.verdict_a != GPOEO_PD_PERIODIC || st.count == 0) {
        if (lane == 0) {
            gpoeo_pd_rolling_result r = {};
            r.verdict = st.verdict_a;
            r.t_init = st.t_init;
            r.best = -1;
            r.flags = st.flags;
            if (st.verdict_a == GPOEO_PD_PERIODIC) {   // too short for a rolling evaluation
                r.period = st.t_init;
                r.err = (float)st.err_a;
                r.smpdur_next = st.short_next;
            }
            *out = r;
        }
        return;
    }
    const int cnt = st.count;
    const int64_t win = b * (int64_t)a.jmax + lane;
    bool periodic = false;
    int32_t tj = 0;
    double e_lo = INFINITY, e_hi = INFINITY, e_v = 0.0;
    bool s_exact = false, r_exact = false;
    double s_v = 0.0, r_v = 0.0;
    if (lane < cnt) {
        const gpoeo_pd_result rc = a.res_c[win];
        per_f[lane] = rc.flags & GPOEO_PD_UNRESOLVED;
        periodic = rc.verdict == GPOEO_PD_PERIODIC;
        per_v[lane] = rc.verdict;
        tj = periodic ? rc.period : 0;
        per_t[lane] = tj;
        if (periodic) {
            const int64_t j = tj - a.tmin;
            const uint32_t bit = 1u << (j & 31);
            s_v = a.s64[win * a.lags + j];
            double s_lo, s_hi;
            if (a.tier2[win * a.words + (j >> 5)] & bit) {
                s_exact = true;
                s_lo = s_hi = s_v;
            } else {
                const double e =
                    (a.tier1[win * a.words + (j >> 5)] & bit) ? a.tau1 : a.tau0;
                s_lo = s_v * (1.0 - e);
                s_hi = s_v * (1.0 + e);
            }
            double r_lo, r_hi;
            if (a.wstate[win].r_is_exact) {
                r_exact = true;
                r_v = r_lo = r_hi = a.wstate[win].r_exact;
            } else {
                const double* v2 = a.var + 2 * win * a.num_channels;
                double acc = 0.0;
                for (int32_t c = 0; c < a.num_channels; ++c) acc = acc + (double)w.w[c] * v2[2 * c];
                r_v = 2.0 * acc;
                const double er =
                    exact::reference_bound(v2, a.num_channels, a.tab_n[win], w, r_v);
                r_lo = r_v - er;
                r_hi = r_v + er;
            }
            const double ulp4 = 4.0 * 2.220446049250313e-16;
            e_lo = s_lo / r_hi * (1.0 - ulp4);
            e_hi = s_hi / r_lo * (1.0 + ulp4);
            e_v = s_v / r_v;
        }
    }
    // the smallest err among the periodic suffixes, first on ties
    double m_hi = e_hi;
    for (int off = 32; off > 0; off >>= 1) m_hi = fmin(m_hi, __shfl_xor(m_hi, off));
    const bool contender = periodic && e_lo <= m_hi;
    const uint64_t mask = __ballot(contender);
    int best;
    if (__popcll(mask) == 1) {
        best = __ffsll((long long)mask) - 1;
    } else {
        // overlapping bounds: the contenders' errs as plain sequential fp64
        if (contender) {
            const float* xw = a.x + a.tab_off[win];
            const int64_t nw = a.tab_n[win];
            const double s = s_exact ? s_v
                                     : exact::exact_score(xw, a.num_channels, a.channel_stride,
                                                          nw, tj, w);
            const double r = r_exact ? r_v
                                     : exact::exact_reference(xw, a.num_channels,
                                                              a.channel_stride, nw, w);
            e_v = s / r;
        }
        double m = contender ? e_v : INFINITY;
        for (int off = 32; off > 0; off >>= 1) m = fmin(m, __shfl_xor(m, off));
        best = __ffsll((long long)__ballot(contender && e_v == m)) - 1;
    }
    if (lane < cnt) per_e[lane] = e_v;
    __syncthreads();
    if (lane != 0) return;
    gpoeo_pd_rolling_result r = {};
    r.verdict = st.verdict_a;
    r.t_init = st.t_init;
    r.n_windows = cnt;
    r.flags = st.flags;
    int32_t np = 0, t_lo = 0, t_hi = 0;
    double sum = 0.0;
    for (int k = 0; k < cnt; ++k) {
        r.flags |= per_f[k];
        r.periods[k] = per_t[k];
        r.starts[k] = a.tab_off[b * (int64_t)a.jmax + k] - b * a.window_stride;
        if (per_v[k] != GPOEO_PD_PERIODIC) continue;
        if (np == 0 || per_t[k] < t_lo) t_lo = per_t[k];
        if (np == 0 || per_t[k] > t_hi) t_hi = per_t[k];
        sum = sum + (double)per_t[k];
        ++np;
    }
    if (np == 0) {
        r.verdict = GPOEO_PD_APERIODIC;
        r.best = -1;
    } else {
        r.best = best;
        r.period = per_t[best];
        r.err = (float)per_e[best];
        const double diff = fabs(((double)t_hi - (double)t_lo) / (sum / (double)np));
        r.diff = (float)diff;
        const double dur = (double)(a.n - 1);
        if (diff < a.diff_threshold) {
            r.stable = 1;
            r.smpdur_next = -1.0;
        } else {
            r.smpdur_next = ceil(dur / (double)t_hi) * (double)t_hi - dur;
        }
    }
    *out = r;
}

}  // namespace

hipError_t launch_rolling_schedule(const Plan& p, const RollingConfig& rc,
                                   const gpoeo_pd_result* res_a, int64_t* tab_off, int64_t* tab_n,
                                   int32_t* tab_tmax, RollState* state, hipStream_t s) {
    const int64_t groups = (p.num_windows + 255) / 256;
    hipLaunchKernelGGL(rolling_schedule_kernel, dim3((unsigned)groups), dim3(256), 0, s, res_a,
                       p.num_windows, p.n, p.window_stride, p.tmin, p.tmax, rc, tab_off, tab_n,
                       tab_tmax, state);
    return hipGetLastError();
}

hipError_t launch_rolling_combine(const RollingCombineArgs& a, const Weights& w,
                                  int64_t num_windows, hipStream_t s) {
    hipLaunchKernelGGL(rolling_combine_kernel, dim3((unsigned)num_windows), dim3(kWave), 0, s, a,
                       w);
    return hipGetLastError();
}

}  // namespace gpoeo
