// Feature sequence similarity (Algorithm 2, Sec. 4.1.2) for finalist lags.
//
// For a window and a candidate period T the trace is cut into Num_T = floor(N/T)
// sub-curves of T samples.  For every adjacent pair (Smp_i, Smp_{i+1}) the
// samples of Smp_i are grouped by a 1-D Gaussian mixture (num_groups
// components, em_iters EM iterations in fp64, then each sample to its most
// responsible component; means initialised evenly over [min, max], variances
// ((max-min)/G)^2 with a floor of 1e-6 times that, weights 1/G; a component
// without responsibility keeps its parameters; a constant sub-curve is one
// group).  Each group's mean relative to its sub-curve's mean is compared with
// the mean of the same sample indices of Smp_{i+1} (relative to that
// sub-curve's mean) by SMAPE(a, b) = |a-b| / ((|a|+|b|)/2), 0/0 := 0; the
// group-size weighted average is err_i, and Err_T is the mean of err_i over
// the pairs, then the weighted mean over channels.  Err_T = -1 when Num_T < 2.
//
// Work mapping.  One workgroup of kThreads lanes per (window, lag) query.  The
// lanes form segments of S lanes (S a power of two, 1..64, chosen per query
// from T and the number of pairs so that the segments stay busy): segment g
// takes the pairs g, g + kThreads/S, ...; its lanes stride over the samples of
// a sub-curve and combine their partial sums with a butterfly of lane
// shuffles inside the segment, so every lane of a segment holds the same
// mixture parameters.  Short periods (many pairs) run one pair per lane with
// no shuffles at all; long ones spread a pair over up to a wavefront.  Each
// segment adds its pair errors in pair order, and the segments' sums are added
// in segment order, so the result does not depend on scheduling.  Queries are
// dealt to the XCDs in contiguous ranges, so the queries of one window (which
// callers list together) share that XCD's L2.
//
// Arithmetic.  The E-step works with base-2 log-densities
//   l_k(v) = log2 pi_k - log2(2 pi var_k) / 2 - (v - mu_k)^2 log2(e) / (2 var_k),
// responsibilities 2^(l_k - max_j l_j) / sum (gmm_exp2_nonpos, a reciprocal
// refined by two Newton steps), and accumulates the responsibility-weighted
// count and first and second moments about the sub-curve mean in one pass;
// the M-step's variance about the new mean follows from them.  These differ
// from the definition's natural-log, divide-and-two-pass evaluation only by
// roundings, which move the fitted parameters by a few 1e-13 relative at most
// (measured between fp64 evaluation orders on the 1024-trace workload).
//
// Fragile labels.  Err depends on the parameters only through the hard
// labels.  For every sample the final pass compares the margin between the
// two largest log-densities with the change that a relative error of
// kParamRel in each fitted parameter (mu, var, pi) can cause in each of them,
// plus their own rounding; a sample whose label such errors could flip marks
// its query GPOEO_PD_UNRESOLVED in the optional flags output.
#include <cmath>

#include "gmm_math.h"
#include "internal.h"

namespace gpoeo {
namespace {

constexpr int kMaxGroups = 8;
constexpr int kThreads = 256;
// Relative parameter error assumed by the label margin test: 25 times the
// largest difference measured between fp64 evaluation orders of the EM.
constexpr double kParamRel = 1e-11;
constexpr double kLog2e = 1.4426950408889634;
constexpr double kTwoPi = 6.283185307179586;

// Butterfly sums over the S lanes of a segment (S a power of two <= 64,
// segments aligned within the wavefront); every lane ends with the same value.
__device__ __forceinline__ double seg_sum(double v, int s) {
    for (int o = s >> 1; o > 0; o >>= 1) v = v + __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ double seg_min(double v, int s) {
    for (int o = s >> 1; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ double seg_max(double v, int s) {
    for (int o = s >> 1; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
    return v;
}

// 1/x for x in [1, G] (a sum of responsibilities, the largest one 1): the
// hardware estimate refined by two Newton steps.
__device__ __forceinline__ double recip(double x) {
    double r = __builtin_amdgcn_rcp(x);
    r = fma(fma(-x, r, 1.0), r, r);
    r = fma(fma(-x, r, 1.0), r, r);
    return r;
}

__device__ __forceinline__ double smape(double a, double b) {
    const double den = (fabs(a) + fabs(b)) / 2.0;
    return den == 0.0 ? 0.0 : fabs(a - b) / den;
}

struct SimArgs {
    const float* x;
    const int32_t* windows;
    const int32_t* lags;
    double* err;
    uint32_t* flags;         // nullable
    int64_t count;
    int64_t num_windows;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t num_channels;
    int32_t groups;
    int32_t iters;
};

// Segment width for a query: the S that minimises the pair rounds times the
// sample steps of a round (plus a per-round allowance for the parameter
// updates and the shuffles).  Every lane computes the same value.
__device__ __forceinline__ int choose_segment(int64_t pairs, int64_t t) {
    int best_s = 1;
    double best = INFINITY;
    for (int s = 1, lg = 0; s <= kWave; s <<= 1, ++lg) {
        const int64_t per_round = kThreads / s;
        const int64_t rounds = (pairs + per_round - 1) / per_round;
        const double cost = (double)rounds * ((double)((t + s - 1) / s) + 3.0 + 0.3 * lg);
        if (cost < best) {
            best = cost;
            best_s = s;
        }
    }
    return best_s;
}

// Base-2 log-density coefficients of the current parameters.
template <int G>
__device__ __forceinline__ void log_coeffs(const double (&mu)[G], const double (&var)[G],
                                           const double (&pi)[G], double (&lp)[G],
                                           double (&h)[G]) {
    (void)mu;
#pragma unroll
    for (int k = 0; k < G; ++k) {
        lp[k] = log2(pi[k]) - 0.5 * log2(kTwoPi * var[k]);
        h[k] = (0.5 * kLog2e) / var[k];
    }
}

// Err_i of the pair (a, b) of sub-curves of t samples, computed by the s lanes
// of a segment (this lane is number ls); also whether a hard label is fragile.
template <int G>
__device__ double pair_error(const float* __restrict__ a, const float* __restrict__ b, int64_t t,
                             int32_t iters, int s, int ls, bool& fragile) {
    double s_a = 0.0, s_b = 0.0, lo = INFINITY, hi = -INFINITY;
    for (int64_t j = ls; j < t; j += s) {
        const double va = (double)a[j], vb = (double)b[j];
        s_a += va;
        s_b += vb;
        lo = fmin(lo, va);
        hi = fmax(hi, va);
    }
    s_a = seg_sum(s_a, s);
    s_b = seg_sum(s_b, s);
    lo = seg_min(lo, s);
    hi = seg_max(hi, s);
    const double mean_prev = s_a / (double)t;
    const double mean_back = s_b / (double)t;

    double mu[G], var[G], pi[G];
    const bool constant = hi == lo;
    if (!constant) {
        const double width = (hi - lo) / (double)G;
        const double floor_var = 1e-6 * width * width;
#pragma unroll
        for (int k = 0; k < G; ++k) {
            mu[k] = lo + ((double)k + 0.5) * width;
            var[k] = width * width;
            pi[k] = 1.0 / (double)G;
        }
        for (int32_t it = 0; it < iters; ++it) {
            double lp[G], h[G];
            log_coeffs<G>(mu, var, pi, lp, h);
            double nk[G], s1[G], s2[G];
#pragma unroll
            for (int k = 0; k < G; ++k) nk[k] = s1[k] = s2[k] = 0.0;
            for (int64_t j = ls; j < t; j += s) {
                const double v = (double)a[j];
                double l[G], best = -INFINITY;
#pragma unroll
                for (int k = 0; k < G; ++k) {
                    const double d = v - mu[k];
                    l[k] = fma(-(d * d), h[k], lp[k]);
                    best = fmax(best, l[k]);
                }
                double e[G], sum = 0.0;
#pragma unroll
                for (int k = 0; k < G; ++k) {
                    e[k] = gmm_exp2_nonpos(l[k] - best);
                    sum += e[k];
                }
                const double inv = recip(sum);
                const double dd = v - mean_prev;
#pragma unroll
                for (int k = 0; k < G; ++k) {
                    const double r = e[k] * inv;
                    const double rd = r * dd;
                    nk[k] += r;
                    s1[k] += rd;
                    s2[k] = fma(rd, dd, s2[k]);
                }
            }
#pragma unroll
            for (int k = 0; k < G; ++k) {
                nk[k] = seg_sum(nk[k], s);
                s1[k] = seg_sum(s1[k], s);
                s2[k] = seg_sum(s2[k], s);
                if (!(nk[k] > 0.0)) continue;
                const double dm = s1[k] / nk[k];
                mu[k] = mean_prev + dm;
                var[k] = s2[k] / nk[k] - dm * dm;
                if (var[k] < floor_var) var[k] = floor_var;
                pi[k] = nk[k] / (double)t;
            }
        }
    }
    // hard groups, their sums on both sub-curves (in the order of the sums of
    // the means above, so a single group reproduces them exactly), and the
    // label margins
    double ga[G], gb[G], gc[G];
#pragma unroll
    for (int k = 0; k < G; ++k) ga[k] = gb[k] = gc[k] = 0.0;
    double lp[G], h[G];
    if (!constant) log_coeffs<G>(mu, var, pi, lp, h);
    double frag = 0.0;
    for (int64_t j = ls; j < t; j += s) {
        const double va = (double)a[j], vb = (double)b[j];
        int arg = 0;
        if (!constant && G > 1) {
            double l[G], e[G];
#pragma unroll
            for (int k = 0; k < G; ++k) {
                const double d = va - mu[k];
                const double q = d * d * h[k];
                l[k] = lp[k] - q;
                // change of l_k under relative errors kParamRel of mu_k, var_k
                // and pi_k, plus four roundings of its terms
                e[k] = kParamRel * (2.0 * fabs(d) * fabs(mu[k]) * h[k] + q + 1.5 * kLog2e) +
                       1e-15 * (fabs(lp[k]) + q);
            }
            double best = l[0], eb = e[0];
#pragma unroll
            for (int k = 1; k < G; ++k)
                if (l[k] > best) {
                    best = l[k];
                    eb = e[k];
                    arg = k;
                }
            double gap = INFINITY;
#pragma unroll
            for (int k = 0; k < G; ++k)
                if (k != arg && best - l[k] <= eb + e[k]) gap = 0.0;
            if (gap == 0.0) frag = 1.0;
        }
#pragma unroll
        for (int k = 0; k < G; ++k) {
            if (k == arg) {
                ga[k] += va;
                gb[k] += vb;
                gc[k] += 1.0;
            }
        }
    }
    if (seg_max(frag, s) > 0.0) fragile = true;
    double err = 0.0;
#pragma unroll
    for (int k = 0; k < G; ++k) {
        const double ca = seg_sum(ga[k], s), cb = seg_sum(gb[k], s), cnt = seg_sum(gc[k], s);
        if (cnt == 0.0) continue;
        err += cnt * smape(ca / cnt - mean_prev, cb / cnt - mean_back);
    }
    return err / (double)t;
}

template <int G>
__global__ __launch_bounds__(kThreads) void similarity_kernel(SimArgs a, Weights w) {
    __shared__ double part[kThreads];
    __shared__ int any_fragile;
    const int tid = threadIdx.x;
    // contiguous query ranges per XCD (workgroups are dealt to the 8 XCDs in turn)
    const int64_t groups = gridDim.x;
    int64_t q = blockIdx.x;
    const int64_t full = groups - groups % 8;
    if (q < full) q = (q % 8) * (full / 8) + q / 8;
    const int64_t win = a.windows[q];
    const int64_t t = a.lags[q];
    if (win < 0 || win >= a.num_windows || t < 1 || t > a.n) {
        if (tid == 0) {
            a.err[q] = NAN;
            if (a.flags) a.flags[q] = 0u;
        }
        return;
    }
    const int64_t num_t = a.n / t;
    if (num_t < 2) {
        if (tid == 0) {
            a.err[q] = -1.0;
            if (a.flags) a.flags[q] = 0u;
        }
        return;
    }
    const int64_t pairs = num_t - 1;
    const int s = choose_segment(pairs, t);
    const int seg = tid / s, ls = tid % s, nseg = kThreads / s;
    if (tid == 0) any_fragile = 0;
    bool fragile = false;
    double acc = 0.0, wsum = 0.0;
    for (int32_t c = 0; c < a.num_channels; ++c) {
        const float* xc = a.x + win * a.window_stride + (int64_t)c * a.channel_stride;
        double mine = 0.0;
        for (int64_t i = seg; i < pairs; i += nseg)
            mine += pair_error<G>(xc + i * t, xc + (i + 1) * t, t, a.iters, s, ls, fragile);
        __syncthreads();
        if (ls == 0) part[seg] = mine;
        __syncthreads();
        double total = 0.0;
        for (int g = 0; g < nseg; ++g) total += part[g];
        const double wc = (double)w.w[c];
        acc += wc * (total / (double)pairs);
        wsum += wc;
    }
    if (fragile) any_fragile = 1;
    __syncthreads();
    if (tid == 0) {
        a.err[q] = acc / wsum;
        if (a.flags) a.flags[q] = any_fragile ? GPOEO_PD_UNRESOLVED : 0u;
    }
}

template <int G>
void launch_g(const SimArgs& a, const Weights& w, hipStream_t s) {
    hipLaunchKernelGGL(similarity_kernel<G>, dim3((unsigned)a.count), dim3(kThreads), 0, s, a, w);
}

}  // namespace

hipError_t launch_similarity(const Plan& p, const Weights& w, int32_t groups, int32_t iters,
                             const float* x, const int32_t* windows, const int32_t* lags,
                             int64_t count, double* err, uint32_t* flags, hipStream_t s) {
    SimArgs a;
    a.x = x;
    a.windows = windows;
    a.lags = lags;
    a.err = err;
    a.flags = flags;
    a.count = count;
    a.num_windows = p.num_windows;
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    a.groups = groups;
    a.iters = iters;
    switch (groups) {
        case 1: launch_g<1>(a, w, s); break;
        case 2: launch_g<2>(a, w, s); break;
        case 3: launch_g<3>(a, w, s); break;
        case 4: launch_g<4>(a, w, s); break;
        case 5: launch_g<5>(a, w, s); break;
        case 6: launch_g<6>(a, w, s); break;
        case 7: launch_g<7>(a, w, s); break;
        default: launch_g<kMaxGroups>(a, w, s); break;
    }
    return hipGetLastError();
}

}  // namespace gpoeo
