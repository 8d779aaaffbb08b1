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
// One workgroup of kWaves wavefronts per (window, lag) query: wavefront v takes
// the pairs i = v, v + kWaves, ...; its lanes stride over the samples of a
// sub-curve, and every sum is a per-lane partial sum combined by a fixed
// shuffle tree, so all lanes hold the same mixture parameters.  The pair
// errors of the wavefronts are added in wavefront order.
#include <cmath>

#include "internal.h"

namespace gpoeo {
namespace {

constexpr int kMaxGroups = 8;
constexpr int kWaves = 4;

__device__ __forceinline__ double wave_sum(double v) {
    for (int off = 32; off > 0; off >>= 1) v = v + __shfl_down(v, off);
    return __shfl(v, 0);
}
__device__ __forceinline__ double wave_min(double v) {
    for (int off = 32; off > 0; off >>= 1) v = fmin(v, __shfl_down(v, off));
    return __shfl(v, 0);
}
__device__ __forceinline__ double wave_max(double v) {
    for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_down(v, off));
    return __shfl(v, 0);
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
    int64_t count;
    int64_t num_windows;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t num_channels;
    int32_t groups;
    int32_t iters;
};

template <int G>
__device__ double pair_error(const float* __restrict__ a, const float* __restrict__ b, int64_t t,
                             int32_t iters, int lane) {
    const double two_pi = 6.283185307179586;
    double s_a = 0.0, s_b = 0.0, lo = INFINITY, hi = -INFINITY;
    for (int64_t j = lane; j < t; j += kWave) {
        const double va = (double)a[j], vb = (double)b[j];
        s_a += va;
        s_b += vb;
        lo = fmin(lo, va);
        hi = fmax(hi, va);
    }
    const double mean_prev = wave_sum(s_a) / (double)t;
    const double mean_back = wave_sum(s_b) / (double)t;
    lo = wave_min(lo);
    hi = wave_max(hi);

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
#pragma unroll
            for (int k = 0; k < G; ++k) {
                lp[k] = log(pi[k]) - 0.5 * log(two_pi * var[k]);
                h[k] = 0.5 / var[k];
            }
            // responsibilities of the current parameters, normalised per
            // sample: exp(l_k - max_k l_k), so the largest term is exactly 1
            // and only the other G - 1 need an exponential
            auto resp = [&](double v, double (&r)[G]) {
                double best = -INFINITY;
                int top = 0;
#pragma unroll
                for (int k = 0; k < G; ++k) {
                    const double d = v - mu[k];
                    r[k] = lp[k] - d * d * h[k];
                    if (r[k] > best) {
                        best = r[k];
                        top = k;
                    }
                }
                double sum = 1.0;
#pragma unroll
                for (int k = 0; k + 1 < G; ++k) {   // the k-th component other than top
                    const int idx = k < top ? k : k + 1;
                    double val = r[0];
#pragma unroll
                    for (int m = 1; m < G; ++m) val = idx == m ? r[m] : val;
                    const double e = exp(val - best);
                    sum += e;
#pragma unroll
                    for (int m = 0; m < G; ++m) r[m] = idx == m ? e : r[m];
                }
                const double inv = 1.0 / sum;
#pragma unroll
                for (int k = 0; k < G; ++k) r[k] = k == top ? inv : r[k] * inv;
            };
            // One pass: responsibility-weighted count, first and second moment
            // about the sub-curve mean c; the M-step's variance about the new
            // mean m_k is then sum r (x-c)^2 / n_k - (m_k - c)^2 (the same value
            // as a second pass about m_k, up to rounding).
            double nk[G], s1[G], s2[G];
#pragma unroll
            for (int k = 0; k < G; ++k) nk[k] = s1[k] = s2[k] = 0.0;
            for (int64_t j = lane; j < t; j += kWave) {
                const double v = (double)a[j];
                const double d = v - mean_prev;
                double r[G];
                resp(v, r);
#pragma unroll
                for (int k = 0; k < G; ++k) {
                    nk[k] += r[k];
                    s1[k] += r[k] * d;
                    s2[k] += r[k] * d * d;
                }
            }
#pragma unroll
            for (int k = 0; k < G; ++k) {
                nk[k] = wave_sum(nk[k]);
                s1[k] = wave_sum(s1[k]);
                s2[k] = wave_sum(s2[k]);
                if (!(nk[k] > 0.0)) continue;
                const double dm = s1[k] / nk[k];
                mu[k] = mean_prev + dm;
                var[k] = s2[k] / nk[k] - dm * dm;
                if (var[k] < floor_var) var[k] = floor_var;
                pi[k] = nk[k] / (double)t;
            }
        }
    }
    // hard groups and their sums on both sub-curves
    double ga[G], gb[G], gc[G];
#pragma unroll
    for (int k = 0; k < G; ++k) ga[k] = gb[k] = gc[k] = 0.0;
    double lp[G], h[G];
    if (!constant) {
#pragma unroll
        for (int k = 0; k < G; ++k) {
            lp[k] = log(pi[k]) - 0.5 * log(two_pi * var[k]);
            h[k] = 0.5 / var[k];
        }
    }
    for (int64_t j = lane; j < t; j += kWave) {
        const double va = (double)a[j], vb = (double)b[j];
        int arg = 0;
        if (!constant) {
            double best = -INFINITY;
#pragma unroll
            for (int k = 0; k < G; ++k) {
                const double d = va - mu[k];
                const double l = lp[k] - d * d * h[k];
                if (l > best) {
                    best = l;
                    arg = k;
                }
            }
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
    double err = 0.0;
#pragma unroll
    for (int k = 0; k < G; ++k) {
        const double ca = wave_sum(ga[k]), cb = wave_sum(gb[k]), cnt = wave_sum(gc[k]);
        if (cnt == 0.0) continue;
        err += cnt * smape(ca / cnt - mean_prev, cb / cnt - mean_back);
    }
    return err / (double)t;
}

template <int G>
__global__ __launch_bounds__(kWave * kWaves) void similarity_kernel(SimArgs a, Weights w) {
    __shared__ double part[kWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t q = blockIdx.x;
    const int64_t win = a.windows[q];
    const int64_t t = a.lags[q];
    if (win < 0 || win >= a.num_windows || t < 1 || t > a.n) {
        if (threadIdx.x == 0) a.err[q] = NAN;
        return;
    }
    const int64_t num_t = a.n / t;
    if (num_t < 2) {
        if (threadIdx.x == 0) a.err[q] = -1.0;
        return;
    }
    double acc = 0.0, wsum = 0.0;
    for (int32_t c = 0; c < a.num_channels; ++c) {
        const float* xc = a.x + win * a.window_stride + (int64_t)c * a.channel_stride;
        double mine = 0.0;
        for (int64_t i = wave; i + 1 < num_t; i += kWaves)
            mine += pair_error<G>(xc + i * t, xc + (i + 1) * t, t, a.iters, lane);
        if (lane == 0) part[wave] = mine;
        __syncthreads();
        double total = 0.0;
        for (int v = 0; v < kWaves; ++v) total += part[v];
        __syncthreads();
        const double wc = (double)w.w[c];
        acc += wc * (total / (double)(num_t - 1));
        wsum += wc;
    }
    if (threadIdx.x == 0) a.err[q] = acc / wsum;
}

template <int G>
void launch_g(const SimArgs& a, const Weights& w, hipStream_t s) {
    hipLaunchKernelGGL(similarity_kernel<G>, dim3((unsigned)a.count), dim3(kWave * kWaves), 0, s,
                       a, w);
}

}  // namespace

hipError_t launch_similarity(const Plan& p, const Weights& w, int32_t groups, int32_t iters,
                             const float* x, const int32_t* windows, const int32_t* lags,
                             int64_t count, double* err, hipStream_t s) {
    SimArgs a;
    a.x = x;
    a.windows = windows;
    a.lags = lags;
    a.err = err;
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
