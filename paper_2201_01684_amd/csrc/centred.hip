// Mean-removed score S_c(T) at finalist periods (Sec. 4.1.2, Algorithm 2's
// relative values with one group per sample).
//
// For a window and a candidate period T the trace is cut into Num_T =
// floor(N/T) whole sub-curves of T samples; every adjacent pair (i, i+1) is
// compared point by point after each sub-curve's own mean is removed:
//   D_c = sum_{i < Num_T - 1} sum_{j<T} ((x[iT+j] - mu_i) - (x[(i+1)T+j] - mu_{i+1}))^2
//   S_c(T) = sum_c w_c D_c / ((Num_T - 1) T).
// Equivalently SSD - T sum_i (mu_i - mu_{i+1})^2 over the whole-sub-curve
// pairs: a linear drift adds the same amount to every difference of a pair and
// leaves S_c unchanged.  Because removing the means also removes most of a
// short lag's differences, S_c suits re-scoring candidate periods (as
// Algorithm 1 applies Algorithm 2 to its candidates), not an exhaustive scan.
//
// One workgroup of kWaves wavefronts per (window, lag) query; wavefront v takes
// the pairs i = v, v + kWaves, ...; its lanes stride over the T points, every
// sum is a per-lane partial sum combined by a fixed shuffle tree, and the
// wavefront totals are added in wavefront order.  All arithmetic is fp64.
#include "internal.h"

namespace gpoeo {
namespace {

constexpr int kWaves = 4;

__device__ __forceinline__ double wave_sum(double v) {
    for (int off = 32; off > 0; off >>= 1) v = v + __shfl_down(v, off);
    return __shfl(v, 0);
}

struct CentredArgs {
    const float* x;
    const int32_t* windows;
    const int32_t* lags;
    double* out;
    int64_t num_windows;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t num_channels;
};

// Sum over j < t of the squared difference of the mean-removed points of the
// sub-curves a and b, as lane partial sums.
__device__ double pair_sum(const float* __restrict__ a, const float* __restrict__ b, int64_t t,
                           int lane) {
    double sa = 0.0, sb = 0.0;
    for (int64_t j = lane; j < t; j += kWave) {
        sa += (double)a[j];
        sb += (double)b[j];
    }
    const double mu_a = wave_sum(sa) / (double)t;
    const double mu_b = wave_sum(sb) / (double)t;
    double q = 0.0;
    for (int64_t j = lane; j < t; j += kWave) {
        const double d = ((double)a[j] - mu_a) - ((double)b[j] - mu_b);
        q += d * d;
    }
    return wave_sum(q);
}

__global__ __launch_bounds__(kWave * kWaves) void centred_kernel(CentredArgs a, Weights w) {
    __shared__ double part[kWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t q = blockIdx.x;
    const int64_t win = a.windows[q];
    const int64_t t = a.lags[q];
    if (win < 0 || win >= a.num_windows || t < 1 || t > a.n) {
        if (threadIdx.x == 0) a.out[q] = NAN;
        return;
    }
    const int64_t pairs = a.n / t - 1;
    if (pairs < 1) {
        if (threadIdx.x == 0) a.out[q] = -1.0;
        return;
    }
    double acc = 0.0;
    for (int32_t c = 0; c < a.num_channels; ++c) {
        const float* xc = a.x + win * a.window_stride + (int64_t)c * a.channel_stride;
        double mine = 0.0;
        for (int64_t i = wave; i < pairs; i += kWaves) mine += pair_sum(xc + i * t, xc + (i + 1) * t, t, lane);
        if (lane == 0) part[wave] = mine;
        __syncthreads();
        double total = 0.0;
        for (int v = 0; v < kWaves; ++v) total += part[v];
        __syncthreads();
        acc += (double)w.w[c] * (total / (double)(pairs * t));
    }
    if (threadIdx.x == 0) a.out[q] = acc;
}

}  // namespace

hipError_t launch_centred(const Plan& p, const Weights& w, const float* x, const int32_t* windows,
                          const int32_t* lags, int64_t count, double* out, hipStream_t s) {
    CentredArgs a;
    a.x = x;
    a.windows = windows;
    a.lags = lags;
    a.out = out;
    a.num_windows = p.num_windows;
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    hipLaunchKernelGGL(centred_kernel, dim3((unsigned)count), dim3(kWave * kWaves), 0, s, a, w);
    return hipGetLastError();
}

}  // namespace gpoeo
