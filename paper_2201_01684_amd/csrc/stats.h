// Window statistics helpers shared by the statistics kernel and the fused
// small-window kernel, so that both compute the same bits: a fixed visiting
// order of a window's samples and a fixed-order workgroup sum.  Every
// translation unit that includes this header is compiled with
// -ffp-contract=off.
#pragma once

#include "internal.h"

namespace gpoeo {
namespace stats {

constexpr int kStatsThreads = 256;

// Sums of two values over the workgroup, in a fixed order: a butterfly of
// lane shuffles inside each wavefront (every lane gets the same bits), then
// the four wavefront sums as (w0 + w1) + (w2 + w3).  red holds 8 doubles.
__device__ inline void block_sum2(double& x, double& y, double* red) {
    static_assert(kStatsThreads == 4 * kWave, "four wavefronts");
    for (int o = kWave / 2; o > 0; o >>= 1) {
        x = x + __shfl_xor(x, o);
        y = y + __shfl_xor(y, o);
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        red[wave] = x;
        red[4 + wave] = y;
    }
    __syncthreads();
    x = (red[0] + red[1]) + (red[2] + red[3]);
    y = (red[4] + red[5]) + (red[6] + red[7]);
    __syncthreads();
}

// Visits x[0..n) once in a fixed order per thread: a scalar head up to 16-byte
// alignment, then 16-byte groups (thread t takes groups t, t + 256, ..., four
// loads in flight), then a scalar tail.
template <typename F>
__device__ __forceinline__ void visit(const float* __restrict__ xw, int64_t n, F&& f) {
    const int64_t mis = (int64_t)((reinterpret_cast<uintptr_t>(xw) >> 2) & 3);
    const int64_t head = ((4 - mis) & 3) < n ? ((4 - mis) & 3) : n;
    for (int64_t i = threadIdx.x; i < head; i += kStatsThreads) f(xw[i]);
    const float4* __restrict__ v = reinterpret_cast<const float4*>(xw + head);
    const int64_t groups = (n - head) >> 2;
    int64_t g = threadIdx.x;
    for (; g + 3 * kStatsThreads < groups; g += 4 * kStatsThreads) {
        const float4 a = v[g], b = v[g + kStatsThreads], c = v[g + 2 * kStatsThreads],
                     d = v[g + 3 * kStatsThreads];
        f(a.x); f(a.y); f(a.z); f(a.w);
        f(b.x); f(b.y); f(b.z); f(b.w);
        f(c.x); f(c.y); f(c.z); f(c.w);
        f(d.x); f(d.y); f(d.z); f(d.w);
    }
    for (; g < groups; g += kStatsThreads) {
        const float4 a = v[g];
        f(a.x); f(a.y); f(a.z); f(a.w);
    }
    for (int64_t i = head + (groups << 2) + threadIdx.x; i < n; i += kStatsThreads) f(xw[i]);
}


// Mean, population variance and mean |x| of one channel of one window, as
// written by the statistics kernel (var[0] = variance, var[1] = mean |x|);
// also the mean and the sums of squared and of absolute deviations (fstat).
// Every thread of the kStatsThreads-wide workgroup returns the same values.
struct ChannelStats {
    double mean, var, absmean, sq, sabs;
};

__device__ inline ChannelStats channel_stats(const float* __restrict__ xw, int64_t n, double* red,
                                             bool with_sabs) {
    double s = 0.0, sa = 0.0;
    visit(xw, n, [&](float x) {
        const double v = (double)x;
        s += v;
        sa += fabs(v);
    });
    block_sum2(s, sa, red);
    ChannelStats r;
    r.mean = s / (double)n;
    r.absmean = sa / (double)n;
    double q = 0.0, qa = 0.0;
    visit(xw, n, [&](float x) {
        const double d = (double)x - r.mean;
        q += d * d;
        qa += fabs(d);
    });
    block_sum2(q, qa, red);
    r.sq = q;
    r.sabs = with_sabs ? qa : 0.0;
    r.var = r.sq / (double)n;
    return r;
}

// S(T) of window b from the fp64 chunk partials of its channels (layout
// [b*C + c][chunk][lags_padded], lag T at index T - t0): each channel's
// partials added in ascending chunk order, divided by the N - T pairs, and
// the weighted channel sum (the composite feature of Sec. 4.2).
// The partials are loaded kFinalizeBatch at a time (all in flight) and added
// in order.  finalize_lags does the same for kFinalizeLags lags at once (lag
// t + k * lag_step, those below t_end), each with exactly finalize_lag's
// operations.
constexpr int kFinalizeBatch = 8;
constexpr int kFinalizeLags = 4;

__device__ inline double finalize_lag(const double* __restrict__ part, const Weights& w,
                                      int32_t num_channels, int64_t b, int64_t n, int64_t t,
                                      int32_t t0, int32_t lags_padded, int32_t chunks) {
    double s = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const double* p =
            part + ((b * num_channels + c) * chunks) * (int64_t)lags_padded + (t - t0);
        double d = 0.0;
        int32_t k = 0;
        for (; k + kFinalizeBatch <= chunks; k += kFinalizeBatch) {
            double v[kFinalizeBatch];
#pragma unroll
            for (int u = 0; u < kFinalizeBatch; ++u) v[u] = p[(int64_t)(k + u) * lags_padded];
#pragma unroll
            for (int u = 0; u < kFinalizeBatch; ++u) d += v[u];
        }
        for (; k < chunks; ++k) d += p[(int64_t)k * lags_padded];
        s += (double)w.w[c] * (d / (double)(n - t));
    }
    return s;
}

__device__ inline void finalize_lags(const double* __restrict__ part, const Weights& w,
                                     int32_t num_channels, int64_t b, int64_t n, int64_t t,
                                     int64_t lag_step, int64_t t_end, int32_t t0,
                                     int32_t lags_padded, int32_t chunks,
                                     double (&out)[kFinalizeLags]) {
    constexpr int L = kFinalizeLags;
    bool live[L];
#pragma unroll
    for (int l = 0; l < L; ++l) {
        live[l] = t + l * lag_step < t_end;
        out[l] = 0.0;
    }
    for (int32_t c = 0; c < num_channels; ++c) {
        const double* p =
            part + ((b * num_channels + c) * chunks) * (int64_t)lags_padded + (t - t0);
        double d[L];
#pragma unroll
        for (int l = 0; l < L; ++l) d[l] = 0.0;
        int32_t k = 0;
        for (; k + kFinalizeBatch <= chunks; k += kFinalizeBatch) {
            double v[L][kFinalizeBatch];
#pragma unroll
            for (int l = 0; l < L; ++l)
#pragma unroll
                for (int u = 0; u < kFinalizeBatch; ++u)
                    v[l][u] = live[l] ? p[l * lag_step + (int64_t)(k + u) * lags_padded] : 0.0;
#pragma unroll
            for (int l = 0; l < L; ++l)
#pragma unroll
                for (int u = 0; u < kFinalizeBatch; ++u) d[l] += v[l][u];
        }
        for (; k < chunks; ++k)
#pragma unroll
            for (int l = 0; l < L; ++l)
                if (live[l]) d[l] += p[l * lag_step + (int64_t)k * lags_padded];
#pragma unroll
        for (int l = 0; l < L; ++l)
            if (live[l]) out[l] += (double)w.w[c] * (d[l] / (double)(n - (t + l * lag_step)));
    }
}

}  // namespace stats
}  // namespace gpoeo
