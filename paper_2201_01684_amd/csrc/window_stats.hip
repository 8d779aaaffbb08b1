// Window statistics and score finalisation.
//
// window_stats: per (window, channel), the population variance in fp64 by two
//   passes (mean, then mean squared deviation), each a fixed-order workgroup
//   reduction, and the mean absolute sample (which bounds how far any fp64
//   evaluation order of the mean, and so of the variance, can stray).  The
//   selection forms R = 2 * sum_c w_c * Var_c from it, the reference the
//   relative-height candidate filter of Algorithm 1 is measured against in
//   the lag domain.  For the FFT scores it also keeps the mean, the sum of
//   squared deviations and the sum of absolute deviations.
// finalize: per (window, lag), combines the fp64 chunk partials of every
//   channel in ascending chunk order, divides by the N-T pairs and forms the
//   weighted channel sum S(T) (the composite detection feature of Sec. 4.2).
#include <algorithm>

#include "internal.h"
#include "stats.h"

namespace gpoeo {
namespace {

__global__ __launch_bounds__(stats::kStatsThreads) void window_stats_kernel(
    const float* __restrict__ x, double* __restrict__ var, int64_t n_all, int64_t window_stride,
    int64_t channel_stride, int32_t num_channels, WindowTable tab, double* __restrict__ fstat) {
    __shared__ double red[stats::kStatsThreads];
    const int64_t bc = blockIdx.x;
    const int64_t b = bc / num_channels;
    const int32_t c = (int32_t)(bc % num_channels);
    const int64_t n = table_n(tab, b, n_all);
    if (n == 0) {   // empty slot of a window table
        if (threadIdx.x == 0) {
            var[2 * bc] = var[2 * bc + 1] = 0.0;
            if (fstat) fstat[4 * bc] = fstat[4 * bc + 1] = fstat[4 * bc + 2] = fstat[4 * bc + 3] = 0.0;
        }
        return;
    }
    const float* __restrict__ xw =
        x + table_off(tab, b, window_stride) + (int64_t)c * channel_stride;
    const stats::ChannelStats st = stats::channel_stats(xw, n, red, fstat != nullptr);
    if (threadIdx.x == 0) {
        var[2 * bc] = st.var;
        var[2 * bc + 1] = st.absmean;
        if (fstat) {   // the FFT scores centre each sequence by this same mean
            fstat[4 * bc] = st.mean;
            fstat[4 * bc + 1] = st.sq;
            fstat[4 * bc + 2] = st.sabs;
            fstat[4 * bc + 3] = 0.0;
        }
    }
}

// One workgroup per (window, block of 256 lags).  A window of a table scores
// only its own lag range [tmin, Tmax_b]; with no fp32 scores requested, the
// fp64 entries past it are left unwritten (nothing reads them), otherwise
// both are zero there.
__global__ __launch_bounds__(256) void finalize_kernel(const double* __restrict__ part,
                                                       double* __restrict__ s64,
                                                       float* __restrict__ scores, Weights w,
                                                       int32_t num_channels, int64_t n_all,
                                                       int32_t tmin, int32_t lags, int32_t t0,
                                                       int32_t lags_padded, int32_t chunks,
                                                       WindowTable tab) {
    const int64_t b = blockIdx.x;
    const int64_t n = table_n(tab, b, n_all);
    const int32_t live = n == 0 ? 0 : min(table_tmax(tab, b, tmin + lags - 1) - tmin + 1, lags);
    const int32_t end = (tab.n && !scores) ? live : lags;
    for (int32_t j = blockIdx.y * 256 + threadIdx.x; j < end; j += gridDim.y * 256) {
        const int64_t e = b * (int64_t)lags + j;
        if (j >= live) {   // outside this window's range
            s64[e] = 0.0;
            if (scores) scores[e] = 0.0f;
            continue;
        }
        const int64_t t = (int64_t)tmin + j;
        const double s = stats::finalize_lag(part, w, num_channels, b, n, t, t0, lags_padded,
                                             chunks);
        s64[e] = s;
        if (scores) scores[e] = (float)s;
    }
}

// Overlapping windows at stride s, N = m s: window b's pairs for lag T cover
// its first m - 1 - q blocks in full (q = floor((T-1)/s): the lag's range ends
// inside block m - 1 - q) and block m - 1 - q up to that end.  So
//   D_b(T) = sum_{k < m-1-q} F_{b+k}(T) + C_{b+m-1-q}(T),
// summed in this fixed order (blocks, then the chunks of each block).
__global__ __launch_bounds__(256) void finalize_blocks_kernel(
    const double* __restrict__ full, const double* __restrict__ cut, double* __restrict__ s64,
    float* __restrict__ scores, Weights w, int64_t num_windows, int32_t num_channels, int64_t n,
    int64_t stride, int32_t m, int32_t tmin, int32_t lags, int32_t t0, int32_t lags_padded,
    int32_t chunks) {
    const int64_t total = num_windows * (int64_t)lags;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = e / lags;
        const int32_t j = (int32_t)(e % lags);
        const int64_t t = (int64_t)tmin + j;
        const int64_t q = (t - 1) / stride;
        double s = 0.0;
        for (int32_t c = 0; c < num_channels; ++c) {
            double d = 0.0;
            for (int64_t k = 0; k + 1 + q < m; ++k) {
                const double* p = full + ((b + k) * num_channels + c) * chunks * (int64_t)lags_padded +
                                  (t - t0);
                for (int32_t h = 0; h < chunks; ++h) d += p[(int64_t)h * lags_padded];
            }
            const double* p = cut + ((b + m - 1 - q) * num_channels + c) * chunks *
                                        (int64_t)lags_padded + (t - t0);
            for (int32_t h = 0; h < chunks; ++h) d += p[(int64_t)h * lags_padded];
            s += (double)w.w[c] * (d / (double)(n - t));
        }
        s64[e] = s;
        if (scores) scores[e] = (float)s;
    }
}

}  // namespace

hipError_t launch_finalize_blocks(const Plan& p, const Weights& w, const double* full,
                                  const double* cut, double* s64, float* scores, hipStream_t s) {
    const int64_t total = p.num_windows * (int64_t)p.lags;
    int64_t groups = (total + 255) / 256;
    if (groups > 65536) groups = 65536;
    hipLaunchKernelGGL(finalize_blocks_kernel, dim3((unsigned)groups), dim3(256), 0, s, full, cut,
                       s64, scores, w, p.num_windows, p.num_channels, p.n, p.window_stride, p.m,
                       p.tmin, p.lags, p.t0, p.lags_padded, p.block_chunks);
    return hipGetLastError();
}

hipError_t launch_window_stats(const Plan& p, const float* x, double* var, double* fstat,
                               hipStream_t s) {
    const int64_t groups = p.num_windows * p.num_channels;
    hipLaunchKernelGGL(window_stats_kernel, dim3((unsigned)groups), dim3(stats::kStatsThreads), 0, s, x,
                       var, p.n, p.window_stride, p.channel_stride, p.num_channels, p.table, fstat);
    return hipGetLastError();
}

hipError_t launch_finalize(const Plan& p, const Weights& w, const double* part, double* s64,
                           float* scores, hipStream_t s) {
    const int64_t lag_groups = std::min<int64_t>((p.lags + 255) / 256, 65535);
    hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)p.num_windows, (unsigned)lag_groups),
                       dim3(256), 0, s, part, s64, scores, w, p.num_channels, p.n, p.tmin, p.lags,
                       p.t0, p.lags_padded, p.chunks, p.table);
    return hipGetLastError();
}

}  // namespace gpoeo
