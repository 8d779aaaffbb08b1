// Exact and tightly bounded fp64 evaluations of the score S(T) and of the
// reference R, shared by the selection and the rolling detection.  Every
// translation unit that includes this header is compiled with
// -ffp-contract=off: the expressions below round once per operation, as
// written.
#pragma once

#include "internal.h"

namespace gpoeo {
namespace exact {

// The exact re-scores below are plain sequential fp64 sums (ascending index,
// one rounding per addition, no contraction).  Their cost is a chain of
// dependent additions; to keep it from also waiting on memory at every step,
// samples are staged through registers in chunks of kChunk and the loads of
// the next chunk are issued before the additions of the current one.
constexpr int kChunk = 32;

template <typename F>
__device__ __forceinline__ void for_pairs(const float* __restrict__ a, const float* __restrict__ b,
                                          int64_t m, F&& step) {
    float ca[kChunk], cb[kChunk], na[kChunk], nb[kChunk];
    const int64_t full = m / kChunk;
    if (full > 0) {
#pragma unroll
        for (int k = 0; k < kChunk; ++k) {
            ca[k] = a[k];
            cb[k] = b[k];
        }
    }
    for (int64_t c = 0; c < full; ++c) {
        const bool more = c + 1 < full;
        if (more) {
            const int64_t o = (c + 1) * kChunk;
#pragma unroll
            for (int k = 0; k < kChunk; ++k) {
                na[k] = a[o + k];
                nb[k] = b[o + k];
            }
        }
#pragma unroll
        for (int k = 0; k < kChunk; ++k) step(ca[k], cb[k]);
        if (more) {
#pragma unroll
            for (int k = 0; k < kChunk; ++k) {
                ca[k] = na[k];
                cb[k] = nb[k];
            }
        }
    }
    for (int64_t i = full * kChunk; i < m; ++i) step(a[i], b[i]);
}

// Plain sequential fp64 evaluation of S(T) = sum_c w_c * D_c(T) / (N - T).
__device__ inline double exact_score(const float* __restrict__ xw, int32_t num_channels,
                              int64_t channel_stride, int64_t n, int64_t t, const Weights& w) {
#pragma clang fp contract(off)
    double s = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* __restrict__ xc = xw + (int64_t)c * channel_stride;
        const int64_t m = n - t;
        double dsum = 0.0;
        for_pairs(xc, xc + t, m, [&](float u, float v) {
#pragma clang fp contract(off)
            const double d = (double)u - (double)v;
            dsum = dsum + d * d;
        });
        s = s + (double)w.w[c] * (dsum / (double)m);
    }
    return s;
}

// Plain sequential fp64 evaluation of R = 2 * sum_c w_c * Var_c (two passes).
__device__ inline double exact_reference(const float* __restrict__ xw, int32_t num_channels,
                                  int64_t channel_stride, int64_t n, const Weights& w) {
#pragma clang fp contract(off)
    double acc = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* __restrict__ xc = xw + (int64_t)c * channel_stride;
        double sum = 0.0;
        for_pairs(xc, xc, n, [&](float u, float) { sum = sum + (double)u; });
        const double mean = sum / (double)n;
        double sq = 0.0;
        for_pairs(xc, xc, n, [&](float u, float) {
#pragma clang fp contract(off)
            const double d = (double)u - mean;
            sq = sq + d * d;
        });
        acc = acc + (double)w.w[c] * (sq / (double)n);
    }
    return 2.0 * acc;
}

// S(T) in fp64 by one wavefront (the tier-1 re-score of the FFT and
// matrix-core fix-ups and of the rolling combination).  Lane l accumulates the
// terms i = l + 64 (4k + r) in four partial sums r = 0..3, which are combined
// as (p0 + p1) + (p2 + p3) and then across lanes by a fixed shuffle tree; every
// lane returns lane 0's value.  Each partial sum holds at most M/256 + 1 terms,
// so the result is within (M/256 + 10) u of the exact sum (u = 2^-53).
__device__ inline double wave_score(const float* __restrict__ xw, int32_t num_channels,
                             int64_t channel_stride, int64_t n, int64_t t, const Weights& w,
                             int lane) {
    double s = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* __restrict__ xc = xw + (int64_t)c * channel_stride;
        const int64_t m = n - t;
        double p[4] = {0.0, 0.0, 0.0, 0.0};
        int64_t i = lane;
        for (; i + 192 < m; i += 256) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const double d = (double)xc[i + 64 * r] - (double)xc[i + 64 * r + t];
                p[r] = p[r] + d * d;
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t k = i + 64 * r;
            if (k < m) {
                const double d = (double)xc[k] - (double)xc[k + t];
                p[r] = p[r] + d * d;
            }
        }
        double part = (p[0] + p[1]) + (p[2] + p[3]);
        for (int off = 32; off > 0; off >>= 1) part = part + __shfl_down(part, off);
        part = __shfl(part, 0);
        s = s + (double)w.w[c] * (part / (double)m);
    }
    return s;
}

// Tier-1 re-score by a workgroup of kG lanes (kG/64 wavefronts; every thread
// calls it; red holds kG/64 doubles): lane l accumulates the terms
// i = l + kG (4k + r) in four partial sums r = 0..3, combined as
// (p0 + p1) + (p2 + p3), then a butterfly of lane shuffles in each wavefront,
// then the wavefront sums in wavefront order.  Each partial sum holds at most
// M/(4 kG) + 1 terms, so the result is within (M/(4 kG) + 12) u of the exact
// sum; every thread returns the same value.
template <int kG>
__device__ inline double group_score(const float* __restrict__ xw, int32_t num_channels,
                                     int64_t channel_stride, int64_t n, int64_t t,
                                     const Weights& w, double* red) {
    constexpr int kWaves = kG / kWave;
    const int tid = threadIdx.x;
    double s = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const float* __restrict__ xc = xw + (int64_t)c * channel_stride;
        const int64_t m = n - t;
        double p[4] = {0.0, 0.0, 0.0, 0.0};
        int64_t i = tid;
        // the operands of kAhead steps are loaded before they are added (in
        // the same order), so that a lane has them in flight together
        constexpr int kAhead = 8;
        for (; i + (4 * kAhead - 1) * (int64_t)kG < m; i += 4 * kAhead * (int64_t)kG) {
            float u[4 * kAhead], v[4 * kAhead];
#pragma unroll
            for (int q = 0; q < 4 * kAhead; ++q) {
                u[q] = xc[i + (int64_t)kG * q];
                v[q] = xc[i + (int64_t)kG * q + t];
            }
#pragma unroll
            for (int q = 0; q < 4 * kAhead; ++q) {
                const double d = (double)u[q] - (double)v[q];
                p[q & 3] = p[q & 3] + d * d;
            }
        }
        for (; i + 3 * kG < m; i += 4 * kG) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const double d = (double)xc[i + kG * r] - (double)xc[i + kG * r + t];
                p[r] = p[r] + d * d;
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t k = i + kG * r;
            if (k < m) {
                const double d = (double)xc[k] - (double)xc[k + t];
                p[r] = p[r] + d * d;
            }
        }
        double part = (p[0] + p[1]) + (p[2] + p[3]);
        for (int off = kWave / 2; off > 0; off >>= 1) part = part + __shfl_xor(part, off);
        if ((tid & (kWave - 1)) == 0) red[tid / kWave] = part;
        __syncthreads();
        double tot = red[0];
        for (int v = 1; v < kWaves; ++v) tot = tot + red[v];
        __syncthreads();
        s = s + (double)w.w[c] * (tot / (double)m);
    }
    return s;
}

// Half-width of the interval around the two-pass fp64 R that contains the
// plain sequential evaluation.  Any evaluation order of the mean of N samples
// errs by at most (N+1) u A (A = mean |x|); the second pass then sums
// Var + dmean^2 exactly, up to (N+4) u relative.  Two orders thus differ by at
// most 4 (N+4) u Var + 4.02 ((N+1) u A)^2 per channel, weighted and doubled
// for R, plus the rounding of the weighted channel sum.
__device__ inline double reference_bound(const double* var2, int32_t num_channels, int64_t n,
                                  const Weights& w, double r) {
    const double u = 1.1102230246251565e-16;
    const double nn = (double)n;
    double e = 0.0;
    for (int32_t c = 0; c < num_channels; ++c) {
        const double v = var2[2 * c], am = var2[2 * c + 1];
        const double dm = (nn + 1.0) * u * am;
        e += (double)w.w[c] * (4.0 * (nn + 4.0) * u * v + 4.02 * dm * dm);
    }
    return 1.01 * (2.0 * e + (num_channels + 4.0) * u * r);
}

}  // namespace exact
}  // namespace gpoeo
