// Lag-score accumulation: D_c(T) = sum_{i<N-T} (x_c[i] - x_c[i+T])^2 for every lag.
//
// This is the score of Algorithm 2 (Sec. 4.1.2) read as the Euclidean distance
// between corresponding points of adjacent sub-curves of length T, taken over
// all N-T overlapping pairs; it is evaluated for every candidate period T.
//
// Work decomposition (one wavefront per task):
//   task = (window*C + channel, lag block, sample chunk), chunk index fastest.
//   A lag block is 1024 consecutive lags: lane l owns lags T_l .. T_l+15 with
//   T_l = t0 + 1024*block + 16*l, so the 64 lanes tile the block.
//   The wave walks its sample chunk in blocks of 16 samples.  x[i..i+15] is the
//   same for every lane and is read with scalar loads; lane l reads its 32-float
//   window x[i+T_l .. i+T_l+31] with vector loads (consecutive lanes read
//   consecutive 64-byte pieces), and every staged value serves up to 16 lags
//   from registers: 256 pairs per lane per block for 16 + 32 loaded floats.
//   Each pair costs one v_sub_f32 and one v_fmac_f32.
//
// Precision: the 16 per-lane accumulators are fp32 and are flushed into fp64
// every 256 samples, so a run sums at most 256 non-negative terms.
//
// Per-lag validity i + T < N: blocks in which every (sample, lag) pair of
// every lane is valid run unmasked; the few blocks near the end of a lag's
// range run a masked variant in which an invalid pair contributes exactly 0
// and no load reaches past sample N-1.
#include "internal.h"

namespace gpoeo {
namespace {

struct ScoreArgs {
    const float* x;
    double* part;          // [window*C + channel][chunk][lags_padded]
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int64_t chunk;
    int64_t tasks;
    int32_t num_channels;
    int32_t t0;
    int32_t lag_blocks;
    int32_t lags_padded;
    int32_t chunks;
};

// Lane window y[k] = x[i + T_l + k], k < 32 (y[31] is loaded but never used).
// kShift in 0..3: the window start sits kShift floats past a 16-byte boundary and
// nine aligned float4 loads cover it; kShift == 4: plain dword loads, any alignment.
template <int kShift>
__device__ __forceinline__ void load_window(const float* __restrict__ p, float (&y)[32]) {
    if constexpr (kShift < 4) {
        const float4* q = reinterpret_cast<const float4*>(p - kShift);
        float t[36];
#pragma unroll
        for (int k = 0; k < 9; ++k) {
            float4 v = q[k];
            t[4 * k + 0] = v.x;
            t[4 * k + 1] = v.y;
            t[4 * k + 2] = v.z;
            t[4 * k + 3] = v.w;
        }
#pragma unroll
        for (int k = 0; k < 32; ++k) y[k] = t[k + kShift];
    } else {
#pragma unroll
        for (int k = 0; k < 31; ++k) y[k] = p[k];
        y[31] = 0.0f;
    }
}

// 16 samples x 16 lags, every pair valid.
__device__ __forceinline__ void block_full(const float (&xs)[16], const float (&y)[32],
                                           float (&acc)[16]) {
#pragma unroll
    for (int s = 0; s < 16; ++s) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            float d = xs[s] - y[s + j];
            acc[j] = __builtin_fmaf(d, d, acc[j]);
        }
    }
}

// 16 samples x 16 lags, pair (s, j) valid iff s + j < rem.
__device__ __forceinline__ void block_masked(const float (&xs)[16], const float (&y)[32], int rem,
                                             float (&acc)[16]) {
#pragma unroll
    for (int s = 0; s < 16; ++s) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            float d = (s + j < rem) ? xs[s] - y[s + j] : 0.0f;
            acc[j] = __builtin_fmaf(d, d, acc[j]);
        }
    }
}

template <int kShift>
__global__ __launch_bounds__(256) void lag_score_kernel(ScoreArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    // Workgroups are dispatched round-robin over the 8 XCDs; remap so that each
    // XCD runs a contiguous range of tasks (the tasks of one window share its
    // samples in that XCD's L2).
    const int64_t groups = gridDim.x;
    int64_t g = blockIdx.x;
    const int64_t full = groups - groups % 8;
    if (g < full) g = (g % 8) * (full / 8) + g / 8;
    const int64_t task = g * (blockDim.x / kWave) + wave;
    if (task >= a.tasks) return;

    const int32_t k = (int32_t)(task % a.chunks);
    const int64_t rest = task / a.chunks;
    const int32_t blk = (int32_t)(rest % a.lag_blocks);
    const int64_t bc = rest / a.lag_blocks;
    const int64_t b = bc / a.num_channels;
    const int32_t c = (int32_t)(bc % a.num_channels);

    const float* __restrict__ xw = a.x + b * a.window_stride + (int64_t)c * a.channel_stride;
    const int64_t t_wave = (int64_t)a.t0 + (int64_t)blk * kLagsPerWave;
    const int64_t t_lane = t_wave + (int64_t)lane * kLagsPerLane;
    const int64_t n = a.n;

    const int64_t i_begin = (int64_t)k * a.chunk;
    const int64_t chunk_end = i_begin + a.chunk;
    // A block starting at i runs unmasked iff i + 16 <= lim_full: then every pair
    // of every lane is valid and the aligned window loads (which reach at most
    // x[i + t_wave_hi + 20]) stay below sample n.
    const int64_t t_wave_hi = t_wave + kLagsPerWave - 1;
    const int64_t lim_full = min(chunk_end, n - t_wave_hi - 5);
    const int64_t lim_any = min(chunk_end, n - t_wave);
    const int64_t nb_full = lim_full > i_begin ? (lim_full - i_begin) / kBlockSamples : 0;
    const int64_t nb_any =
        lim_any > i_begin ? (lim_any - i_begin + kBlockSamples - 1) / kBlockSamples : 0;

    float acc[16];
    double acc64[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        acc[j] = 0.0f;
        acc64[j] = 0.0;
    }
    const int64_t runs_per = kRunSamples / kBlockSamples;

    // Unmasked blocks, flushed to fp64 every kRunSamples samples.
    for (int64_t q0 = 0; q0 < nb_full; q0 += runs_per) {
        const int64_t q1 = min(nb_full, q0 + runs_per);
        for (int64_t q = q0; q < q1; ++q) {
            const int64_t i = i_begin + q * kBlockSamples;
            float xs[16];
#pragma unroll
            for (int s = 0; s < 16; ++s) xs[s] = xw[i + s];
            float y[32];
            load_window<kShift>(xw + i + t_lane, y);
            block_full(xs, y, acc);
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            acc64[j] += (double)acc[j];
            acc[j] = 0.0f;
        }
    }
    // Masked blocks at the end of the lags' ranges.
    for (int64_t q0 = nb_full; q0 < nb_any; q0 += runs_per) {
        const int64_t q1 = min(nb_any, q0 + runs_per);
        for (int64_t q = q0; q < q1; ++q) {
            const int64_t i = i_begin + q * kBlockSamples;
            float xs[16];
#pragma unroll
            for (int s = 0; s < 16; ++s) xs[s] = (i + s < n) ? xw[i + s] : 0.0f;
            const int64_t rem64 = n - i - t_lane;   // pair (s, j) valid iff s + j < rem
            const int rem = (int)max((int64_t)-1, min(rem64, (int64_t)64));
            float y[32];
#pragma unroll
            for (int kk = 0; kk < 32; ++kk) y[kk] = (kk < rem) ? xw[i + t_lane + kk] : 0.0f;
            block_masked(xs, y, rem, acc);
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            acc64[j] += (double)acc[j];
            acc[j] = 0.0f;
        }
    }

    double* out = a.part + (bc * a.chunks + k) * (int64_t)a.lags_padded + (t_lane - a.t0);
#pragma unroll
    for (int j = 0; j < 16; ++j) out[j] = acc64[j];
}

}  // namespace

hipError_t launch_lag_score(const Plan& p, const float* x, double* part, hipStream_t s) {
    ScoreArgs a;
    a.x = x;
    a.part = part;
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.chunk = p.chunk;
    a.tasks = p.tasks;
    a.num_channels = p.num_channels;
    a.t0 = p.t0;
    a.lag_blocks = p.lag_blocks;
    a.lags_padded = p.lags_padded;
    a.chunks = p.chunks;
    const int waves_per_group = 4;
    const int64_t groups = (p.tasks + waves_per_group - 1) / waves_per_group;
    dim3 grid((unsigned)groups), block(kWave * waves_per_group);
    switch (p.aligned ? (p.t0 & 3) : 4) {
        case 0: hipLaunchKernelGGL(lag_score_kernel<0>, grid, block, 0, s, a); break;
        case 1: hipLaunchKernelGGL(lag_score_kernel<1>, grid, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL(lag_score_kernel<2>, grid, block, 0, s, a); break;
        case 3: hipLaunchKernelGGL(lag_score_kernel<3>, grid, block, 0, s, a); break;
        default: hipLaunchKernelGGL(lag_score_kernel<4>, grid, block, 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace gpoeo
