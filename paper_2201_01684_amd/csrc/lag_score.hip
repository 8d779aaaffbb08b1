// Lag-score accumulation: D_c(T) = sum_{i<N-T} (x_c[i] - x_c[i+T])^2 for every lag.
//
// This is the score of Algorithm 2 (Sec. 4.1.2) read as the Euclidean distance
// between corresponding points of adjacent sub-curves of length T, taken over
// all N-T overlapping pairs; it is evaluated for every candidate period T.
//
// Work decomposition (one wavefront per task):
//   task = (window*C + channel, lag block, sample chunk), chunk index fastest.
//   A lag block is 64*BT consecutive lags (BT = 8 or 16 lags per lane): lane l
//   owns lags T_l .. T_l+BT-1 with T_l = t0 + 64*BT*block + BT*l, so the 64
//   lanes tile the block.  The wave walks its sample chunk in blocks of 16
//   samples.  x[i..i+15] is the same for every lane and is read with scalar
//   loads; lane l reads its (16+BT)-float window x[i+T_l ..] with vector loads
//   (consecutive lanes read consecutive pieces), and every staged value serves
//   up to BT lags from registers: 16*BT pairs per lane per block.  Each pair
//   costs one v_sub_f32 and one v_fmac_f32.
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
    int64_t n;             // pair bound: pair (i, i+T) counts iff i + T < n
    int64_t range;         // samples scored per window: i < range
    int64_t trace_len;     // > 0: also i + T < trace_len - window start
    int64_t cut;           // > 0: also i + T < (floor((T_wave - 1) / cut) + 1) * cut
    int64_t window_stride;
    int64_t channel_stride;
    int64_t chunk;
    int64_t tasks;
    int32_t num_channels;
    int32_t t0;
    int32_t lag_blocks;
    int32_t lags_padded;
    int32_t chunks;
    WindowTable tab;
};

// Lane window y[k] = x[i + T_l + k], k < kW = 16 + kBT - 1 (rounded up to a
// multiple of 4; the extra entries are loaded but never used).
// kShift in 0..3: the window start sits kShift floats past a 16-byte boundary
// and kNQ aligned float4 loads cover it; kShift == 4: dword loads, any alignment.
template <int kBT>
struct Geometry {
    static constexpr int kW = 16 + kBT;               // y entries kept (last one unused)
    static constexpr int kNQ = (kW + 6) / 4;          // float4 loads covering kW + shift
};

template <int kBT, int kShift>
__device__ __forceinline__ void load_window(const float* __restrict__ p,
                                            float (&y)[Geometry<kBT>::kW]) {
    constexpr int kW = Geometry<kBT>::kW, kNQ = Geometry<kBT>::kNQ;
    if constexpr (kShift < 4) {
        const float4* q = reinterpret_cast<const float4*>(p - kShift);
        float t[4 * kNQ];
#pragma unroll
        for (int k = 0; k < kNQ; ++k) {
            float4 v = q[k];
            t[4 * k + 0] = v.x;
            t[4 * k + 1] = v.y;
            t[4 * k + 2] = v.z;
            t[4 * k + 3] = v.w;
        }
#pragma unroll
        for (int k = 0; k < kW; ++k) y[k] = t[k + kShift];
    } else {
#pragma unroll
        for (int k = 0; k < kW - 1; ++k) y[k] = p[k];
        y[kW - 1] = 0.0f;
    }
}

// 16 samples x kBT lags, every pair valid.  The differences of four lags go
// to four registers before their four multiply-adds (the scheduling barriers
// keep the groups): left alone, the compiler reuses one register for every
// difference, so each instruction waits on the one before it, and that chain
// cost the launch on 1024 traces of 262,144 samples about 2.5% of its time.
template <int kBT>
__device__ __forceinline__ void block_full(const float (&xs)[16],
                                           const float (&y)[Geometry<kBT>::kW],
                                           float (&acc)[kBT]) {
    constexpr int kG = kBT < 4 ? kBT : 4;
#pragma unroll
    for (int s = 0; s < 16; ++s) {
#pragma unroll
        for (int j = 0; j < kBT; j += kG) {
            float d[kG];
#pragma unroll
            for (int u = 0; u < kG; ++u) d[u] = xs[s] - y[s + j + u];
            __builtin_amdgcn_sched_group_barrier(0x2, kG, 0);   // kG VALU: the subtractions
#pragma unroll
            for (int u = 0; u < kG; ++u) acc[j + u] = __builtin_fmaf(d[u], d[u], acc[j + u]);
            __builtin_amdgcn_sched_group_barrier(0x2, kG, 0);   // kG VALU: the multiply-adds
        }
    }
}

// 16 samples x kBT lags, pair (s, j) valid iff s + j < rem.
template <int kBT>
__device__ __forceinline__ void block_masked(const float (&xs)[16],
                                             const float (&y)[Geometry<kBT>::kW], int rem,
                                             float (&acc)[kBT]) {
#pragma unroll
    for (int s = 0; s < 16; ++s) {
#pragma unroll
        for (int j = 0; j < kBT; ++j) {
            float d = (s + j < rem) ? xs[s] - y[s + j] : 0.0f;
            acc[j] = __builtin_fmaf(d, d, acc[j]);
        }
    }
}

// Sixteen lags a lane run at most four waves a SIMD: that leaves the compiler
// 128 registers (it uses 109 instead of 92 at five waves), 0.6-0.9% faster on
// the 1024- and 256-trace workloads (A/B on one GPU).  The same bound slows the
// eight-lag instance by 4%, so the others keep the default.
template <int kBT, int kWavesPerGroup, int kShift>
__global__ __launch_bounds__(kWave * kWavesPerGroup)
__attribute__((amdgpu_waves_per_eu(kBT == 16 ? 4 : 1, kBT == 16 ? 4 : 8)))
void lag_score_kernel(ScoreArgs a) {
    constexpr int kW = Geometry<kBT>::kW;
    constexpr int kLagsPerBlock = kWave * kBT;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    // Workgroups are dispatched round-robin over the 8 XCDs; remap so that each
    // XCD runs a contiguous range of tasks (the tasks of one window share its
    // samples in that XCD's L2).
    const int64_t groups = gridDim.x;
    int64_t g = blockIdx.x;
    const int64_t full = groups - groups % 8;
    if (g < full) g = (g % 8) * (full / 8) + g / 8;
    const int64_t task = g * kWavesPerGroup + wave;
    if (task >= a.tasks) return;

    const int32_t k = (int32_t)(task % a.chunks);
    const int64_t rest = task / a.chunks;
    const int32_t blk = (int32_t)(rest % a.lag_blocks);
    const int64_t bc = rest / a.lag_blocks;
    const int64_t b = bc / a.num_channels;
    const int32_t c = (int32_t)(bc % a.num_channels);

    const float* __restrict__ xw =
        a.x + table_off(a.tab, b, a.window_stride) + (int64_t)c * a.channel_stride;
    const int64_t t_wave = (int64_t)a.t0 + (int64_t)blk * kLagsPerBlock;
    const int64_t t_lane = t_wave + (int64_t)lane * kBT;
    // Pair bound of this wave (wave-uniform): the window length, or for the
    // shared block partials of overlapping windows the trace end and, for the
    // cut partials, the end of the block the lags' ranges stop in.
    int64_t n = table_n(a.tab, b, a.n);
    // samples that exist from xw on: the window, or with shared block
    // partials the rest of the trace (the cut bound below only limits pairs)
    const int64_t mem_end = a.trace_len > 0 ? a.trace_len - b * a.window_stride : n;
    if (a.trace_len > 0) n = min(n, a.trace_len - b * a.window_stride);
    if (a.cut > 0) n = min(n, ((t_wave - 1) / a.cut + 1) * a.cut);

    const int64_t i_begin = (int64_t)k * a.chunk;
    const int64_t chunk_end = min(i_begin + a.chunk, a.range);
    // A block starting at i runs unmasked iff i + 16 <= lim_full: then every pair
    // of every lane is valid and the aligned window loads (which reach at most
    // x[i + t_wave_hi + 20] for both lane widths) stay below sample n.
    const int64_t t_wave_hi = t_wave + kLagsPerBlock - 1;
    const int64_t lim_full = min(chunk_end, n - t_wave_hi - 5);
    const int64_t lim_any = min(chunk_end, n - t_wave);
    const int64_t nb_full = lim_full > i_begin ? (lim_full - i_begin) / kBlockSamples : 0;
    const int64_t nb_any =
        lim_any > i_begin ? (lim_any - i_begin + kBlockSamples - 1) / kBlockSamples : 0;

    float acc[kBT];
    double acc64[kBT];
#pragma unroll
    for (int j = 0; j < kBT; ++j) {
        acc[j] = 0.0f;
        acc64[j] = 0.0;
    }
    const int64_t runs_per = kRunSamples / kBlockSamples;

    // Unmasked blocks, flushed to fp64 every kRunSamples samples.
    auto load_block = [&](int64_t q, float(&xs)[16], float(&y)[kW]) {
        const int64_t i = i_begin + q * kBlockSamples;
#pragma unroll
        for (int s = 0; s < 16; ++s) xs[s] = xw[i + s];
        load_window<kBT, kShift>(xw + i + t_lane, y);
    };
    for (int64_t q0 = 0; q0 < nb_full; q0 += runs_per) {
        const int64_t q1 = min(nb_full, q0 + runs_per);
        if constexpr (kBT <= 8) {
            // Two register sets: the loads of the next block are in flight
            // while this block's products run (a wave's own latency stays
            // hidden even when few waves share a SIMD, as for short windows).
            float xa[16], ya[kW], xb[16], yb[kW];
            load_block(q0, xa, ya);
            for (int64_t q = q0; q < q1; q += 2) {
                if (q + 1 < q1) load_block(q + 1, xb, yb);
                block_full<kBT>(xa, ya, acc);
                if (q + 1 >= q1) break;
                if (q + 2 < q1) load_block(q + 2, xa, ya);
                block_full<kBT>(xb, yb, acc);
            }
        } else {
            for (int64_t q = q0; q < q1; ++q) {
                float xs[16], y[kW];
                load_block(q, xs, y);
                block_full<kBT>(xs, y, acc);
            }
        }
#pragma unroll
        for (int j = 0; j < kBT; ++j) {
            acc64[j] += (double)acc[j];
            acc[j] = 0.0f;
        }
    }
    // Masked blocks at the end of the lags' ranges.  A block whose loads stay
    // below mem_end (the loads of an unmasked block reach at most sample
    // i + t_wave_hi + 20) loads like one and masks only the arithmetic: the
    // cut partials of shared blocks, whose pair bound lies inside the trace.
    // Otherwise no load passes the last sample.
    for (int64_t q0 = nb_full; q0 < nb_any; q0 += runs_per) {
        const int64_t q1 = min(nb_any, q0 + runs_per);
        for (int64_t q = q0; q < q1; ++q) {
            const int64_t i = i_begin + q * kBlockSamples;
            const int64_t rem64 = n - i - t_lane;   // pair (s, j) valid iff s + j < rem
            const int rem = (int)max((int64_t)-1, min(rem64, (int64_t)64));
            float xs[16], y[kW];
            if (i + t_wave_hi + 21 <= mem_end) {
                load_block(q, xs, y);
            } else {
#pragma unroll
                for (int s = 0; s < 16; ++s) xs[s] = (i + s < n) ? xw[i + s] : 0.0f;
#pragma unroll
                for (int kk = 0; kk < kW; ++kk) y[kk] = (kk < rem) ? xw[i + t_lane + kk] : 0.0f;
            }
            block_masked<kBT>(xs, y, rem, acc);
        }
#pragma unroll
        for (int j = 0; j < kBT; ++j) {
            acc64[j] += (double)acc[j];
            acc[j] = 0.0f;
        }
    }

    double* out = a.part + (bc * a.chunks + k) * (int64_t)a.lags_padded + (t_lane - a.t0);
#pragma unroll
    for (int j = 0; j < kBT; ++j) out[j] = acc64[j];
}

// Tiny problems (one short trace, a few lags: the online case of Algorithm
// 3): one workgroup of kTinyLags lanes per (sequence, block of kTinyLags lags,
// chunk of kTinyChunk samples).  The chunk x[i0 .. i0 + kTinyChunk) and its
// partners x[i0 + T0 .. i0 + T0 + kTinyChunk + kTinyLags) are staged in LDS
// once (zeros past the window); lane l sums the pairs of lag T0 + l whose
// partner lies in the window, as one fp32 run of at most kTinyChunk terms
// (the same bound as the main kernel), and writes it as that chunk's partial.
// Every load is issued at the start, so the kernel takes about one memory
// round trip plus kTinyChunk steps.
__global__ __launch_bounds__(kTinyLags) void lag_score_tiny_kernel(ScoreArgs a) {
    __shared__ float xa[kTinyChunk];
    __shared__ float xb[kTinyChunk + kTinyLags];
    const int tid = threadIdx.x;
    const int64_t task = blockIdx.x;
    const int32_t k = (int32_t)(task % a.chunks);
    const int64_t rest = task / a.chunks;
    const int32_t blk = (int32_t)(rest % a.lag_blocks);
    const int64_t bc = rest / a.lag_blocks;
    const int64_t b = bc / a.num_channels;
    const int32_t c = (int32_t)(bc % a.num_channels);
    const float* __restrict__ xw = a.x + b * a.window_stride + (int64_t)c * a.channel_stride;
    const int64_t n = a.n;
    const int64_t i0 = (int64_t)k * kTinyChunk;
    const int64_t t_blk = (int64_t)a.t0 + (int64_t)blk * kTinyLags;
    for (int j = tid; j < kTinyChunk; j += kTinyLags) xa[j] = i0 + j < n ? xw[i0 + j] : 0.0f;
    for (int j = tid; j < kTinyChunk + kTinyLags; j += kTinyLags) {
        const int64_t idx = i0 + t_blk + j;
        xb[j] = idx < n ? xw[idx] : 0.0f;
    }
    __syncthreads();
    const int64_t t = t_blk + tid;
    int64_t m = n - t - i0;                 // pairs (i0 + i, i0 + i + t) with i0 + i + t < n
    m = m < 0 ? 0 : (m > kTinyChunk ? kTinyChunk : m);
    float acc = 0.0f;
    for (int i = 0; i < (int)m; ++i) {
        const float d = xa[i] - xb[i + tid];
        acc = __builtin_fmaf(d, d, acc);
    }
    a.part[(bc * a.chunks + k) * (int64_t)a.lags_padded + (t - a.t0)] = (double)acc;
}

template <int kBT, int kWPG>
void launch_shifted(const Plan& p, const ScoreArgs& a, hipStream_t s) {
    const int64_t groups = (a.tasks + kWPG - 1) / kWPG;
    const dim3 grid((unsigned)groups), block(kWave * kWPG);
    switch (p.aligned ? (p.t0 & 3) : 4) {
        case 0: hipLaunchKernelGGL((lag_score_kernel<kBT, kWPG, 0>), grid, block, 0, s, a); break;
        case 1: hipLaunchKernelGGL((lag_score_kernel<kBT, kWPG, 1>), grid, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL((lag_score_kernel<kBT, kWPG, 2>), grid, block, 0, s, a); break;
        case 3: hipLaunchKernelGGL((lag_score_kernel<kBT, kWPG, 3>), grid, block, 0, s, a); break;
        default: hipLaunchKernelGGL((lag_score_kernel<kBT, kWPG, 4>), grid, block, 0, s, a); break;
    }
}

template <int kBT>
void launch_bt(const Plan& p, const ScoreArgs& a, hipStream_t s) {
    if (p.waves_per_group == 1) launch_shifted<kBT, 1>(p, a, s);
    else launch_shifted<kBT, 4>(p, a, s);
}

// bt: lags per lane of this launch (the plan's, or half of it for the cut
// partials of shared blocks)
void launch(const Plan& p, const ScoreArgs& a, hipStream_t s, int bt) {
    if (bt == 4) launch_bt<4>(p, a, s);
    else if (bt == 8) launch_bt<8>(p, a, s);
    else launch_bt<16>(p, a, s);
}

ScoreArgs common(const Plan& p, const float* x) {
    ScoreArgs a;
    a.x = x;
    a.part = nullptr;
    a.n = p.n;
    a.range = p.n;
    a.trace_len = 0;
    a.cut = 0;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.chunk = p.chunk;
    a.tasks = p.tasks;
    a.num_channels = p.num_channels;
    a.t0 = p.t0;
    a.lag_blocks = p.lag_blocks;
    a.lags_padded = p.lags_padded;
    a.chunks = p.chunks;
    a.tab = p.table;
    return a;
}

}  // namespace

hipError_t launch_lag_score(const Plan& p, const float* x, double* part, hipStream_t s) {
    ScoreArgs a = common(p, x);
    a.part = part;
    if (p.tiny) {
        const int64_t groups = p.num_windows * p.num_channels * p.lag_blocks * (int64_t)p.chunks;
        hipLaunchKernelGGL(lag_score_tiny_kernel, dim3((unsigned)groups), dim3(kTinyLags), 0, s,
                           a);
    } else {
        launch(p, a, s, p.lags_per_lane);
    }
    return hipGetLastError();
}

hipError_t launch_lag_score_blocks(const Plan& p, const float* x, double* full, double* cut,
                                   hipStream_t s) {
    // Overlapping windows at stride B_s = p.window_stride with N = m * B_s: the
    // trace is cut into G = num_windows + m - 1 blocks of B_s samples, scored
    // as "windows" of B_s samples whose pairs may reach past the block.
    ScoreArgs a = common(p, x);
    a.range = p.window_stride;
    a.n = p.window_stride + p.lags_padded + p.t0;   // no bound beyond the trace end
    a.trace_len = p.trace_len;
    a.tasks = p.block_tasks;
    a.chunk = p.block_chunk;
    a.chunks = p.block_chunks;
    a.part = full;                                  // full-block partials F_g(T)
    launch(p, a, s, p.lags_per_lane);
    // Cut-block partials C_g(T): every pair range of a lag block ends inside
    // the block, along a diagonal as long as the lag block is wide, which the
    // masked blocks cover; lag blocks of half the width halve that stretch.
    // They still start at 1 (mod their width), which divides the stride.
    a.part = cut;
    a.cut = p.window_stride;
    a.lag_blocks = 2 * p.lag_blocks;
    a.tasks = 2 * p.block_tasks;
    launch(p, a, s, p.lags_per_lane / 2);
    return hipGetLastError();
}

}  // namespace gpoeo
