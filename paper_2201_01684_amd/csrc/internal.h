// Internal launch plan and kernel entry points of libgpoeo_pd (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gpoeo_pd.h"

namespace gpoeo {

constexpr int kWave = 64;            // CDNA wavefront width
constexpr int kBlockSamples = 16;    // samples per register block of the score kernel
constexpr int kRunSamples = 256;     // samples per fp32 run before the fp64 flush
constexpr int kMaxChannels = GPOEO_PD_MAX_CHANNELS;   // weights travel as a kernel argument
// Tiny plans (at most kTinyMaxPairs pairs, windows of at most kFusedMaxN
// samples): one LDS-staged workgroup per (sequence, kTinyLags lags,
// kTinyChunk samples) instead of the register-blocked wavefronts.
constexpr int kTinyLags = 256;
constexpr int kTinyChunk = 256;
constexpr double kTinyMaxPairs = 1e8;

// Relative error bound of a score accumulated in fp32 runs of kRunSamples
// non-negative terms (each run: kRunSamples roundings plus the rounding of the
// difference, about 258 * 2^-24 = 1.54e-5) and combined in fp64; rounded up.
constexpr double kScoreRelBound = 2.5e-5;

// Relative half-width of a tier-0 score from the fp64 FFT path: a lag whose
// rigorous FFT error bound exceeds half of this (times the score) is re-scored
// in fp64 before the selection.
constexpr double kFftRelBound = 1e-6;

// FFT path: complex fp64 points per transform workgroup (held in LDS): 2^11
// (32 KiB, four workgroups per CU) for transforms up to 2^20 points, 2^12
// beyond (a row pair must fit one tile); threads per transform workgroup;
// the largest transform.
constexpr int kFftSmallTileLog2 = 11;
constexpr int kFftTileLog2 = 12;
constexpr int kFftThreadsLog2 = 8;
constexpr int kFftMaxLog2 = 2 * (kFftTileLog2 - 1);
constexpr int kFftMinLog2 = 6;
// Wrap-corrected transforms (see Plan): the head-tail transform is always a
// split one (at least 2^12 points) and at most 2^20 points (its row kernel
// holds four rows of up to 2^10 points in one 2^12-point tile).
constexpr int kFftWrapMinLog2 = 12;
constexpr int kFftWrapMaxLog2 = 20;
constexpr int kFftClasses = kFftMaxLog2 + 1;   // length classes 2^lg of a ragged batch, by lg
// Matrix-core scores (GPOEO_PD_MFMA_SCORES): lags per wavefront tile, zero
// padding before and after each digit plane (bytes; the LDS staging reads
// 16-byte chunks that start before N, so at most 15 bytes past N, and A rows
// from 64 bytes before sample 0), and the steps between two flushes of the
// int32 shift groups (each stays below 2^31: 4 digit pairs x 32 products of at
// most 2^14 per step).
constexpr int kMfmaTileLags = 1024;
constexpr int kMfmaPadL = 64;
constexpr int kMfmaPadR = 64;
constexpr int kMfmaFlush = 512;
// A batch with fewer than kMfmaTargetWaves (sequence, lag tile) waves splits
// each tile's sample steps into chunks of at least kMfmaMinChunkSteps, whose
// partial cross terms a combination kernel adds in chunk order.
constexpr int kMfmaTargetWaves = 4096;
constexpr int kMfmaMinChunkSteps = 64;
inline int fft_tile_log2(int lg) { return lg <= 2 * (kFftSmallTileLog2 - 1) ? kFftSmallTileLog2 : kFftTileLog2; }

struct Weights {
    float w[kMaxChannels];
};

// Optional per-window table (device arrays) for batches of windows of
// different lengths: window b starts at off[b] (channel 0), has n[b] samples
// (0: an empty slot) and lags up to tmax[b].  Null pointers: window b starts at
// b * window_stride with the descriptor's N and Tmax.
struct WindowTable {
    const int64_t* off;
    const int64_t* n;
    const int32_t* tmax;
};

__device__ __forceinline__ int64_t table_off(const WindowTable& t, int64_t b, int64_t stride) {
    return t.off ? t.off[b] : b * stride;
}
__device__ __forceinline__ int64_t table_n(const WindowTable& t, int64_t b, int64_t n) {
    return t.n ? t.n[b] : n;
}
__device__ __forceinline__ int32_t table_tmax(const WindowTable& t, int64_t b, int32_t tmax) {
    return t.tmax ? t.tmax[b] : tmax;
}

// Longest window of a fused plan: a tier-1 re-score of one lag is then at most
// 256 fp64 steps per lane of one wavefront.
constexpr int64_t kFusedMaxN = GPOEO_PD_FUSED_MAX_N;
// Most lags of a fused plan: the kernel keeps the window's fp64 scores and
// four bitmaps in LDS (at most about 49 KiB, so the workgroup stays within
// 64 KiB of LDS).
constexpr int32_t kFusedMaxLags = GPOEO_PD_FUSED_MAX_LAGS;

// Selection passes (with one re-score round between consecutive passes) and the
// capacity of each re-score queue (per tier, per round, all windows together).
constexpr int kPasses = 4;
constexpr int kQueueCap = 1 << 16;

// Per-window selection state kept in the workspace between selection passes.
struct WinState {
    double r_exact;          // R as a plain sequential fp64 evaluation, once computed
    int32_t done;            // result written
    int32_t r_queued;        // R queued for the sequential evaluation
    int32_t r_is_exact;
    int32_t rescored;        // lags re-scored in fp64 so far
    int32_t tier2;           // a score or R was recomputed as a plain sequential sum
};

// Workspace buffers of the selection.
struct SelectBuffers {
    uint32_t* tier1;         // [B][words] bitmaps
    uint32_t* tier2;
    uint32_t* queued1;
    uint32_t* queued2;
    WinState* state;         // [B]
    int32_t* q_win;          // [2][kQueueCap]
    int32_t* q_lag;          // [2][kQueueCap]
    int32_t* q_count;        // [kPasses][2]
};

// Everything the kernels need, derived on the host from a validated descriptor.
struct Plan {
    int64_t num_windows;
    int32_t num_channels;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t tmin, tmax;
    int32_t lags;            // tmax - tmin + 1
    int32_t t0;              // first lag of lag block 0 (tmin rounded down to a multiple of 4)
    int32_t lags_per_lane;   // consecutive lags in one lane's accumulators (8 or 16)
    int32_t waves_per_group; // score-kernel wavefronts per workgroup (1 or 4)
    int32_t lag_blocks;      // blocks of 64 * lags_per_lane lags covering [t0, tmax]
    int32_t lags_padded;     // lag_blocks * 64 * lags_per_lane
    int32_t chunks;          // sample chunks per (window, channel, lag block)
    int64_t chunk;           // samples per chunk, a multiple of kBlockSamples
    int64_t tasks;           // waves of the score kernel
    bool aligned;            // x and strides allow 16-byte vector loads
    // Overlapping windows at stride s with N = m * s share per-block partials:
    // the trace (trace_len = (B-1) s + N samples per channel) is cut into
    // blocks = B + m - 1 blocks of s samples, each scored for every lag as a
    // full block (pairs up to the trace end) and as a cut block (pairs up to
    // the end of the block the lag's range stops in).
    bool sliding;
    int32_t m;               // N / s
    int64_t blocks;
    int64_t trace_len;
    int64_t block_chunk;     // samples per chunk of a block
    int32_t block_chunks;
    int64_t block_tasks;     // waves of each of the two block-partial launches
    // FFT scores: every (window, channel) sequence, centred and zero-padded to
    // fft_len = 2^fft_log2 >= N + Tmax, is paired with the next one as the real
    // and imaginary parts of one complex transform.  Up to 2^12 points one
    // workgroup transforms a pair in LDS; beyond that the transform is split
    // as fft_len = fft_m1 * fft_m2 (columns of fft_m1 points, rows of fft_m2).
    // A ragged FFT plan (windows from a table, of different lengths) gives
    // each pair the shortest transform its two sequences need: the pairs are
    // sorted into length classes 2^lg, lg in [kFftMinLog2, fft_log2], on the
    // GPU, and every class runs at its own length.
    bool fft;
    bool fft_ragged;
    int32_t fft_log2, fft_m1, fft_m2, fft_cols;
    int64_t fft_len;
    int64_t fft_pairs;
    // Wrap correction (uniform FFT plans): fft_len >= N only, so lags T > W =
    // fft_len - N also collect the circular term sum_{j < T-W} y_j y_{j+L-T},
    // the cross-correlation at shift Tmax - T of the first and the last M =
    // Tmax - W samples of the sequence.  A second transform of
    // 2^fft_wrap_log2 >= 2M points per pair computes it, and it is subtracted.
    bool fft_wrap;
    int32_t fft_wrap_m, fft_wrap_log2;
    // Matrix-core scores: every sequence as four int8 digit planes of
    // mfma_plane bytes (padded); lag tiles of kMfmaTileLags from mfma_t0
    // (Tmin).
    bool mfma;
    bool mfma_table;         // windows from a table (rolling suffixes)
    int32_t mfma_t0, mfma_tiles;
    int32_t mfma_chunks;     // sample chunks per tile (1: one wave per tile)
    int64_t mfma_chunk_steps;   // 32-sample steps per chunk (even)
    int64_t mfma_plane;
    // Fused plans: after the lag scores, one kernel (one workgroup per window)
    // computes the statistics, finalises the scores and runs the whole
    // selection, re-scoring in place: direct scores of windows of at most
    // kFusedMaxN samples, each scored on its own (no table, no shared blocks).
    bool fused;
    bool tiny;               // lag_score_tiny_kernel (t0 = tmin, kTinyLags-lag blocks,
                             // kTinyChunk-sample chunks)
    double c_lag, err_max;
    uint32_t flags;
    WindowTable table;       // per-window offsets / lengths / Tmax, or all null
    int32_t bitmap_words;    // 32-bit words per window of the exactness bitmap
    // workspace layout (byte offsets, 256-byte aligned)
    size_t off_var, off_s64, off_bits, off_state, off_queue, off_part, off_cut;
    size_t off_fstat, off_edge, off_tw, off_z, off_cls, off_zw, off_wrap, off_dig, off_qstat,
        off_rpart, bytes;
};

// Rolling detection (Algorithm 3).
struct RollingConfig {
    double c_measure, step, c_eval, diff_threshold;
    int32_t jmax;            // suffix-window slots per window
};

struct RollState {           // per window, between the schedule and the combination
    double err_a;            // err of the whole-window pass
    double short_next;       // next sampling duration when too short
    int32_t t_init;
    int32_t verdict_a;
    int32_t count;           // suffix windows scheduled
    uint32_t flags;
};

struct RollingCombineArgs {
    const float* x;
    const gpoeo_pd_result* res_c;   // [B * jmax] results of the suffix pass
    const double* s64;       // suffix pass workspace: scores, tiers, states, variances
    const uint32_t* tier1;
    const uint32_t* tier2;
    const WinState* wstate;
    const double* var;
    const RollState* state;
    gpoeo_pd_rolling_result* out;   // [B]
    const int64_t* tab_off;
    const int64_t* tab_n;
    int64_t lags;
    int64_t words;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t tmin;
    int32_t num_channels;
    int32_t jmax;
    double tau0;
    double tau1;
    double diff_threshold;
};

// Kernel launchers; each returns hipGetLastError() after enqueueing.
// var: [B][C][2] = population variance, mean |x| per window and channel.
// fstat (nullable): [B*C][4] = mean, sum (x - mean)^2, sum |x - mean|, 0.
hipError_t launch_window_stats(const Plan& p, const float* x, double* var, double* fstat,
                               hipStream_t s);
hipError_t launch_lag_score(const Plan& p, const float* x, double* part, hipStream_t s);
// Sliding mode: full-block partials into `full`, cut-block partials into `cut`,
// each [blocks*C + channel][block_chunks][lags_padded].
hipError_t launch_lag_score_blocks(const Plan& p, const float* x, double* full, double* cut,
                                   hipStream_t s);
hipError_t launch_finalize_blocks(const Plan& p, const Weights& w, const double* full,
                                  const double* cut, double* s64, float* scores, hipStream_t s);
hipError_t launch_finalize(const Plan& p, const Weights& w, const double* part, double* s64,
                           float* scores, hipStream_t s);
// FFT scores.  fstat: [B*C][4] = mean, sum of squares and sum of |.| of the
// centred sequence, and its absolute error bound on D(T); edge: [B*C][2][Tmax+1]
// prefix sums of squares from the head and from the tail; tw: twiddle tables;
// z: [pairs][fft_len] complex fp64.  Writes D_c(T) into part ([B*C][lags]).
// cls (ragged plans): [pairs] class of each pair, [pairs] pairs sorted by class,
// [kFftClasses + 1] start of each class; null otherwise.
int64_t fft_twiddle_count(const Plan& p);
int64_t fft_class_ints(const Plan& p);
// zw, wrap (wrap-corrected plans): [2][pairs][2^fft_wrap_log2] complex fp64
// head and tail transforms; [B*C][M] fp64 wrap terms.  Null otherwise.
// With one channel the transforms also do the finalisation: s64 and scores
// (nullable) receive S(T) = w_0 D(T) / (N - T) directly and `part` is not
// written.  Not for a window table (ragged plans) with fp32 scores requested:
// lags past a short window's transform are then zeroed by the finalisation.
inline bool fft_fused_finalize(const Plan& p, bool with_scores) {
    return p.fft && p.num_channels == 1 && (!p.fft_ragged || !with_scores);
}
hipError_t launch_fft_scores(const Plan& p, const float* x, double* fstat, double* edge,
                             double* tw, double* z, double* part, int32_t* cls, double* zw,
                             double* wrap, double* s64, float* scores, float w0,
                             hipStream_t s);
// After the finalisation: every lag whose FFT bound does not give the tier-0
// guarantee is re-scored in fp64 (score, fp32 score and tier-1 bit).
hipError_t launch_fft_fixup(const Plan& p, const Weights& w, const float* x, const double* fstat,
                            const int32_t* cls, double* s64, float* scores,
                            const SelectBuffers& sb, hipStream_t s);

// Matrix-core scores: per sequence the centre, scale and exactness (qstat
// [S][4]), the digit planes, the edge sums and D(T) into `part`, or with one
// channel S(T) straight into s64 and scores (nullable; not for a window table
// with fp32 scores requested, whose lags past a window's own Tmax the
// finalisation zeroes).  Then the fix-up of the lags whose bound exceeds half
// the tier-0 width, before the selection.
inline bool mfma_fused_finalize(const Plan& p, bool with_scores) {
    return p.mfma && p.num_channels == 1 && (!p.mfma_table || !with_scores);
}
hipError_t launch_mfma_scores(const Plan& p, const float* x, double* qstat, int8_t* dig,
                              double* edge, double* rpart, double* part, double* s64,
                              float* scores, float w0, hipStream_t s);
hipError_t launch_mfma_fixup(const Plan& p, const Weights& w, const float* x,
                             const double* qstat, double* s64, float* scores,
                             const SelectBuffers& sb, hipStream_t s);
hipError_t launch_select_init(const Plan& p, const SelectBuffers& sb, hipStream_t s);
// Spectral candidates (Algorithm 1's FFT front end) of every window: a plan
// whose FFT geometry is that of L = 2^k >= N; amp: [B*C][L/2 + 1] fp64.
hipError_t launch_spectral(const Plan& p, const Weights& w, const float* x, const double* fstat,
                           double* tw, double* z, double* amp, double c_peak, int32_t k_max,
                           gpoeo_pd_spectral_result* out, hipStream_t s);
// Transform of 2^lg points: one workgroup (m2 = 1), or m1 columns of m2 rows
// with `cols` columns per column workgroup.
void fft_geometry(int32_t lg, int32_t* m1, int32_t* m2, int32_t* cols);
// Sets the transform geometry of a plan for 2^lg points; false if too large.
bool set_fft_geometry(Plan* p, int32_t lg);
hipError_t launch_select(const Plan& p, const Weights& w, const float* x, const double* var,
                         double* s64, const SelectBuffers& sb, void* results, hipStream_t s);
// Fused plans (p.fused): window statistics, finalisation of the lag-score
// partials and the whole selection with its re-scores, one workgroup per
// window, in one launch after the lag scores.
hipError_t launch_finish(const Plan& p, const Weights& w, const float* x, double* var,
                         const double* part, double* s64, float* scores,
                         const SelectBuffers& sb, void* results, hipStream_t s);
hipError_t launch_rolling_schedule(const Plan& p, const RollingConfig& rc,
                                   const gpoeo_pd_result* res_a, int64_t* tab_off, int64_t* tab_n,
                                   int32_t* tab_tmax, RollState* state, hipStream_t s);
hipError_t launch_rolling_combine(const RollingCombineArgs& a, const Weights& w,
                                  int64_t num_windows, hipStream_t s);
hipError_t launch_centred(const Plan& p, const Weights& w, const float* x, const int32_t* windows,
                          const int32_t* lags, int64_t count, double* out, hipStream_t s);
// flags (nullable): [count] GPOEO_PD_UNRESOLVED where a hard label is fragile.
hipError_t launch_similarity(const Plan& p, const Weights& w, int32_t groups, int32_t iters,
                             const float* x, const int32_t* windows, const int32_t* lags,
                             int64_t count, double* err, uint32_t* flags, hipStream_t s);

}  // namespace gpoeo
