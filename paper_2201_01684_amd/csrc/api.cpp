// C ABI of libgpoeo_pd: argument validation, launch plan, workspace layout and
// the kernel sequence (window statistics, lag scores, finalisation, selection).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <algorithm>
#include <cstring>

#include "gpoeo_pd.h"
#include "internal.h"

namespace gpoeo {
namespace {

// Enough score wavefronts for about 8 rounds of 5 resident waves on each of
// the 1024 SIMDs, so that the last, partly filled round costs little.
constexpr int64_t kTargetWaves = 40960;
constexpr size_t kAlign = 256;

}  // namespace

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

namespace {

// Lags per lane of the score kernel.  16 lets each staged sample serve more
// lags and suits long windows; 8 halves the masked stretch at the end of each
// lag block (64 * 16 samples at 16 lags per lane) and doubles occupancy (59
// instead of 92 VGPRs), which pays once that stretch exceeds about 1% of the
// mean pair range N - T.  Measured on MI355X with the grouped differences
// and the four-wave bound of the sixteen-lag instance: 16 is best for 262144-
// and 131072-sample windows (1.5% ahead of 8 on the latter), 8 for 65536- and
// 16384-sample windows (3-6% ahead of 16 on the former).
int32_t choose_lags_per_lane(int64_t n, int32_t tmin, int32_t tmax) {
    const double mean_range = (double)n - 0.5 * ((double)tmin + (double)tmax);
    return (64.0 * 16.0 > 0.01 * mean_range) ? 8 : 16;
}

// Wavefronts per score workgroup: with 8 lags per lane, single-wave groups
// measured faster (no wave of a group waits on a longer sibling).
int32_t choose_waves_per_group(int32_t lags_per_lane) { return lags_per_lane == 8 ? 1 : 4; }

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
    if (a < 0 || b < 0) return false;
    if (a != 0 && b > INT64_MAX / a) return false;
    *out = a * b;
    return true;
}

}  // namespace

void fft_geometry(int32_t lg, int32_t* m1, int32_t* m2, int32_t* cols) {
    const int tile = fft_tile_log2(lg);
    if (lg <= tile) {
        *m1 = 1 << lg;
        *m2 = 1;
        *cols = 1;
    } else {
        const int32_t lg1 = lg / 2, lg2 = lg - lg1;   // a row pair fits one tile
        *m1 = 1 << lg1;
        *m2 = 1 << lg2;
        *cols = std::min<int32_t>(*m2, 1 << (tile - lg1));
    }
}

bool set_fft_geometry(Plan* p, int32_t lg) {
    if (lg > kFftMaxLog2) return false;
    p->fft_log2 = lg;
    p->fft_len = int64_t(1) << lg;
    fft_geometry(lg, &p->fft_m1, &p->fft_m2, &p->fft_cols);
    return true;
}

namespace {

// Every launch of a plan must keep its global size (workgroups times threads)
// within HIP's 32-bit limit: one workgroup of up to 1024 threads per window
// (selection), 256 per (window, channel) sequence (statistics) or two (FFT
// edge sums), 64 per lag-score wave, 256 per transform tile.
bool launches_fit(const Plan& p) {
    const int64_t kMax = (int64_t(1) << 32) - 1;
    auto fits = [&](int64_t blocks, int64_t threads) { return blocks <= kMax / threads; };
    const int64_t seqs = p.num_windows * (int64_t)p.num_channels;
    if (!fits(p.num_windows, 1024) || !fits(seqs, 256)) return false;
    if (p.fft) {
        if (!fits(2 * seqs, 256)) return false;
        if (!p.fft_ragged) {   // uniform transforms: one workgroup per tile of each pair
            const int64_t per_pair =
                p.fft_m2 == 1 ? 1 : std::max<int64_t>(p.fft_m2 / p.fft_cols, p.fft_m1 / 2 + 1);
            if (p.fft_pairs > kMax / 256 / per_pair) return false;
        }
        if (p.fft_wrap) {
            int32_t m1, m2, cols;
            fft_geometry(p.fft_wrap_log2, &m1, &m2, &cols);
            const int64_t per_pair = std::max<int64_t>(m2 / cols, m1 / 2 + 1);
            if (p.fft_pairs > kMax / 256 / per_pair) return false;
        }
    } else if (p.mfma) {   // statistics and edge sums per sequence, four lag tiles a workgroup
        if (!fits(2 * seqs, 256) ||
            !fits((seqs + 7) / 8 * 8 * ((p.mfma_tiles + 3) / 4) * p.mfma_chunks, 256) ||
            !fits(seqs * ((p.lags + 255) / 256), 256))
            return false;
    } else if (p.sliding) {
        if (!fits(2 * p.block_tasks, kWave)) return false;   // the cut launch has twice the waves
    } else if (!fits(p.tasks, kWave)) {
        return false;
    }
    return true;
}

// ragged: the windows will come from a table (lengths up to d->n, Tmax up to
// d->tmax); an FFT plan then sizes its transforms per pair (length classes).
int make_plan(const gpoeo_pd_desc* d, Plan* p, bool ragged = false) {
    if (!d) return GPOEO_PD_EINVAL;
    if (d->reserved0 != 0 || d->reserved1 != 0) return GPOEO_PD_EINVAL;
    if (d->flags & ~(GPOEO_PD_SCORES_ONLY | GPOEO_PD_NO_RESCUE | GPOEO_PD_FFT_SCORES |
                     GPOEO_PD_MFMA_SCORES | GPOEO_PD_UNFUSED))
        return GPOEO_PD_EINVAL;
    const bool mfma = (d->flags & GPOEO_PD_MFMA_SCORES) != 0;
    // one score source per call
    if (mfma && (d->flags & GPOEO_PD_FFT_SCORES)) return GPOEO_PD_EINVAL;
    if (d->num_windows < 1 || d->num_windows > GPOEO_PD_MAX_WINDOWS) return GPOEO_PD_EINVAL;
    if (d->num_channels < 1 || d->num_channels > kMaxChannels) return GPOEO_PD_EINVAL;
    if (d->n < 8 || d->n > (int64_t(1) << 40)) return GPOEO_PD_EINVAL;
    if (d->tmin < 1 || (int64_t)d->tmin + 2 > (int64_t)d->tmax || (int64_t)d->tmax > d->n / 2)
        return GPOEO_PD_EINVAL;
    if (d->window_stride < 0 || (d->num_windows > 1 && d->window_stride < 1))
        return GPOEO_PD_EINVAL;
    if (d->channel_stride < 0 || (d->num_channels > 1 && d->channel_stride < d->n))
        return GPOEO_PD_EINVAL;
    if (!(d->c_lag > 0.0 && d->c_lag < 1.0)) return GPOEO_PD_EINVAL;
    if (std::isnan(d->err_max)) return GPOEO_PD_EINVAL;
    if (d->channel_weights)
        for (int32_t c = 0; c < d->num_channels; ++c) {
            const float w = d->channel_weights[c];
            if (!(w > 0.0f) || !std::isfinite(w)) return GPOEO_PD_EINVAL;
        }

    std::memset(p, 0, sizeof(*p));
    p->num_windows = d->num_windows;
    p->num_channels = d->num_channels;
    p->n = d->n;
    p->window_stride = d->window_stride;
    p->channel_stride = d->channel_stride;
    p->tmin = d->tmin;
    p->tmax = d->tmax;
    p->lags = d->tmax - d->tmin + 1;
    p->c_lag = d->c_lag;
    p->err_max = d->err_max;
    p->flags = d->flags;

    p->fft = (d->flags & GPOEO_PD_FFT_SCORES) != 0;
    p->fft_ragged = p->fft && ragged;
    if (p->fft) {
        // smallest power of two (at least 64) holding N + Tmax points
        int32_t lg = kFftMinLog2;
        while ((int64_t(1) << lg) < d->n + d->tmax) ++lg;
        // Or one holding N, with the wrap correction, when that costs less:
        // four sweeps of a 2^lgn transform plus six of a 2^lgw one (two
        // forward, one inverse) against four sweeps of 2^(lgn+1); the
        // shorter transform must itself be a split one.
        int32_t lgn = kFftMinLog2;
        while ((int64_t(1) << lgn) < d->n) ++lgn;
        p->fft_wrap = false;
        if (!ragged && lgn < lg && lgn > kFftSmallTileLog2) {
            const int64_t m = (int64_t)d->tmax - ((int64_t(1) << lgn) - d->n);
            int32_t lgw = kFftWrapMinLog2;
            while ((int64_t(1) << lgw) < 2 * m) ++lgw;
            if (lgw <= lgn - 1 && lgw <= kFftWrapMaxLog2) {
                lg = lgn;
                p->fft_wrap = true;
                p->fft_wrap_m = (int32_t)m;
                p->fft_wrap_log2 = lgw;
            }
        }
        if (!set_fft_geometry(p, lg)) return GPOEO_PD_EINVAL;
    }

    p->lags_per_lane = choose_lags_per_lane(d->n, d->tmin, d->tmax);
    p->waves_per_group = choose_waves_per_group(p->lags_per_lane);
    const int32_t lags_per_block = kWave * p->lags_per_lane;
    p->lag_blocks = (p->lags + lags_per_block - 1) / lags_per_block;

    int64_t bc, base;
    if (!mul_ok(d->num_windows, d->num_channels, &bc)) return GPOEO_PD_EINVAL;

    // Overlapping windows whose stride divides N (and is a whole number of lag
    // blocks) share block partials when that saves at least a third of the work.
    const int64_t ws_ = d->window_stride;
    if (!p->fft && !mfma && d->num_windows >= 2 && ws_ > 0 && ws_ < d->n && d->n % ws_ == 0 &&
        ws_ % lags_per_block == 0) {
        const int64_t m = d->n / ws_;
        const double direct =
            (double)d->num_windows * ((double)d->n - 0.5 * ((double)d->tmin + (double)d->tmax));
        const double shared = (double)(d->num_windows + m - 1) * 1.5 * (double)ws_;
        if (direct > 1.5 * shared) {
            p->sliding = true;
            p->m = (int32_t)m;
            p->blocks = d->num_windows + m - 1;
            p->trace_len = (d->num_windows - 1) * ws_ + d->n;
        }
    }
    int64_t t0;
    if (p->sliding) {
        // lag blocks start at 1 (mod 64 * lags_per_lane), so that no block
        // straddles a multiple of the stride (the cut partials need one
        // floor((T - 1) / s) per wavefront)
        t0 = 1 + (int64_t)lags_per_block * ((d->tmin - 1) / lags_per_block);
        p->lag_blocks = (int32_t)((d->tmax - t0 + lags_per_block) / lags_per_block);
    } else {
        // lag blocks end exactly at tmax when possible, so that no block is
        // mostly outside [tmin, tmax]; lags below tmin are computed and discarded
        t0 = (int64_t)d->tmax + 1 - (int64_t)p->lag_blocks * lags_per_block;
        if (t0 < 0) t0 = 0;
    }
    p->t0 = (int32_t)t0;
    p->lags_padded = p->lag_blocks * lags_per_block;

    const int64_t kMinChunk = 128;
    if (!mul_ok(bc, p->lag_blocks, &base)) return GPOEO_PD_EINVAL;
    const int64_t span = d->n - p->t0;             // longest sample range of any lag
    {
        const int64_t max_chunks = (span + kMinChunk - 1) / kMinChunk;
        int64_t chunks = (kTargetWaves + base - 1) / base;
        if (chunks < 1) chunks = 1;
        if (chunks > max_chunks) chunks = max_chunks;
        int64_t chunk = (span + chunks - 1) / chunks;
        chunk = (chunk + kBlockSamples - 1) / kBlockSamples * kBlockSamples;
        chunks = (span + chunk - 1) / chunk;
        p->chunk = chunk;
        p->chunks = (int32_t)chunks;
        if (!mul_ok(base, chunks, &p->tasks)) return GPOEO_PD_EINVAL;
        if (p->tasks / p->waves_per_group + 1 > INT32_MAX) return GPOEO_PD_EINVAL;
    }
    if (p->sliding) {
        int64_t bbase;
        if (!mul_ok(p->blocks * d->num_channels, p->lag_blocks, &bbase)) return GPOEO_PD_EINVAL;
        // Two launches (full and cut partials) share the target, and every
        // extra chunk adds one partial per lag and block for the finalisation
        // to read, so blocks are split only when there are few of them.
        const int64_t max_chunks = (ws_ + kMinChunk - 1) / kMinChunk;
        int64_t chunks = (kTargetWaves / 4 + bbase - 1) / bbase;
        if (chunks < 1) chunks = 1;
        if (chunks > max_chunks) chunks = max_chunks;
        int64_t chunk = (ws_ + chunks - 1) / chunks;
        chunk = (chunk + kBlockSamples - 1) / kBlockSamples * kBlockSamples;
        chunks = (ws_ + chunk - 1) / chunk;
        p->block_chunk = chunk;
        p->block_chunks = (int32_t)chunks;
        if (!mul_ok(bbase, chunks, &p->block_tasks)) return GPOEO_PD_EINVAL;
        if (2 * p->block_tasks / p->waves_per_group + 1 > INT32_MAX) return GPOEO_PD_EINVAL;
    }
    if (p->fft) {   // one D(T) per (window, channel, lag), lags from tmin
        p->t0 = d->tmin;
        p->lags_padded = p->lags;
        p->chunks = 1;
        p->fft_pairs = (bc + 1) / 2;
    }
    p->mfma = mfma;
    p->mfma_table = mfma && ragged;
    if (p->mfma) {   // as FFT plans: one D(T) per (window, channel, lag)
        p->t0 = d->tmin;
        p->lags_padded = p->lags;
        p->chunks = 1;
        p->mfma_t0 = d->tmin;                     // lag tiles from Tmin: the lags past Tmax cost least
        p->mfma_tiles = (d->tmax - p->mfma_t0) / kMfmaTileLags + 1;
        p->mfma_plane = (kMfmaPadL + d->n + kMfmaPadR + 255) / 256 * 256;
        // steps of the first tile (the most), even; chunks when the waves are few
        const int64_t steps = ((d->n - p->mfma_t0 + 62) / 32 + 1) & ~int64_t(1);
        const int64_t waves = bc * (int64_t)p->mfma_tiles;
        int64_t k = (kMfmaTargetWaves + waves - 1) / waves;
        k = std::min<int64_t>(k, std::max<int64_t>(1, steps / kMfmaMinChunkSteps));
        int64_t cs = (steps + k - 1) / k;
        cs = (cs + 1) & ~int64_t(1);
        p->mfma_chunk_steps = cs;
        p->mfma_chunks = (int32_t)((steps + cs - 1) / cs);
    }
    p->bitmap_words = (p->lags + 31) / 32;
    {
        // Tiny plans: few pairs in short windows, each scored on its own.
        const double lags = (double)p->lags;
        const double pairs = (double)bc * lags * ((double)d->n - 0.5 * ((double)d->tmin + d->tmax));
        p->tiny = !p->fft && !mfma && !p->sliding && !ragged && d->n <= kFusedMaxN &&
                  pairs <= kTinyMaxPairs;
        if (p->tiny) {
            p->t0 = d->tmin;
            p->lag_blocks = (p->lags + kTinyLags - 1) / kTinyLags;
            p->lags_padded = p->lag_blocks * kTinyLags;
            p->chunk = kTinyChunk;
            p->chunks = (int32_t)((d->n - d->tmin + kTinyChunk - 1) / kTinyChunk);
            if (!mul_ok(bc * p->lag_blocks, (int64_t)p->chunks * (kTinyLags / kWave), &p->tasks))
                return GPOEO_PD_EINVAL;
        }
    }
    p->fused = !p->fft && !p->mfma && !p->sliding && !ragged && d->n <= kFusedMaxN &&
               p->lags <= kFusedMaxLags && !(d->flags & GPOEO_PD_UNFUSED);

    int64_t n_var, n_s, n_bits, n_part;
    if (!mul_ok(bc, 2, &n_var)) return GPOEO_PD_EINVAL;      // variance, mean |x|
    if (!mul_ok(d->num_windows, p->lags, &n_s)) return GPOEO_PD_EINVAL;
    if (!mul_ok(d->num_windows, p->bitmap_words, &n_bits)) return GPOEO_PD_EINVAL;
    int64_t tmp;
    if (p->sliding) {
        if (!mul_ok(p->blocks * d->num_channels, p->block_chunks, &tmp) ||
            !mul_ok(tmp, p->lags_padded, &n_part))
            return GPOEO_PD_EINVAL;
    } else {
        if (!mul_ok(bc, p->chunks, &tmp) || !mul_ok(tmp, p->lags_padded, &n_part))
            return GPOEO_PD_EINVAL;
    }
    if (n_part > (INT64_MAX / 16)) return GPOEO_PD_EINVAL;
    int64_t n_fstat = 0, n_edge = 0, n_tw = 0, n_z = 0, n_cls = 0, n_zw = 0, n_wrap = 0;
    int64_t n_dig = 0, n_qstat = 0, n_rpart = 0;
    if (p->mfma &&
        (!mul_ok(bc, 4, &n_qstat) || !mul_ok(bc, 2 * ((int64_t)d->tmax + 1), &n_edge) ||
         !mul_ok(bc, 4 * p->mfma_plane, &n_dig) || n_dig > (INT64_MAX / 4)))
        return GPOEO_PD_EINVAL;
    if (p->mfma && p->mfma_chunks > 1 &&   // per-chunk cross terms of every tile lag
        (!mul_ok(bc * p->mfma_chunks, (int64_t)p->mfma_tiles * kMfmaTileLags, &n_rpart) ||
         n_rpart > (INT64_MAX / 16)))
        return GPOEO_PD_EINVAL;
    if (p->fft) {
        if (!mul_ok(bc, 4, &n_fstat) || !mul_ok(bc, 2 * ((int64_t)d->tmax + 1), &n_edge) ||
            !mul_ok(p->fft_pairs, p->fft_len, &n_z) || n_z > (INT64_MAX / 64))
            return GPOEO_PD_EINVAL;
        n_tw = fft_twiddle_count(*p);
        n_cls = fft_class_ints(*p);
        if (p->fft_wrap &&
            (!mul_ok(2 * p->fft_pairs, int64_t(1) << p->fft_wrap_log2, &n_zw) ||
             n_zw > (INT64_MAX / 64) || !mul_ok(bc, p->fft_wrap_m, &n_wrap)))
            return GPOEO_PD_EINVAL;
    }
    size_t off = 0;
    p->off_var = off;
    off = align_up(off + (size_t)n_var * sizeof(double));
    p->off_s64 = off;
    off = align_up(off + (size_t)n_s * sizeof(double));
    p->off_bits = off;                            // four bitmaps
    off = align_up(off + 4 * (size_t)n_bits * sizeof(uint32_t));
    p->off_state = off;
    off = align_up(off + (size_t)d->num_windows * sizeof(WinState));
    p->off_queue = off;                           // q_win, q_lag, q_count
    off = align_up(off + (4 * (size_t)kQueueCap + 2 * kPasses) * sizeof(int32_t));
    p->off_part = off;
    off = align_up(off + (size_t)n_part * sizeof(double));
    p->off_cut = off;                             // cut-block partials (sliding mode)
    if (p->sliding) off = align_up(off + (size_t)n_part * sizeof(double));
    p->off_fstat = off;                           // FFT mode: per-sequence sums
    off = align_up(off + (size_t)n_fstat * sizeof(double));
    p->off_edge = off;                            // head and tail sums of squares
    off = align_up(off + (size_t)n_edge * sizeof(double));
    p->off_tw = off;                              // twiddle tables (complex fp64)
    off = align_up(off + (size_t)n_tw * 2 * sizeof(double));
    p->off_z = off;                               // transforms (complex fp64)
    off = align_up(off + (size_t)n_z * 2 * sizeof(double));
    p->off_cls = off;                             // length classes (ragged FFT plans)
    off = align_up(off + (size_t)n_cls * sizeof(int32_t));
    p->off_zw = off;                              // head and tail transforms (wrap)
    off = align_up(off + (size_t)n_zw * 2 * sizeof(double));
    p->off_wrap = off;                            // wrap terms
    off = align_up(off + (size_t)n_wrap * sizeof(double));
    p->off_dig = off;                             // matrix-core scores: int8 digit planes
    off = align_up(off + (size_t)n_dig);
    p->off_qstat = off;                           // centre, scale, exactness, sum X^2
    off = align_up(off + (size_t)n_qstat * sizeof(double));
    p->off_rpart = off;                           // per-chunk cross terms (chunked tiles)
    off = align_up(off + (size_t)n_rpart * sizeof(double));
    p->bytes = off;
    if (!launches_fit(*p)) return GPOEO_PD_EINVAL;
    return GPOEO_PD_OK;
}

}  // namespace
}  // namespace gpoeo

namespace {

struct Carved {
    double* var;
    double* s64;
    gpoeo::SelectBuffers sb;
    double* part;
    double* cut;
};

Carved carve(const gpoeo::Plan& p, void* workspace) {
    char* ws = static_cast<char*>(workspace);
    Carved c;
    c.var = reinterpret_cast<double*>(ws + p.off_var);
    c.s64 = reinterpret_cast<double*>(ws + p.off_s64);
    const size_t words = (size_t)p.num_windows * p.bitmap_words;
    uint32_t* bits = reinterpret_cast<uint32_t*>(ws + p.off_bits);
    int32_t* queue = reinterpret_cast<int32_t*>(ws + p.off_queue);
    c.sb.tier1 = bits;
    c.sb.tier2 = bits + words;
    c.sb.queued1 = bits + 2 * words;
    c.sb.queued2 = bits + 3 * words;
    c.sb.state = reinterpret_cast<gpoeo::WinState*>(ws + p.off_state);
    c.sb.q_win = queue;
    c.sb.q_lag = queue + 2 * gpoeo::kQueueCap;
    c.sb.q_count = queue + 4 * gpoeo::kQueueCap;
    c.part = reinterpret_cast<double*>(ws + p.off_part);
    c.cut = reinterpret_cast<double*>(ws + p.off_cut);
    return c;
}

gpoeo::Weights weights_of(const gpoeo_pd_desc* d, int32_t num_channels) {
    gpoeo::Weights w;
    for (int c = 0; c < gpoeo::kMaxChannels; ++c)
        w.w[c] = (d->channel_weights && c < num_channels) ? d->channel_weights[c] : 1.0f;
    return w;
}

bool x_aligned(const float* x, const gpoeo::Plan& p) {
    return (reinterpret_cast<uintptr_t>(x) % 16 == 0) &&
           (p.num_windows == 1 || p.window_stride % 4 == 0) &&
           (p.num_channels == 1 || p.channel_stride % 4 == 0);
}

// Enqueues the four stages of one plan (stats, scores, finalisation, selection).
int run_plan(const gpoeo::Plan& p, const gpoeo::Weights& w, const float* x, float* scores,
             gpoeo_pd_result* results, void* workspace, hipStream_t stream, hipEvent_t* ev) {
    const bool scores_only = (p.flags & GPOEO_PD_SCORES_ONLY) != 0;
    const Carved c = carve(p, workspace);
    auto mark = [&](int k) { return !ev || hipEventRecord(ev[k], stream) == hipSuccess; };
    if (!mark(0)) return GPOEO_PD_EHIP;
    double* fstat = p.fft ? reinterpret_cast<double*>(static_cast<char*>(workspace) + p.off_fstat)
                          : nullptr;
    if ((!scores_only || p.fft) && !p.fused &&
        gpoeo::launch_window_stats(p, x, c.var, fstat, stream) != hipSuccess)
        return GPOEO_PD_EHIP;
    if (!mark(1)) return GPOEO_PD_EHIP;
    if (p.fft) {
        char* ws = static_cast<char*>(workspace);
        int32_t* cls = p.fft_ragged ? reinterpret_cast<int32_t*>(ws + p.off_cls) : nullptr;
        double* zw = p.fft_wrap ? reinterpret_cast<double*>(ws + p.off_zw) : nullptr;
        double* wrap = p.fft_wrap ? reinterpret_cast<double*>(ws + p.off_wrap) : nullptr;
        if (gpoeo::launch_fft_scores(p, x, fstat, reinterpret_cast<double*>(ws + p.off_edge),
                                     reinterpret_cast<double*>(ws + p.off_tw),
                                     reinterpret_cast<double*>(ws + p.off_z), c.part, cls, zw,
                                     wrap, c.s64, scores, w.w[0], stream) != hipSuccess)
            return GPOEO_PD_EHIP;
        if (!mark(2)) return GPOEO_PD_EHIP;
        if ((!gpoeo::fft_fused_finalize(p, scores != nullptr) &&
             gpoeo::launch_finalize(p, w, c.part, c.s64, scores, stream) != hipSuccess) ||
            gpoeo::launch_select_init(p, c.sb, stream) != hipSuccess ||
            gpoeo::launch_fft_fixup(p, w, x, fstat, cls, c.s64, scores, c.sb, stream) !=
                hipSuccess)
            return GPOEO_PD_EHIP;
    } else if (p.mfma) {
        char* ws = static_cast<char*>(workspace);
        double* qstat = reinterpret_cast<double*>(ws + p.off_qstat);
        if (gpoeo::launch_mfma_scores(p, x, qstat, reinterpret_cast<int8_t*>(ws + p.off_dig),
                                      reinterpret_cast<double*>(ws + p.off_edge),
                                      reinterpret_cast<double*>(ws + p.off_rpart), c.part, c.s64,
                                      scores, w.w[0], stream) != hipSuccess)
            return GPOEO_PD_EHIP;
        if (!mark(2)) return GPOEO_PD_EHIP;
        if ((!gpoeo::mfma_fused_finalize(p, scores != nullptr) &&
             gpoeo::launch_finalize(p, w, c.part, c.s64, scores, stream) != hipSuccess) ||
            gpoeo::launch_select_init(p, c.sb, stream) != hipSuccess ||
            gpoeo::launch_mfma_fixup(p, w, x, qstat, c.s64, scores, c.sb, stream) != hipSuccess)
            return GPOEO_PD_EHIP;
    } else if (p.sliding) {
        if (gpoeo::launch_lag_score_blocks(p, x, c.part, c.cut, stream) != hipSuccess)
            return GPOEO_PD_EHIP;
        if (!mark(2)) return GPOEO_PD_EHIP;
        if (gpoeo::launch_finalize_blocks(p, w, c.part, c.cut, c.s64, scores, stream) != hipSuccess)
            return GPOEO_PD_EHIP;
    } else if (p.fused) {
        // statistics, finalisation and selection all run in the finish kernel
        // (timed as the finalisation stage; the other two stages are empty)
        if (gpoeo::launch_lag_score(p, x, c.part, stream) != hipSuccess) return GPOEO_PD_EHIP;
        if (!mark(2)) return GPOEO_PD_EHIP;
        if (gpoeo::launch_finish(p, w, x, c.var, c.part, c.s64, scores, c.sb, results, stream) !=
            hipSuccess)
            return GPOEO_PD_EHIP;
        if (!mark(3) || !mark(4)) return GPOEO_PD_EHIP;
        return GPOEO_PD_OK;
    } else {
        if (gpoeo::launch_lag_score(p, x, c.part, stream) != hipSuccess) return GPOEO_PD_EHIP;
        if (!mark(2)) return GPOEO_PD_EHIP;
        if (gpoeo::launch_finalize(p, w, c.part, c.s64, scores, stream) != hipSuccess)
            return GPOEO_PD_EHIP;
    }
    if (!mark(3)) return GPOEO_PD_EHIP;
    if (!scores_only) {
        if (!p.fft && !p.mfma && gpoeo::launch_select_init(p, c.sb, stream) != hipSuccess)
            return GPOEO_PD_EHIP;
        if (gpoeo::launch_select(p, w, x, c.var, c.s64, c.sb, results, stream) != hipSuccess)
            return GPOEO_PD_EHIP;
    }
    if (!mark(4)) return GPOEO_PD_EHIP;
    return GPOEO_PD_OK;
}

int detect_impl(const gpoeo_pd_desc* desc, const float* x, float* scores,
                gpoeo_pd_result* results, void* workspace, size_t workspace_bytes,
                hipStream_t stream, hipEvent_t* ev) {
    gpoeo::Plan p;
    const int rc = gpoeo::make_plan(desc, &p);
    if (rc != GPOEO_PD_OK) return rc;
    const bool scores_only = (p.flags & GPOEO_PD_SCORES_ONLY) != 0;
    if (!x || (!results && !scores_only) || !workspace) return GPOEO_PD_EINVAL;
    if (reinterpret_cast<uintptr_t>(workspace) % gpoeo::kAlign) return GPOEO_PD_EINVAL;
    if (reinterpret_cast<uintptr_t>(x) % sizeof(float)) return GPOEO_PD_EINVAL;
    if (workspace_bytes < p.bytes) return GPOEO_PD_ENOMEM;
    p.aligned = x_aligned(x, p);
    return run_plan(p, weights_of(desc, p.num_channels), x, scores, results, workspace, stream,
                    ev);
}

// Rolling detection: the whole-window plan, the suffix-window plan (a window
// table of B * jmax slots) and the workspace around them.
struct RollingPlan {
    gpoeo::Plan a, c;
    gpoeo::RollingConfig rc;
    size_t off_res_a, off_tab_off, off_tab_n, off_tab_tmax, off_res_c, off_state, off_detect;
    size_t bytes;
};

int make_rolling(const gpoeo_pd_desc* d, const gpoeo_pd_rolling_params* rp, RollingPlan* r) {
    if (!d || !rp) return GPOEO_PD_EINVAL;
    if (d->flags & GPOEO_PD_SCORES_ONLY) return GPOEO_PD_EINVAL;
    if (!(rp->c_measure > 0.0) || !(rp->step > 0.0) || !(rp->c_eval >= 0.0) ||
        !std::isfinite(rp->c_measure) || !std::isfinite(rp->step) ||
        !std::isfinite(rp->c_eval) || std::isnan(rp->diff_threshold))
        return GPOEO_PD_EINVAL;
    // Suffix windows per window: durations 2 + c_eval * step, minus k * step,
    // down to c_measure periods; one slot of margin for rounding.
    const double span = (2.0 + rp->c_eval * rp->step - rp->c_measure) / rp->step;
    if (!(span < GPOEO_PD_ROLLING_MAX)) return GPOEO_PD_EINVAL;
    const int32_t jmax = span < 0.0 ? 1 : (int32_t)std::floor(span) + 2;
    if (jmax > GPOEO_PD_ROLLING_MAX) return GPOEO_PD_EINVAL;
    int rc = gpoeo::make_plan(d, &r->a);
    if (rc != GPOEO_PD_OK) return rc;
    gpoeo_pd_desc dc = *d;
    if (d->num_windows > INT32_MAX / jmax) return GPOEO_PD_EINVAL;
    dc.num_windows = d->num_windows * jmax;
    dc.window_stride = d->n;     // placeholder: the window table gives every offset
    // The longest suffix starts at floor(D - (2 + c_eval step) T_init) (or 0), so
    // it holds at most (2 + c_eval step) Tmax + 2 samples: the suffix plan is
    // sized for that (its Tmax stays within half of it, as 2 + c_eval step >= 2).
    const double longest = std::ceil((2.0 + rp->c_eval * rp->step) * (double)d->tmax) + 2.0;
    if (longest < (double)d->n) dc.n = (int64_t)longest;
    rc = gpoeo::make_plan(&dc, &r->c, true);
    if (rc != GPOEO_PD_OK) return rc;
    r->rc.c_measure = rp->c_measure;
    r->rc.step = rp->step;
    r->rc.c_eval = rp->c_eval;
    r->rc.diff_threshold = rp->diff_threshold;
    r->rc.jmax = jmax;
    const size_t b = (size_t)d->num_windows, bj = b * jmax;
    size_t off = 0;
    r->off_res_a = off;
    off = gpoeo::align_up(off + b * sizeof(gpoeo_pd_result));
    r->off_tab_off = off;
    off = gpoeo::align_up(off + bj * sizeof(int64_t));
    r->off_tab_n = off;
    off = gpoeo::align_up(off + bj * sizeof(int64_t));
    r->off_tab_tmax = off;
    off = gpoeo::align_up(off + bj * sizeof(int32_t));
    r->off_res_c = off;
    off = gpoeo::align_up(off + bj * sizeof(gpoeo_pd_result));
    r->off_state = off;
    off = gpoeo::align_up(off + b * sizeof(gpoeo::RollState));
    r->off_detect = off;           // shared by the two detection passes, one after the other
    off = gpoeo::align_up(off + std::max(r->a.bytes, r->c.bytes));
    r->bytes = off;
    return GPOEO_PD_OK;
}

}  // namespace

extern "C" {

int gpoeo_pd_abi_version(void) { return GPOEO_PD_ABI_VERSION; }

const char* gpoeo_pd_strerror(int status) {
    switch (status) {
        case GPOEO_PD_OK: return "success";
        case GPOEO_PD_EINVAL: return "invalid argument";
        case GPOEO_PD_ENOMEM: return "workspace too small";
        case GPOEO_PD_EHIP: return "HIP launch failed";
        case GPOEO_PD_ETOOBIG: return "workspace larger than the static no-allocation scratch";
        default: return "unknown status";
    }
}

int gpoeo_pd_workspace_bytes(const gpoeo_pd_desc* desc, size_t* bytes) {
    if (!bytes) return GPOEO_PD_EINVAL;
    gpoeo::Plan p;
    const int rc = gpoeo::make_plan(desc, &p);
    if (rc != GPOEO_PD_OK) return rc;
    *bytes = p.bytes;
    return GPOEO_PD_OK;
}

int gpoeo_pd_describe_plan(const gpoeo_pd_desc* desc, gpoeo_pd_plan_info* info) {
    if (!info) return GPOEO_PD_EINVAL;
    gpoeo::Plan p;
    const int rc = gpoeo::make_plan(desc, &p);
    if (rc != GPOEO_PD_OK) return rc;
    info->mode = p.fft ? 2 : (p.mfma ? 3 : (p.sliding ? 1 : 0));
    info->lags_per_lane = p.lags_per_lane;
    info->score_waves = p.fft ? 0
                        : p.mfma ? (int64_t)p.num_windows * p.num_channels * p.mfma_tiles *
                                       p.mfma_chunks
                        : (p.sliding ? 3 * p.block_tasks : p.tasks);
    info->workspace_bytes = p.bytes;
    const double wc = (double)p.num_windows * p.num_channels;
    double defined = 0.0, scored = 0.0;
    for (int64_t t = p.tmin; t <= p.tmax; ++t) {
        defined += wc * (double)(p.n - t);
        if (!p.sliding) continue;
        const int64_t s = p.window_stride;
        const int64_t e = p.trace_len - t;          // positions whose partner exists
        const int64_t q = (t - 1) / s;
        const int64_t r = (q + 1) * s - t;          // pairs per cut block
        double cut = 0.0;
        if (e >= r) {
            int64_t full = (e - r) / s + 1;
            if (full > p.blocks) full = p.blocks;
            cut = (double)full * (double)r;
            if (full < p.blocks) cut += (double)std::max<int64_t>(0, e - full * s);
        } else {
            cut = (double)std::max<int64_t>(0, e);
        }
        scored += (double)p.num_channels * ((double)std::max<int64_t>(0, e) + cut);
    }
    info->pairs_defined = defined;
    info->pairs_scored = p.fft ? 0.0 : (p.sliding ? scored : defined);
    info->fft_len = p.fft ? p.fft_len : 0;
    info->fft_wrap_len = p.fft_wrap ? int64_t(1) << p.fft_wrap_log2 : 0;
    info->fft_wrap_lags = p.fft_wrap ? p.fft_wrap_m : 0;
    return GPOEO_PD_OK;
}

int gpoeo_pd_detect(const gpoeo_pd_desc* desc, const float* x, float* scores,
                    gpoeo_pd_result* results, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
    return detect_impl(desc, x, scores, results, workspace, workspace_bytes, stream, nullptr);
}

int gpoeo_pd_detect_staged(const gpoeo_pd_desc* desc, const float* x, float* scores,
                           gpoeo_pd_result* results, void* workspace, size_t workspace_bytes,
                           hipStream_t stream, hipEvent_t stage_events[5]) {
    if (!stage_events) return GPOEO_PD_EINVAL;
    for (int k = 0; k < 5; ++k)
        if (!stage_events[k]) return GPOEO_PD_EINVAL;
    return detect_impl(desc, x, scores, results, workspace, workspace_bytes, stream,
                       stage_events);
}

}  // extern "C"

extern "C" {

int gpoeo_pd_rolling_workspace_bytes(const gpoeo_pd_desc* desc,
                                     const gpoeo_pd_rolling_params* params, size_t* bytes) {
    if (!bytes) return GPOEO_PD_EINVAL;
    RollingPlan r;
    const int rc = make_rolling(desc, params, &r);
    if (rc != GPOEO_PD_OK) return rc;
    *bytes = r.bytes;
    return GPOEO_PD_OK;
}

int gpoeo_pd_detect_rolling(const gpoeo_pd_desc* desc, const gpoeo_pd_rolling_params* params,
                            const float* x, gpoeo_pd_rolling_result* results, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
    RollingPlan r;
    int rc = make_rolling(desc, params, &r);
    if (rc != GPOEO_PD_OK) return rc;
    if (!x || !results || !workspace) return GPOEO_PD_EINVAL;
    if (reinterpret_cast<uintptr_t>(workspace) % gpoeo::kAlign) return GPOEO_PD_EINVAL;
    if (reinterpret_cast<uintptr_t>(x) % sizeof(float)) return GPOEO_PD_EINVAL;
    if (workspace_bytes < r.bytes) return GPOEO_PD_ENOMEM;
    char* ws = static_cast<char*>(workspace);
    auto* res_a = reinterpret_cast<gpoeo_pd_result*>(ws + r.off_res_a);
    auto* tab_off = reinterpret_cast<int64_t*>(ws + r.off_tab_off);
    auto* tab_n = reinterpret_cast<int64_t*>(ws + r.off_tab_n);
    auto* tab_tmax = reinterpret_cast<int32_t*>(ws + r.off_tab_tmax);
    auto* res_c = reinterpret_cast<gpoeo_pd_result*>(ws + r.off_res_c);
    auto* state = reinterpret_cast<gpoeo::RollState*>(ws + r.off_state);
    void* detect_ws = ws + r.off_detect;
    const gpoeo::Weights w = weights_of(desc, r.a.num_channels);

    r.a.aligned = x_aligned(x, r.a);
    rc = run_plan(r.a, w, x, nullptr, res_a, detect_ws, stream, nullptr);
    if (rc != GPOEO_PD_OK) return rc;
    if (gpoeo::launch_rolling_schedule(r.a, r.rc, res_a, tab_off, tab_n, tab_tmax, state,
                                       stream) != hipSuccess)
        return GPOEO_PD_EHIP;
    r.c.table.off = tab_off;
    r.c.table.n = tab_n;
    r.c.table.tmax = tab_tmax;
    r.c.aligned = false;         // suffix windows start at any sample
    rc = run_plan(r.c, w, x, nullptr, res_c, detect_ws, stream, nullptr);
    if (rc != GPOEO_PD_OK) return rc;
    const Carved cv = carve(r.c, detect_ws);
    gpoeo::RollingCombineArgs ca;
    ca.x = x;
    ca.res_c = res_c;
    ca.s64 = cv.s64;
    ca.tier1 = cv.sb.tier1;
    ca.tier2 = cv.sb.tier2;
    ca.wstate = cv.sb.state;
    ca.var = cv.var;
    ca.state = state;
    ca.out = results;
    ca.tab_off = tab_off;
    ca.tab_n = tab_n;
    ca.lags = r.c.lags;
    ca.words = r.c.bitmap_words;
    ca.n = r.a.n;
    ca.window_stride = r.a.window_stride;
    ca.channel_stride = r.a.channel_stride;
    ca.tmin = r.a.tmin;
    ca.num_channels = r.a.num_channels;
    ca.jmax = r.rc.jmax;
    const double u = 1.1102230246251565e-16;
    ca.tau0 = r.c.fft ? gpoeo::kFftRelBound : gpoeo::kScoreRelBound;
    ca.tau1 = 1.01 * u * ((double)r.c.n * (1.0 + 1.0 / 256.0) + 2.0 * r.c.num_channels + 22.0);
    ca.diff_threshold = r.rc.diff_threshold;
    if (gpoeo::launch_rolling_combine(ca, w, r.a.num_windows, stream) != hipSuccess)
        return GPOEO_PD_EHIP;
    return GPOEO_PD_OK;
}

}  // extern "C"

namespace {

int similarity_impl(const gpoeo_pd_desc* desc, const gpoeo_pd_similarity_params* params,
                    const float* x, const int32_t* windows, const int32_t* lags, int64_t count,
                    double* err, uint32_t* flags, hipStream_t stream) {
    gpoeo::Plan p;
    const int rc = gpoeo::make_plan(desc, &p);
    if (rc != GPOEO_PD_OK) return rc;
    if (!params || params->num_groups < 1 || params->num_groups > 8 || params->em_iters < 0)
        return GPOEO_PD_EINVAL;
    if (count < 0 || count > GPOEO_PD_MAX_QUERIES) return GPOEO_PD_EINVAL;
    if (count == 0) return GPOEO_PD_OK;
    if (!x || !windows || !lags || !err) return GPOEO_PD_EINVAL;
    if (gpoeo::launch_similarity(p, weights_of(desc, p.num_channels), params->num_groups,
                                 params->em_iters, x, windows, lags, count, err, flags,
                                 stream) != hipSuccess)
        return GPOEO_PD_EHIP;
    return GPOEO_PD_OK;
}

}  // namespace

extern "C" int gpoeo_pd_similarity(const gpoeo_pd_desc* desc,
                                   const gpoeo_pd_similarity_params* params, const float* x,
                                   const int32_t* windows, const int32_t* lags, int64_t count,
                                   double* err, hipStream_t stream) {
    return similarity_impl(desc, params, x, windows, lags, count, err, nullptr, stream);
}

extern "C" int gpoeo_pd_similarity_flagged(const gpoeo_pd_desc* desc,
                                           const gpoeo_pd_similarity_params* params,
                                           const float* x, const int32_t* windows,
                                           const int32_t* lags, int64_t count, double* err,
                                           uint32_t* flags, hipStream_t stream) {
    if (count > 0 && !flags) return GPOEO_PD_EINVAL;
    return similarity_impl(desc, params, x, windows, lags, count, err, flags, stream);
}

extern "C" int gpoeo_pd_score_centred(const gpoeo_pd_desc* desc, const float* x,
                                      const int32_t* windows, const int32_t* lags, int64_t count,
                                      double* score, hipStream_t stream) {
    gpoeo::Plan p;
    const int rc = gpoeo::make_plan(desc, &p);
    if (rc != GPOEO_PD_OK) return rc;
    if (count < 0 || count > GPOEO_PD_MAX_QUERIES) return GPOEO_PD_EINVAL;
    if (count == 0) return GPOEO_PD_OK;
    if (!x || !windows || !lags || !score) return GPOEO_PD_EINVAL;
    if (gpoeo::launch_centred(p, weights_of(desc, p.num_channels), x, windows, lags, count, score,
                              stream) != hipSuccess)
        return GPOEO_PD_EHIP;
    return GPOEO_PD_OK;
}

namespace {

// Spectral candidates: the descriptor's window layout and lag range, an FFT
// geometry for L = 2^k >= N, and the workspace (window statistics, twiddles,
// transforms, amplitudes).
struct SpectralPlan {
    gpoeo::Plan p;
    size_t off_var, off_fstat, off_tw, off_z, off_amp, bytes;
};

int make_spectral(const gpoeo_pd_desc* d, const gpoeo_pd_spectral_params* sp, SpectralPlan* r) {
    if (!d || !sp) return GPOEO_PD_EINVAL;
    if (!(sp->c_peak > 0.0 && sp->c_peak < 1.0) || sp->reserved != 0 || sp->max_candidates < 1 ||
        sp->max_candidates > GPOEO_PD_SPECTRAL_MAX)
        return GPOEO_PD_EINVAL;
    gpoeo_pd_desc dd = *d;
    dd.flags = 0;
    const int rc = gpoeo::make_plan(&dd, &r->p);
    if (rc != GPOEO_PD_OK) return rc;
    int32_t lg = 6;
    while ((int64_t(1) << lg) < d->n) ++lg;
    if (!gpoeo::set_fft_geometry(&r->p, lg)) return GPOEO_PD_EINVAL;
    r->p.fft = true;
    r->p.table = gpoeo::WindowTable{nullptr, nullptr, nullptr};
    const int64_t seqs = d->num_windows * (int64_t)d->num_channels;
    r->p.fft_pairs = (seqs + 1) / 2;
    int64_t n_z = 0, n_amp = 0;
    if (!gpoeo::mul_ok(r->p.fft_pairs, r->p.fft_len, &n_z) || n_z > (INT64_MAX / 64) ||
        !gpoeo::mul_ok(seqs, r->p.fft_len / 2 + 1, &n_amp) || n_amp > (INT64_MAX / 16))
        return GPOEO_PD_EINVAL;
    if (r->p.fft_m2 == 1) n_z = 0;                 // one workgroup per pair: no transform buffer
    size_t off = 0;
    r->off_var = off;
    off = gpoeo::align_up(off + (size_t)seqs * 2 * sizeof(double));
    r->off_fstat = off;
    off = gpoeo::align_up(off + (size_t)seqs * 4 * sizeof(double));
    r->off_tw = off;
    off = gpoeo::align_up(off + (size_t)gpoeo::fft_twiddle_count(r->p) * 2 * sizeof(double));
    r->off_z = off;
    off = gpoeo::align_up(off + (size_t)n_z * 2 * sizeof(double));
    r->off_amp = off;
    off = gpoeo::align_up(off + (size_t)n_amp * sizeof(double));
    r->bytes = off;
    return GPOEO_PD_OK;
}

}  // namespace

extern "C" {

int gpoeo_pd_spectral_workspace_bytes(const gpoeo_pd_desc* desc,
                                      const gpoeo_pd_spectral_params* params, size_t* bytes) {
    if (!bytes) return GPOEO_PD_EINVAL;
    SpectralPlan r;
    const int rc = make_spectral(desc, params, &r);
    if (rc != GPOEO_PD_OK) return rc;
    *bytes = r.bytes;
    return GPOEO_PD_OK;
}

int gpoeo_pd_spectral_candidates(const gpoeo_pd_desc* desc, const gpoeo_pd_spectral_params* params,
                                 const float* x, gpoeo_pd_spectral_result* results,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream) {
    SpectralPlan r;
    const int rc = make_spectral(desc, params, &r);
    if (rc != GPOEO_PD_OK) return rc;
    if (!x || !results || !workspace) return GPOEO_PD_EINVAL;
    if (reinterpret_cast<uintptr_t>(workspace) % gpoeo::kAlign) return GPOEO_PD_EINVAL;
    if (reinterpret_cast<uintptr_t>(x) % sizeof(float)) return GPOEO_PD_EINVAL;
    if (workspace_bytes < r.bytes) return GPOEO_PD_ENOMEM;
    char* ws = static_cast<char*>(workspace);
    double* var = reinterpret_cast<double*>(ws + r.off_var);
    double* fstat = reinterpret_cast<double*>(ws + r.off_fstat);
    const gpoeo::Weights w = weights_of(desc, r.p.num_channels);
    if (gpoeo::launch_window_stats(r.p, x, var, fstat, stream) != hipSuccess) return GPOEO_PD_EHIP;
    if (gpoeo::launch_spectral(r.p, w, x, fstat, reinterpret_cast<double*>(ws + r.off_tw),
                               reinterpret_cast<double*>(ws + r.off_z),
                               reinterpret_cast<double*>(ws + r.off_amp), params->c_peak,
                               params->max_candidates, results, stream) != hipSuccess)
        return GPOEO_PD_EHIP;
    return GPOEO_PD_OK;
}

}  // extern "C"
