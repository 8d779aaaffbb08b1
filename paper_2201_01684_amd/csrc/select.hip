// Period selection per window (Algorithm 1 of Sec. 4.1.2, in the lag domain),
// with exact re-decision of every comparison the score error bound leaves open.
//
// Rule (one workgroup per window):
//   R      = 2 * sum_c w_c * Var_c; R == 0 -> CONSTANT
//   peaks  = { Tmin < T < Tmax : S(T) < S(T-1) and S(T) <= S(T+1) }
//            (Algorithm 1's "find peaks": interior local minima of the score;
//            strict on the left so a flat bottom contributes its first lag)
//   S_pk   = min S over peaks; thr = R - c_lag * (R - S_pk)
//            (candidate filter "peak > c_peak * max peak" on the height 1 - S/R)
//   T_c    = smallest peak with S(T) < thr (the fundamental; the spectrum of a
//            periodic signal has no component at multiples of its period)
//   window = [max(Tmin, ceil(T_c D / (D + T_c))), min(Tmax, floor(T_c D / (D - T_c)))],
//            D = N - 1: the periods of the two neighbouring Fourier bins of
//            T_c = D / k, i.e. Algorithm 1's local search at a one-sample step
//   period = smallest T in the window attaining min S; err = S(period) / R
//
// Every score carries a tier and is handled as an interval [v(1-e), v(1+e)]
// that contains the value a plain sequential fp64 evaluation of the definition
// gives:
//   tier 0  from the score kernels: e = kScoreRelBound for fp32 runs combined
//           in fp64, kFftRelBound for the fp64 FFT scores (whose lags without
//           that guarantee were raised to tier 1 before the first pass)
//   tier 1  re-scored in fp64 by one wavefront (64 strided partial sums and a
//           fixed-order tree): e = tau1, derived from N (about 3e-11 at
//           N = 262144) - it covers the rounding of both evaluation orders
//   tier 2  re-scored as the plain sequential fp64 sum itself (ascending i,
//           one rounding per operation, no contraction): a point
// R is an fp64 two-pass value whose distance to the sequential evaluation is
// bounded from N, the variances and the mean absolute samples (see
// reference_bound), or a point once recomputed sequentially.  A comparison the intervals decide is final.
// Otherwise the lags involved are queued for the next tier (R for a point),
// a re-score kernel spread over the whole GPU raises them, and the rule runs
// again.  The launcher runs kPasses selection passes with a re-score round
// between consecutive ones; a window still open in the last pass is decided
// on the unwidened values and flagged GPOEO_PD_UNRESOLVED.
#include <algorithm>

#include "internal.h"
#include "exact.h"
#include "gpoeo_pd.h"
#include "stats.h"

namespace gpoeo {
namespace {

using exact::exact_reference;
using exact::exact_score;
using exact::reference_bound;
using exact::group_score;

constexpr int kThreads = 256;       // re-score and initialisation kernels and short windows
// Selection passes run one workgroup per window; from this many lags on, four
// times as many threads keep more of a window's scores in flight.  A window
// table (suffix windows, mostly far shorter than the plan's lag range) keeps
// the narrow workgroups: more windows in flight at once; so does a batch of
// more than kChunkWideWindows windows whose scans stream through LDS in
// chunks.
constexpr int kWideLags = 4096;
constexpr int kRescoreGroups = 1024;   // workgroups of one re-score round
constexpr int64_t kChunkWideWindows = 256;   // MI355X's CUs: one 1024-thread workgroup each

struct SelectArgs {
    const float* x;
    const double* var;       // [B][C][2]: variance, mean |x|
    double* s64;             // [B][L], overwritten in place by re-scores
    uint32_t* tier1;         // [B][words]: value is tier >= 1
    uint32_t* tier2;         // [B][words]: value is tier 2
    uint32_t* queued1;       // [B][words]: queued for a tier-1 re-score
    uint32_t* queued2;       // [B][words]: queued for a tier-2 re-score
    WinState* state;         // [B]
    int32_t* q_win;          // [2][kQueueCap] queued (window, lag) pairs, per tier
    int32_t* q_lag;          //   lag -1 in the tier-2 queue: R of that window
    int32_t* q_count;        // [kPasses][2] queue lengths per round and tier
    gpoeo_pd_result* results;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t num_channels;
    int32_t tmin, tmax, lags, words;
    double c_lag, err_max, tau0, tau1;
    uint32_t flags;
    int32_t pass;
    int32_t last;
    int32_t stage;           // select passes copy a window's scores and tier bitmaps to LDS
    int32_t chunk;           // ... or stream them through LDS a chunk of lags at a time
    WindowTable tab;
};

enum Tri : int { kNo = 0, kYes = 1, kUnk = 2 };

struct Iv {
    double lo, hi, v;
    bool exact;
};

__device__ __forceinline__ Tri lt(const Iv& a, const Iv& b) {
    if (a.hi < b.lo) return kYes;
    if (a.lo >= b.hi) return kNo;
    return kUnk;
}
__device__ __forceinline__ Tri le(const Iv& a, const Iv& b) {
    if (a.hi <= b.lo) return kYes;
    if (a.lo > b.hi) return kNo;
    return kUnk;
}

// Wavefront reductions with DPP lane moves (VALU operations, where a lane
// shuffle is a round trip through the LDS unit): a butterfly inside each quad,
// then each lane with its mirror in the other half row and in the other half
// of the row, so that every lane of a row of 16 holds the row's value; then
// lane 15 of rows 0 and 2 into rows 1 and 3, and lane 31 into rows 2 and 3,
// so that lane 63 holds the wavefront's value.  Rows a broadcast does not
// enable take the operation's identity.  (min and integer sums: the result
// does not depend on the order.)
constexpr int kDppQuadXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;

template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint64_t dpp64(uint64_t v, uint64_t old) {
    const int lo = __builtin_amdgcn_update_dpp((int)(uint32_t)old, (int)(uint32_t)v, kCtrl,
                                               kRowMask, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(old >> 32), (int)(uint32_t)(v >> 32),
                                               kCtrl, kRowMask, 0xF, false);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// op(v, v of the lane kCtrl selects) for the three kinds of value
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double dpp_min_d(double v) {
    const uint64_t id = (uint64_t)__double_as_longlong(INFINITY);
    return fmin(v, __longlong_as_double((long long)dpp64<kCtrl, kRowMask>(
                       (uint64_t)__double_as_longlong(v), id)));
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int64_t dpp_sum_i(int64_t v) {
    return v + (int64_t)dpp64<kCtrl, kRowMask>((uint64_t)v, 0u);
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int64_t dpp_min_i(int64_t v) {
    return min(v, (int64_t)dpp64<kCtrl, kRowMask>((uint64_t)v, (uint64_t)INT64_MAX));
}

__device__ __forceinline__ double wave_min_d(double v) {
    v = dpp_min_d<kDppQuadXor1, 0xF>(v);
    v = dpp_min_d<kDppQuadXor2, 0xF>(v);
    v = dpp_min_d<kDppRowHalfMirror, 0xF>(v);
    v = dpp_min_d<kDppRowMirror, 0xF>(v);
    v = dpp_min_d<kDppRowBcast15, 0xA>(v);
    return dpp_min_d<kDppRowBcast31, 0xC>(v);
}

// Block reductions: the wavefront reductions above, the per-wave results
// (lane 63) through LDS, then every thread folds them in wave order.
template <int kT>
__device__ double block_min_d(double v, double* red) {
    v = wave_min_d(v);
    if ((threadIdx.x & (kWave - 1)) == kWave - 1) red[threadIdx.x / kWave] = v;
    __syncthreads();
    double r = red[0];
    for (int w = 1; w < kT / kWave; ++w) r = fmin(r, red[w]);
    __syncthreads();
    return r;
}

// The reductions of one step of the rule at once (one exchange through LDS,
// two barriers): three double minima, two int64 sums and one int64 minimum
// (unused ones are passed as neutral values).  Wavefront reductions, then the
// per-wave values folded in wave order; every thread gets the results.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ void reduce_step(double (&dmin)[3], int64_t (&isum)[2], int64_t& imin) {
#pragma unroll
    for (int k = 0; k < 3; ++k) dmin[k] = dpp_min_d<kCtrl, kRowMask>(dmin[k]);
#pragma unroll
    for (int k = 0; k < 2; ++k) isum[k] = dpp_sum_i<kCtrl, kRowMask>(isum[k]);
    imin = dpp_min_i<kCtrl, kRowMask>(imin);
}

template <int kT, typename Sh>
__device__ void block_reduce(double (&dmin)[3], int64_t (&isum)[2], int64_t& imin, Sh& sh) {
    reduce_step<kDppQuadXor1, 0xF>(dmin, isum, imin);
    reduce_step<kDppQuadXor2, 0xF>(dmin, isum, imin);
    reduce_step<kDppRowHalfMirror, 0xF>(dmin, isum, imin);
    reduce_step<kDppRowMirror, 0xF>(dmin, isum, imin);
    reduce_step<kDppRowBcast15, 0xA>(dmin, isum, imin);
    reduce_step<kDppRowBcast31, 0xC>(dmin, isum, imin);
    const int wv = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == kWave - 1) {
#pragma unroll
        for (int k = 0; k < 3; ++k) sh.red_md[k][wv] = dmin[k];
#pragma unroll
        for (int k = 0; k < 2; ++k) sh.red_ms[k][wv] = isum[k];
        sh.red_mi[wv] = imin;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        double r = sh.red_md[k][0];
        for (int w = 1; w < kT / kWave; ++w) r = fmin(r, sh.red_md[k][w]);
        dmin[k] = r;
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        int64_t r = sh.red_ms[k][0];
        for (int w = 1; w < kT / kWave; ++w) r += sh.red_ms[k][w];
        isum[k] = r;
    }
    int64_t r = sh.red_mi[0];
    for (int w = 1; w < kT / kWave; ++w) r = min(r, sh.red_mi[w]);
    imin = r;
    __syncthreads();
}

// Windows of up to this many lags keep the outcome of the first peak scan
// (bit t - tmin set: a decided peak) in LDS, so that the later scans test a
// bit instead of evaluating three score intervals again.
constexpr int kPeakWords = 2048;

template <int kT>
struct Shared {
    double red_d[kT / kWave];
    double red_d2[kT / kWave];
    int64_t red_i[kT / kWave];
    int64_t red_j[kT / kWave];
    double red_md[3][kT / kWave];     // multi-value reductions: double minima,
    int64_t red_ms[2][kT / kWave];    //   int64 sums,
    int64_t red_mi[kT / kWave];       //   one int64 minimum
    uint32_t peaks[kPeakWords];
    int done;
    double r_approx;
    double r_err;
};

// Where the rule reads window b's fp64 scores and tier bitmaps and marks its
// re-score requests: the workspace (global), or copies in LDS (fused kernel).
struct WindowView {
    const double* s;
    const uint32_t* t1;
    const uint32_t* t2;
    uint32_t* qd1;
    uint32_t* qd2;
    // Deferred requests (selection passes of windows of at most 32 kReqWords
    // lags): qd1 and qd2 above are this pass's request bitmaps in LDS, and
    // these are the window's queued bitmaps in the workspace, which the
    // requests join after the rule (one aggregated append per wavefront).
    uint32_t* gq1;
    uint32_t* gq2;
    // Windows not staged whole (too long, or too many of them): an LDS buffer
    // for the scores and tier words of one chunk of lags (ChunkGeom), or null.
    double* cs;
    uint32_t* ct1;
    uint32_t* ct2;
};

// The chunks of a workgroup of kT threads: 4 kT scores (4 kT - 2 lags and one
// neighbour either side), four loads a thread, and the tier words they touch.
template <int kT>
struct ChunkGeom {
    static constexpr int kEntries = 4 * kT;
    static constexpr int kLags = kEntries - 2;
    static constexpr int kWords = kEntries / 32 + 2;
    static constexpr size_t kBytes = sizeof(double) * kEntries + 2 * sizeof(uint32_t) * kWords;
};

// One evaluation of the rule for window b (every thread of the workgroup
// calls it).  Returns true once the window's result is written (now or in an
// earlier pass).  Requests for higher tiers are marked in the window's queued
// bitmaps; kLocal = false also appends them to the global re-score queues
// (one re-score kernel serves every window), at once or, with view.gq1 set,
// all together after the rule; kLocal = true leaves them to the caller, which
// re-scores the marked lags of its own window.
template <int kSelThreads, bool kLocal>
__device__ bool select_window(const SelectArgs& a, const Weights& w, int64_t b, int pass,
                              bool last, Shared<kSelThreads>& sh, const WindowView& view) {
    const int tid = threadIdx.x;
    const int32_t tmin = a.tmin;
    const int32_t tmax = table_tmax(a.tab, b, a.tmax);   // this window's lag range and length
    const int64_t n = table_n(a.tab, b, a.n);
    const double* __restrict__ s = view.s;
    const uint32_t* __restrict__ t1 = view.t1;
    const uint32_t* __restrict__ t2 = view.t2;
    uint32_t* __restrict__ qd1 = view.qd1;
    uint32_t* __restrict__ qd2 = view.qd2;
    WinState* st = a.state + b;
    gpoeo_pd_result* res = a.results + b;
    int32_t* count = a.q_count + 2 * pass;

    if (tid == 0) {
        sh.done = pass == 0 ? 0 : st->done;
        const double* v2 = a.var + 2 * b * a.num_channels;
        double acc = 0.0;
        for (int32_t c = 0; c < a.num_channels; ++c) acc = acc + (double)w.w[c] * v2[2 * c];
        sh.r_approx = 2.0 * acc;
        sh.r_err = reference_bound(v2, a.num_channels, n, w, sh.r_approx);
    }
    __syncthreads();
    if (sh.done) return true;
    if (n == 0 || tmax < tmin + 2) {   // empty or too short a slot of a window table
        if (tid == 0) {
            gpoeo_pd_result o = {};
            o.verdict = GPOEO_PD_APERIODIC;
            o.flags = GPOEO_PD_SHORT;
            *res = o;
            st->done = 1;
        }
        return true;
    }
    const double r_approx = sh.r_approx;
    const double r_err = sh.r_err;
    if (r_approx == 0.0) {   // every weighted channel constant (exact: see window_stats)
        if (tid == 0) {
            gpoeo_pd_result o = {};
            o.verdict = GPOEO_PD_CONSTANT;
            *res = o;
            st->done = 1;
        }
        return true;
    }
    const bool r_exact = pass > 0 && st->r_is_exact;
    const double r_x = r_exact ? st->r_exact : 0.0;
    const double c_lag = a.c_lag;
    // the window's lags as bits of the peak cache (bit t - tmin)
    const int64_t lag_span = (int64_t)tmax - tmin + 1;
    const bool cache = lag_span <= 32 * (int64_t)kPeakWords;
    const int words_of_window = cache ? (int)((lag_span + 31) >> 5) : 0;

    const bool deferred = !kLocal && view.gq1 != nullptr;
    // Queue (window b, lag t) for the next tier; lag -1 queues R (never
    // deferred).
    auto enqueue = [&](int tier, int32_t t) {
        if constexpr (kLocal) {   // the queued bitmaps (and r_queued) are the request
            (void)tier;
            (void)t;
            (void)count;
            return true;
        } else {
            if (deferred && t >= 0) return true;   // the request bitmap holds it
            // one atomic per wavefront and tier: the calling lanes of a tier
            // take consecutive slots from a range their first lane reserves
            const int lane = threadIdx.x & (kWave - 1);
            bool ok = true;
            for (int tr = 1; tr <= 2; ++tr) {
                const bool mine = tier == tr;
                const uint64_t m = __ballot(mine);
                if (m == 0) continue;
                const int leader = __ffsll((unsigned long long)m) - 1;
                int base = 0;
                if (lane == leader) base = atomicAdd(&count[tr - 1], __popcll(m));
                base = __shfl(base, leader);
                if (mine) {
                    const int k = base + __popcll(m & ((uint64_t(1) << lane) - 1));
                    if (k >= kQueueCap) {
                        ok = false;
                    } else {
                        a.q_win[(tr - 1) * kQueueCap + k] = (int32_t)b;
                        a.q_lag[(tr - 1) * kQueueCap + k] = t;
                    }
                }
            }
            return ok;
        }
    };
    auto want_r = [&]() {
        if (atomicExch(&st->r_queued, 1) == 0 && !enqueue(2, -1)) atomicExch(&st->r_queued, 0);
    };

    // One evaluation of the rule with tier-0 / tier-1 / reference half-widths.
    // Returns true with `o` filled when every comparison was decided;
    // otherwise queues what decides the open ones (when may_push).
    auto rule = [&](double tau0, double tau1, double e_r, bool may_push,
                    gpoeo_pd_result& o) -> bool {
        const double r_lo = r_exact ? r_x : r_approx - e_r;
        const double r_hi = r_exact ? r_x : r_approx + e_r;
        const double r_v = r_exact ? r_x : r_approx;
        // the interval of the score v of lag index j with tier words w1, w2
        auto make_iv = [&](double v, uint32_t w1, uint32_t w2, int64_t j) -> Iv {
            const uint32_t bit = 1u << (j & 31);
            Iv r;
            r.v = v;
            if (w2 & bit) {
                r.exact = true;
                r.lo = r.hi = v;
            } else {
                const double e = (w1 & bit) ? tau1 : tau0;
                r.exact = false;
                r.lo = v * (1.0 - e);
                r.hi = v * (1.0 + e);
            }
            return r;
        };
        auto iv = [&](int64_t t) -> Iv {
            const int64_t j = t - tmin;
            return make_iv(s[j], t1[j >> 5], t2[j >> 5], j);
        };
        // the same from the staged chunk (lag index cj0 at cs[0], word cw0 at ct1[0])
        int64_t cj0 = 0, cw0 = 0;
        auto iv_c = [&](int64_t t) -> Iv {
            const int64_t j = t - tmin;
            return make_iv(view.cs[j - cj0], view.ct1[(j >> 5) - cw0], view.ct2[(j >> 5) - cw0], j);
        };
        // Stage the scores of lags c0 - 1 .. c1 (at most ChunkGeom::kEntries)
        // and their tier words; every thread calls it.
        auto stage_chunk = [&](int64_t c0, int64_t c1) {
            constexpr int kPer = ChunkGeom<kSelThreads>::kEntries / kSelThreads;
            const int64_t j0 = c0 - 1 - tmin, cnt = c1 - c0 + 2;
            const int64_t w0 = j0 >> 5, wc = ((c1 - tmin) >> 5) - w0 + 1;
            __syncthreads();   // the previous chunk's readers are done
            double v[kPer];
#pragma unroll
            for (int r = 0; r < kPer; ++r) {
                const int64_t k = tid + r * kSelThreads;
                v[r] = k < cnt ? s[j0 + k] : 0.0;
            }
            uint32_t u1 = 0u, u2 = 0u;
            if (tid < wc) {
                u1 = t1[w0 + tid];
                u2 = t2[w0 + tid];
            }
#pragma unroll
            for (int r = 0; r < kPer; ++r) {
                const int64_t k = tid + r * kSelThreads;
                if (k < cnt) view.cs[k] = v[r];
            }
            if (tid < wc) {
                view.ct1[tid] = u1;
                view.ct2[tid] = u2;
            }
            cj0 = j0;
            cw0 = w0;
            __syncthreads();
        };
        const bool chunked = view.cs != nullptr;
        auto push = [&](int64_t t, const Iv& z) {
            if (z.exact || !may_push) return;
            const int64_t j = t - tmin;
            const uint32_t bit = 1u << (j & 31);
            const bool at1 = (t1[j >> 5] & bit) != 0;
            uint32_t* qd = at1 ? qd2 : qd1;
            if (atomicOr(&qd[j >> 5], bit) & bit) return;   // already queued
            if (!enqueue(at1 ? 2 : 1, (int32_t)t)) atomicAnd(&qd[j >> 5], ~bit);   // full
        };
        auto peak_of = [&](auto&& ivf, int64_t t, Iv& z, bool do_push) -> Tri {
            const Iv m = ivf(t - 1);
            z = ivf(t);
            const Iv p = ivf(t + 1);
            const Tri c1 = lt(z, m), c2 = le(z, p);
            if (c1 == kNo || c2 == kNo) return kNo;
            if (c1 == kYes && c2 == kYes) return kYes;
            if (do_push) {
                push(t - 1, m);
                push(t, z);
                push(t + 1, p);
            }
            return kUnk;
        };
        auto peak = [&](int64_t t, Iv& z, bool do_push) -> Tri { return peak_of(iv, t, z, do_push); };
        const double ulp4 = 4.0 * 2.220446049250313e-16;
        o = gpoeo_pd_result{};

        // 1. peaks.  An open local-minimum test only matters for a lag that
        // could be a candidate (S < thr) or the smallest peak; thr is at most
        // thr(R_hi, min hi over decided peaks), so open tests of lags whose
        // lower bound lies above that (and above the smallest decided peak)
        // are left open.
        int64_t npk = 0, unk = 0;
        double pk_lo = INFINITY, pk_hi = INFINITY, unk_lo = INFINITY;
        if (cache) {   // (after the scans of an earlier evaluation of the rule)
            __syncthreads();
            for (int i = tid; i < words_of_window; i += kSelThreads) sh.peaks[i] = 0u;
            __syncthreads();
        }
        auto tally_peak = [&](int64_t t, Tri q, const Iv& z) {
            if (q == kYes) {
                ++npk;
                pk_lo = fmin(pk_lo, z.lo);
                pk_hi = fmin(pk_hi, z.hi);
                if (cache) {
                    const int64_t j = t - tmin;
                    atomicOr(&sh.peaks[j >> 5], 1u << (j & 31));
                }
            } else if (q == kUnk) {
                ++unk;
                unk_lo = fmin(unk_lo, z.lo);
            }
        };
        if (chunked) {
            for (int64_t c0 = tmin + 1; c0 < tmax; c0 += ChunkGeom<kSelThreads>::kLags) {
                const int64_t c1 = min(c0 + (int64_t)ChunkGeom<kSelThreads>::kLags, (int64_t)tmax);
                stage_chunk(c0, c1);
                for (int64_t t = c0 + tid; t < c1; t += kSelThreads) {
                    Iv z;
                    tally_peak(t, peak_of(iv_c, t, z, false), z);
                }
            }
        } else {
            for (int64_t t = tmin + 1 + tid; t < tmax; t += kSelThreads) {
                Iv z;
                tally_peak(t, peak(t, z, false), z);
            }
        }
        {
            double dm[3] = {pk_lo, pk_hi, unk_lo};
            int64_t is[2] = {unk, npk};
            int64_t im = 0;
            block_reduce<kSelThreads>(dm, is, im, sh);
            pk_lo = dm[0];
            pk_hi = dm[1];
            unk_lo = dm[2];
            unk = is[0];
            npk = is[1];
        }
        if (unk > 0) {
            const double cut =
                npk > 0 ? fmax(r_hi - c_lag * (r_hi - pk_hi) + ulp4 * r_hi, pk_hi) : INFINITY;
            if (unk_lo < cut) {
                for (int64_t t = tmin + 1 + tid; t < tmax; t += kSelThreads) {
                    Iv z;
                    if (peak(t, z, false) == kUnk && z.lo < cut) peak(t, z, true);
                }
                return false;
            }
        }
        if (npk == 0) {
            o.verdict = GPOEO_PD_APERIODIC;
            return true;
        }
        // 2. threshold and candidates
        Iv thr;
        if (pk_lo == pk_hi && r_lo == r_hi) {
            thr.lo = thr.hi = r_v - c_lag * (r_v - pk_lo);
        } else {
            thr.lo = r_lo - c_lag * (r_lo - pk_lo) - ulp4 * r_hi;
            thr.hi = r_hi - c_lag * (r_hi - pk_hi) + ulp4 * r_hi;
        }
        thr.v = 0.5 * (thr.lo + thr.hi);
        thr.exact = thr.lo == thr.hi;
        int64_t ncand = 0, tc = INT64_MAX;
        unk = 0;
        auto cand = [&](auto&& ivf, int64_t t) {
            Iv z;
            if (cache) {
                const int64_t j = t - tmin;
                if (!((sh.peaks[j >> 5] >> (j & 31)) & 1u)) return;
                z = ivf(t);
            } else if (peak_of(ivf, t, z, false) != kYes) {
                return;
            }
            const Tri q = lt(z, thr);
            if (q == kYes) {
                ++ncand;
                tc = min(tc, t);
            } else if (q == kUnk) {
                ++unk;
                push(t, z);
            }
        };
        if (chunked) {
            for (int64_t c0 = tmin + 1; c0 < tmax; c0 += ChunkGeom<kSelThreads>::kLags) {
                const int64_t c1 = min(c0 + (int64_t)ChunkGeom<kSelThreads>::kLags, (int64_t)tmax);
                stage_chunk(c0, c1);
                for (int64_t t = c0 + tid; t < c1; t += kSelThreads) cand(iv_c, t);
            }
        } else {
            for (int64_t t = tmin + 1 + tid; t < tmax; t += kSelThreads) cand(iv, t);
        }
        {
            double dm[3] = {INFINITY, INFINITY, INFINITY};
            int64_t is[2] = {unk, ncand};
            block_reduce<kSelThreads>(dm, is, tc, sh);
            unk = is[0];
            ncand = is[1];
        }
        if (unk > 0) {
            // the threshold must tighten too: R and every peak that can be
            // the smallest one
            if (r_lo != r_hi && tid == 0 && may_push) want_r();
            if (pk_lo != pk_hi) {
                for (int64_t t = tmin + 1 + tid; t < tmax; t += kSelThreads) {
                    Iv z;
                    if (cache) {
                        const int64_t j = t - tmin;
                        if (!((sh.peaks[j >> 5] >> (j & 31)) & 1u)) continue;
                        z = iv(t);
                        if (z.lo <= pk_hi) push(t, z);
                    } else if (peak(t, z, false) == kYes && z.lo <= pk_hi) {
                        push(t, z);
                    }
                }
            }
            return false;
        }
        o.n_candidates = (int32_t)ncand;
        if (ncand == 0) {
            o.verdict = GPOEO_PD_APERIODIC;
            return true;
        }
        o.t_cand = (int32_t)tc;
        // 3. local search window
        const int64_t d = n - 1;
        int64_t lo = (tc * d + (d + tc) - 1) / (d + tc);
        int64_t hi = (tc * d) / (d - tc);
        lo = max(lo, (int64_t)tmin);
        hi = min(hi, (int64_t)tmax);
        o.t_low = (int32_t)lo;
        o.t_up = (int32_t)hi;
        double m_hi = INFINITY;
        for (int64_t t = lo + tid; t <= hi; t += kSelThreads) m_hi = fmin(m_hi, iv(t).hi);
        m_hi = block_min_d<kSelThreads>(m_hi, sh.red_d);
        int64_t ncont = 0, nopen = 0, tbest = INT64_MAX;
        for (int64_t t = lo + tid; t <= hi; t += kSelThreads) {
            const Iv z = iv(t);
            if (z.lo <= m_hi) {
                ++ncont;
                if (!z.exact) ++nopen;
                tbest = min(tbest, t);
            }
        }
        {
            double dm[3] = {INFINITY, INFINITY, INFINITY};
            int64_t is[2] = {ncont, nopen};
            block_reduce<kSelThreads>(dm, is, tbest, sh);
            ncont = is[0];
            nopen = is[1];
        }
        if (ncont > 1 && nopen > 0 && tau0 > 0.0) {
            for (int64_t t = lo + tid; t <= hi; t += kSelThreads) {
                const Iv z = iv(t);
                if (z.lo <= m_hi) push(t, z);
            }
            return false;
        }
        // One contender is the strict argmin; several exact contenders all
        // equal m_hi, so the smallest lag wins the tie.
        o.period = (int32_t)tbest;
        const Iv z = iv(tbest);
        // 4. err and verdict
        bool aper;
        if ((z.exact && r_lo == r_hi) || tau0 == 0.0) {
            aper = z.v / r_v >= a.err_max;
        } else {
            const double e_lo = z.lo / r_hi * (1.0 - ulp4);
            const double e_hi = z.hi / r_lo * (1.0 + ulp4);
            if (e_lo >= a.err_max) {
                aper = true;
            } else if (e_hi < a.err_max) {
                aper = false;
            } else {
                if (tid == 0 && may_push) {
                    push(tbest, z);
                    want_r();
                }
                return false;
            }
        }
        o.err = (float)(z.v / r_v);
        o.verdict = aper ? GPOEO_PD_APERIODIC : GPOEO_PD_PERIODIC;
        return true;
    };

    const bool rescue = (a.flags & GPOEO_PD_NO_RESCUE) == 0;
    gpoeo_pd_result o;
    bool done, unresolved = false;
    if (!rescue) {
        done = rule(0.0, 0.0, 0.0, false, o);
    } else {
        done = rule(a.tau0, a.tau1, r_err, !last, o);
        if (!done && last) {
            done = rule(0.0, 0.0, 0.0, false, o);
            unresolved = true;
        }
    }
    __syncthreads();
    if (deferred && !done) {
        // This pass's requests (marked in the LDS bitmaps, read after the
        // barrier above) join the window's queued bitmaps; the lags not queued
        // in an earlier pass go to the global queue, each wavefront's lanes
        // into consecutive slots that one atomic reserves.  A request that
        // does not fit is dropped and its queued bit cleared, as at once.
        const int lane = tid & (kWave - 1);
        for (int k0 = 0; k0 < a.words; k0 += kSelThreads) {
            const int k = k0 + tid;
#pragma unroll
            for (int tr = 1; tr <= 2; ++tr) {
                uint32_t* req = tr == 1 ? qd1 : qd2;
                uint32_t* gq = tr == 1 ? view.gq1 : view.gq2;
                uint32_t bits = k < a.words ? req[k] : 0u;
                if (bits) {
                    bits &= ~atomicOr(&gq[k], bits);
                    req[k] = 0u;
                }
                const int cnt = __popc(bits);
                int incl = cnt;
                for (int o = 1; o < kWave; o <<= 1) {
                    const int u = __shfl_up(incl, o);
                    if (lane >= o) incl += u;
                }
                const int total = __shfl(incl, kWave - 1);
                if (total == 0) continue;
                int base = 0;
                if (lane == kWave - 1) base = atomicAdd(&count[tr - 1], total);
                base = __shfl(base, kWave - 1);
                int slot = base + incl - cnt;
                while (bits) {
                    const int bit = __builtin_ctz(bits);
                    bits &= bits - 1;
                    if (slot < kQueueCap) {
                        a.q_win[(tr - 1) * kQueueCap + slot] = (int32_t)b;
                        a.q_lag[(tr - 1) * kQueueCap + slot] = tmin + 32 * k + bit;
                    } else {
                        atomicAnd(&gq[k], ~(1u << bit));
                    }
                    ++slot;
                }
            }
        }
    }
    if (tid == 0 && done) {
        o.n_rescored = st->rescored;
        o.flags = (unresolved ? GPOEO_PD_UNRESOLVED : 0u) | (st->tier2 ? GPOEO_PD_TIER2 : 0u);
        *res = o;
        st->done = 1;
    }
    return done;
}

// Windows of at most 32 kReqWords lags collect a selection pass's re-score
// requests in LDS bitmaps before they join the global queues.
constexpr int kReqWords = 1024;

// Windows of at most this many lags are staged in LDS by the selection passes
// (their fp64 scores and two tier bitmaps: at most about 113 KiB).
constexpr int32_t kSelLdsLags = 14000;
constexpr int64_t kSelLdsWindows = 1024;

// One pass of the rule over every window not yet decided.  With a.stage the
// window's scores and tier bitmaps are first copied to LDS with coalesced
// loads (all in flight together), so that the rule's scans read LDS.
template <int kSelThreads>
__global__ __launch_bounds__(kSelThreads) void select_pass_kernel(SelectArgs a, Weights w) {
    __shared__ Shared<kSelThreads> sh;
    __shared__ uint32_t req[2][kReqWords];
    extern __shared__ double dyn[];
    const int64_t b = blockIdx.x;
    if (a.pass > 0 && a.state[b].done) return;   // decided earlier (the same for every thread)
    WindowView view = {a.s64 + b * (int64_t)a.lags, a.tier1 + b * (int64_t)a.words,
                       a.tier2 + b * (int64_t)a.words, a.queued1 + b * (int64_t)a.words,
                       a.queued2 + b * (int64_t)a.words, nullptr, nullptr,
                       nullptr, nullptr, nullptr};
    if (a.chunk) {
        view.cs = dyn;
        view.ct1 = reinterpret_cast<uint32_t*>(dyn + ChunkGeom<kSelThreads>::kEntries);
        view.ct2 = view.ct1 + ChunkGeom<kSelThreads>::kWords;
    }
    if (a.words <= kReqWords) {   // deferred requests (cleared here; select_window's
                                  // first barrier orders this before the rule)
        for (int32_t k = threadIdx.x; k < a.words; k += kSelThreads) req[0][k] = req[1][k] = 0u;
        view.gq1 = view.qd1;
        view.gq2 = view.qd2;
        view.qd1 = req[0];
        view.qd2 = req[1];
    }
    if (a.stage) {
        double* s_l = dyn;
        uint32_t* t1_l = reinterpret_cast<uint32_t*>(dyn + a.lags);
        uint32_t* t2_l = t1_l + a.words;
        // kBatch loads of a thread in flight before their LDS stores
        constexpr int kBatch = 8;
        for (int32_t j0 = 0; j0 < a.lags; j0 += kBatch * kSelThreads) {
            double v[kBatch];
#pragma unroll
            for (int r = 0; r < kBatch; ++r) {
                const int32_t j = j0 + r * kSelThreads + (int32_t)threadIdx.x;
                v[r] = j < a.lags ? view.s[j] : 0.0;
            }
#pragma unroll
            for (int r = 0; r < kBatch; ++r) {
                const int32_t j = j0 + r * kSelThreads + (int32_t)threadIdx.x;
                if (j < a.lags) s_l[j] = v[r];
            }
        }
        for (int32_t k0 = 0; k0 < a.words; k0 += kBatch * kSelThreads) {
            uint32_t u1[kBatch], u2[kBatch];
#pragma unroll
            for (int r = 0; r < kBatch; ++r) {
                const int32_t k = k0 + r * kSelThreads + (int32_t)threadIdx.x;
                u1[r] = k < a.words ? view.t1[k] : 0u;
                u2[r] = k < a.words ? view.t2[k] : 0u;
            }
#pragma unroll
            for (int r = 0; r < kBatch; ++r) {
                const int32_t k = k0 + r * kSelThreads + (int32_t)threadIdx.x;
                if (k < a.words) {
                    t1_l[k] = u1[r];
                    t2_l[k] = u2[r];
                }
            }
        }
        __syncthreads();
        view.s = s_l;
        view.t1 = t1_l;
        view.t2 = t2_l;
    }
    select_window<kSelThreads, false>(a, w, b, a.pass, a.last != 0, sh, view);
}

// One re-score round: every workgroup takes queued tier-1 requests (one lag
// per workgroup at a time), then every lane takes queued tier-2 requests (one
// lag, or one window's R, per lane).
__global__ __launch_bounds__(kThreads) void rescore_kernel(SelectArgs a, Weights w) {
    __shared__ double red[kThreads / kWave];
    const int32_t* count = a.q_count + 2 * a.pass;
    const int n1 = min(count[0], kQueueCap), n2 = min(count[1], kQueueCap);
    if (n1 == 0 && n2 == 0) return;
    for (int64_t e = blockIdx.x; e < n1; e += gridDim.x) {
        const int64_t b = a.q_win[e];
        const int64_t t = a.q_lag[e];
        const int64_t j = t - a.tmin;
        uint32_t* t1 = a.tier1 + b * (int64_t)a.words;
        const uint32_t done = (t1[j >> 5] >> (j & 31)) & 1u;
        __syncthreads();                    // every thread has read the bit
        if (done) continue;
        const float* __restrict__ xw = a.x + table_off(a.tab, b, a.window_stride);
        const double v = group_score<kThreads>(xw, a.num_channels, a.channel_stride,
                                               table_n(a.tab, b, a.n), t, w, red);
        if (threadIdx.x == 0) {
            a.s64[b * (int64_t)a.lags + j] = v;
            __threadfence();
            const uint32_t old = atomicOr(&t1[j >> 5], 1u << (j & 31));
            if (!((old >> (j & 31)) & 1u)) atomicAdd(&a.state[b].rescored, 1);
        }
    }
    const int64_t lanes = (int64_t)gridDim.x * kThreads;
    for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < n2; e += lanes) {
        const int64_t b = a.q_win[kQueueCap + e];
        const int64_t t = a.q_lag[kQueueCap + e];
        const float* __restrict__ xw = a.x + table_off(a.tab, b, a.window_stride);
        const int64_t n = table_n(a.tab, b, a.n);
        if (t < 0) {
            WinState* st = a.state + b;
            st->r_exact = exact_reference(xw, a.num_channels, a.channel_stride, n, w);
            st->tier2 = 1;
            __threadfence();
            st->r_is_exact = 1;
            continue;
        }
        const int64_t j = t - a.tmin;
        uint32_t* t2 = a.tier2 + b * (int64_t)a.words;
        if ((t2[j >> 5] >> (j & 31)) & 1u) continue;
        a.s64[b * (int64_t)a.lags + j] = exact_score(xw, a.num_channels, a.channel_stride, n, t, w);
        a.state[b].tier2 = 1;
        __threadfence();
        atomicOr(&t2[j >> 5], 1u << (j & 31));
    }
}

// Clears the tier and queue bitmaps and the state of every window (a fill
// kernel rather than a memset, so that the sequence stays capturable).
__global__ __launch_bounds__(kThreads) void select_init_kernel(SelectBuffers sb, int64_t words,
                                                               int64_t num_windows) {
    const int64_t total = words * num_windows;
    const int64_t step = (int64_t)gridDim.x * kThreads;
    for (int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x; k < total; k += step) {
        sb.tier1[k] = 0u;
        sb.tier2[k] = 0u;
        sb.queued1[k] = 0u;
        sb.queued2[k] = 0u;
    }
    for (int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x; b < num_windows; b += step) {
        WinState z;
        z.r_exact = 0.0;
        z.done = 0;
        z.r_queued = 0;
        z.r_is_exact = 0;
        z.rescored = 0;
        z.tier2 = 0;
        sb.state[b] = z;
    }
    if (blockIdx.x == 0 && (int)threadIdx.x < 2 * kPasses) sb.q_count[threadIdx.x] = 0;
}

// Re-scores the lags window b's rule marked in its queued bitmaps (and R), on
// the LDS copies of the fused kernel: tier 1 by the whole workgroup (one lag at
// a time), tier 2 and R by single lanes, with the same evaluations as
// rescore_kernel.
template <int kT>
__device__ void rescore_window(const SelectArgs& a, const Weights& w, int64_t b, double* s,
                               uint32_t* t1, uint32_t* t2, const uint32_t* qd1,
                               const uint32_t* qd2, double* red) {
    const int tid = threadIdx.x;
    WinState* st = a.state + b;
    const float* __restrict__ xw = a.x + b * a.window_stride;
    for (int k = 0; k < a.words; ++k) {
        // read by every thread before group_score's barriers let thread 0 set a bit of k
        uint32_t m = qd1[k] & ~t1[k];
        while (m) {
            const int bit = __builtin_ctz(m);
            m &= m - 1;
            const int64_t j = 32 * (int64_t)k + bit;
            const double v = group_score<kT>(xw, a.num_channels, a.channel_stride, a.n,
                                             a.tmin + j, w, red);
            if (tid == 0) {
                s[j] = v;
                atomicOr(&t1[k], 1u << bit);
                atomicAdd(&st->rescored, 1);
            }
        }
        __syncthreads();
    }
    for (int k = tid; k < a.words; k += kT) {
        uint32_t m = qd2[k] & ~t2[k];
        while (m) {
            const int bit = __builtin_ctz(m);
            m &= m - 1;
            const int64_t j = 32 * (int64_t)k + bit;
            s[j] = exact_score(xw, a.num_channels, a.channel_stride, a.n, a.tmin + j, w);
            st->tier2 = 1;
            atomicOr(&t2[k], 1u << bit);
        }
    }
    if (tid == 0 && st->r_queued && !st->r_is_exact) {
        st->r_exact = exact_reference(xw, a.num_channels, a.channel_stride, a.n, w);
        st->tier2 = 1;
        st->r_is_exact = 1;
    }
}

struct FinishArgs {
    const double* part;      // lag-score chunk partials
    double* var;             // [B][C][2], written here
    float* scores;           // nullable
    int32_t t0, lags_padded, chunks;
};

// Everything after the lag scores of a window, in one workgroup: the window
// statistics (stats::channel_stats, as window_stats_kernel), the finalisation
// (stats::finalize_lags, as finalize_kernel), the selection state, and up to
// kPasses evaluations of the rule with this workgroup re-scoring the lags
// each one marks.  The window's fp64 scores and its four bitmaps live in LDS
// (dynamic shared memory: lags doubles, then 4 x words words) for the
// selection.  Same values, decisions and results as the separate kernels;
// one launch instead of nine, for windows short enough that one workgroup
// re-scores a lag quickly.
__global__ __launch_bounds__(stats::kStatsThreads) void finish_kernel(SelectArgs a, FinishArgs f,
                                                                     Weights w) {
    constexpr int kT = stats::kStatsThreads;
    __shared__ Shared<kT> sh;
    __shared__ double red[kT];
    extern __shared__ double dyn[];
    double* s_l = dyn;
    uint32_t* bits = reinterpret_cast<uint32_t*>(dyn + a.lags);
    uint32_t* t1 = bits;
    uint32_t* t2 = bits + a.words;
    uint32_t* qd1 = bits + 2 * a.words;
    uint32_t* qd2 = bits + 3 * a.words;
    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const float* __restrict__ xw = a.x + b * a.window_stride;
    const bool scores_only = (a.flags & GPOEO_PD_SCORES_ONLY) != 0;
    if (!scores_only)
        for (int32_t c = 0; c < a.num_channels; ++c) {
            const stats::ChannelStats cs =
                stats::channel_stats(xw + (int64_t)c * a.channel_stride, a.n, red, false);
            if (tid == 0) {
                const int64_t bc = b * a.num_channels + c;
                f.var[2 * bc] = cs.var;
                f.var[2 * bc + 1] = cs.absmean;
            }
        }
    constexpr int L = stats::kFinalizeLags;
    for (int32_t j = tid; j < a.lags; j += kT * L) {
        double v[L];
        stats::finalize_lags(f.part, w, a.num_channels, b, a.n, (int64_t)a.tmin + j, kT,
                             (int64_t)a.tmin + a.lags, f.t0, f.lags_padded, f.chunks, v);
#pragma unroll
        for (int l = 0; l < L; ++l) {
            const int64_t jj = j + (int64_t)l * kT;
            if (jj >= a.lags) break;
            s_l[jj] = v[l];
            if (f.scores) f.scores[b * (int64_t)a.lags + jj] = (float)v[l];
        }
    }
    if (scores_only) return;
    for (int k = tid; k < 4 * a.words; k += kT) bits[k] = 0u;
    if (tid == 0) {
        WinState z;
        z.r_exact = 0.0;
        z.done = 0;
        z.r_queued = 0;
        z.r_is_exact = 0;
        z.rescored = 0;
        z.tier2 = 0;
        a.state[b] = z;
    }
    __syncthreads();
    const int passes = (a.flags & GPOEO_PD_NO_RESCUE) ? 1 : kPasses;
    const WindowView view = {s_l, t1, t2, qd1, qd2};
    for (int pass = 0; pass < passes; ++pass) {
        if (select_window<kT, true>(a, w, b, pass, pass == passes - 1, sh, view)) break;
        __syncthreads();
        rescore_window<kT>(a, w, b, s_l, t1, t2, qd1, qd2, red);
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_finish(const Plan& p, const Weights& w, const float* x, double* var,
                         const double* part, double* s64, float* scores,
                         const SelectBuffers& sb, void* results, hipStream_t s) {
    SelectArgs a = {};
    a.x = x;
    a.var = var;
    a.s64 = s64;
    a.tier1 = sb.tier1;
    a.tier2 = sb.tier2;
    a.queued1 = sb.queued1;
    a.queued2 = sb.queued2;
    a.state = sb.state;
    a.q_win = sb.q_win;
    a.q_lag = sb.q_lag;
    a.q_count = sb.q_count;
    a.results = static_cast<gpoeo_pd_result*>(results);
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    a.tmin = p.tmin;
    a.tmax = p.tmax;
    a.lags = p.lags;
    a.words = p.bitmap_words;
    a.c_lag = p.c_lag;
    a.err_max = p.err_max;
    a.flags = p.flags;
    a.tab = p.table;
    a.tau0 = kScoreRelBound;
    const double u = 1.1102230246251565e-16;
    a.tau1 = 1.01 * u * ((double)p.n * (1.0 + 1.0 / 256.0) + 2.0 * p.num_channels + 22.0);
    FinishArgs f;
    f.part = part;
    f.var = var;
    f.scores = scores;
    f.t0 = p.t0;
    f.lags_padded = p.lags_padded;
    f.chunks = p.chunks;
    const size_t lds = (size_t)p.lags * sizeof(double) + 4 * (size_t)p.bitmap_words * 4;
    hipLaunchKernelGGL(finish_kernel, dim3((unsigned)p.num_windows), dim3(stats::kStatsThreads),
                       lds, s, a, f, w);
    return hipGetLastError();
}

hipError_t launch_select_init(const Plan& p, const SelectBuffers& sb, hipStream_t s) {
    const int64_t total = std::max<int64_t>((int64_t)p.bitmap_words * p.num_windows, p.num_windows);
    int64_t groups = (total + kThreads - 1) / kThreads;
    if (groups > 4096) groups = 4096;
    hipLaunchKernelGGL(select_init_kernel, dim3((unsigned)groups), dim3(kThreads), 0, s, sb,
                       (int64_t)p.bitmap_words, p.num_windows);
    return hipGetLastError();
}

hipError_t launch_select(const Plan& p, const Weights& w, const float* x, const double* var,
                         double* s64, const SelectBuffers& sb, void* results, hipStream_t s) {
    SelectArgs a;
    a.x = x;
    a.var = var;
    a.s64 = s64;
    a.tier1 = sb.tier1;
    a.tier2 = sb.tier2;
    a.queued1 = sb.queued1;
    a.queued2 = sb.queued2;
    a.state = sb.state;
    a.q_win = sb.q_win;
    a.q_lag = sb.q_lag;
    a.q_count = sb.q_count;
    a.results = static_cast<gpoeo_pd_result*>(results);
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    a.tmin = p.tmin;
    a.tmax = p.tmax;
    a.lags = p.lags;
    a.words = p.bitmap_words;
    a.c_lag = p.c_lag;
    a.err_max = p.err_max;
    a.flags = p.flags;
    a.tab = p.table;
    a.tau0 = p.fft ? kFftRelBound : kScoreRelBound;
    // Tier-1 half-width: the sequential sum (at most n + C + 6 roundings of
    // u = 2^-53 each, relative to the exact value) plus the wavefront sum
    // (n/256 + C + 16 roundings), with 1% margin.
    const double u = 1.1102230246251565e-16;
    a.tau1 = 1.01 * u * ((double)p.n * (1.0 + 1.0 / 256.0) + 2.0 * p.num_channels + 22.0);
    const bool rescue = (p.flags & GPOEO_PD_NO_RESCUE) == 0;
    const int passes = rescue ? kPasses : 1;
    const dim3 grid_sel((unsigned)p.num_windows);
    const dim3 grid_re(kRescoreGroups);
    // (for a few windows each pass is a chain of scans that LDS shortens; for
    // many windows the copies would cost more occupancy than they save)
    a.stage = p.lags <= kSelLdsLags && p.num_windows <= kSelLdsWindows;
    // (windows too long for that, or too many of them, stream their two full
    // scans through LDS: a chunk's loads all in flight together, instead of a
    // dependent load per lag and thread)
    a.chunk = !a.stage;
    // Chunked scans are paced by their barriers and interval tests: a batch
    // with more windows than the GPU has CUs runs them in 256-thread
    // workgroups, several windows a CU (1024 windows of 32,767 lags: 290 ->
    // 215 us a pass), a smaller batch keeps the 1024 threads a window.
    const bool wide = p.lags >= kWideLags && !p.table.n &&
                      !(a.chunk && p.num_windows > kChunkWideWindows);
    const size_t lds =
        a.stage ? (size_t)p.lags * sizeof(double) + 2 * (size_t)p.bitmap_words * 4
        : a.chunk ? (wide ? ChunkGeom<1024>::kBytes : ChunkGeom<kThreads>::kBytes)
                  : 0;
    for (int pass = 0; pass < passes; ++pass) {
        a.pass = pass;
        a.last = pass == passes - 1;
        if (wide)
            hipLaunchKernelGGL(select_pass_kernel<1024>, grid_sel, dim3(1024), lds, s, a, w);
        else
            hipLaunchKernelGGL(select_pass_kernel<kThreads>, grid_sel, dim3(kThreads), lds, s, a,
                               w);
        if (!a.last) hipLaunchKernelGGL(rescore_kernel, grid_re, dim3(kThreads), 0, s, a, w);
    }
    return hipGetLastError();
}

}  // namespace gpoeo
