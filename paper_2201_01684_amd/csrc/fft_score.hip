// Scores of every lag from an fp64 FFT autocorrelation.
//
// The spectrum of the trace is the starting point of period detection in
// Sec. 4.1.1 (Algorithm 1 transforms the samples and looks for amplitude
// peaks).  Here the transform serves the lag domain instead: for one window's
// channel y (centred by its fp64 mean, zero-padded to L = 2^lg >= N + Tmax
// points so that no lag up to Tmax wraps around),
//   D(T) = sum_{i<N-T} (y_i - y_{i+T})^2 = E1(T) + E2(T) - 2 r(T),
//   E1(T) = sum_{i<N-T} y_i^2,  E2(T) = sum_{i>=T} y_i^2,  r(T) = sum_i y_i y_{i+T},
// with r the inverse transform of |FFT(y)|^2.  Two real sequences a, b travel
// as one complex one, z = y_a + i y_b: from Z = FFT(z) the spectra of a and b
// are (Z(k) + conj Z(L-k)) / 2 and (Z(k) - conj Z(L-k)) / 2i, and the inverse
// transform of |X_a|^2 + i |X_b|^2 returns r_a + i r_b.
//
// Transforms: radix-2 butterflies in LDS, decimation in frequency forward
// (natural order in, bit-reversed out) and in time inverse (bit-reversed in,
// natural out), so no permutation pass is needed.  Up to 2^12 points one
// workgroup holds a whole pair.  Longer transforms use L = L1 * L2 (index
// n = n1 L2 + n2, frequency k = k1 + L1 k2): L2 column transforms of L1
// points, the twiddles W_L^(k1 n2), then L1 row transforms of L2 points.  The
// row kernel holds row k1 together with its mirror row L1 - k1, so the
// separation of the two sequences, the power spectrum, the inverse row
// transform and the inverse twiddles all happen while the two rows are in LDS;
// the inverse column kernel then forms D(T) for the lags it produces.
//
// Accuracy: every lag's D(T) is within an absolute bound derived from the
// sequence norms (fft_bound below); the lags for which that bound is not a
// small fraction of the score are re-scored in fp64 before any decision.
#include <algorithm>
#include <cmath>

#include "internal.h"
#include "exact.h"

namespace gpoeo {
namespace {

constexpr int kThreads = 256;                          // edge and fix-up kernels
constexpr int kTThreads = 1 << kFftThreadsLog2;        // transform kernels


struct FftArgs {
    const float* x;
    const double* fstat;       // [S][4]: mean, sum y^2, sum |y|, unused (window statistics)
    double* edge;              // [S][2][tmax + 1]: head and tail sums of y^2
    const double2* tw;         // twiddle tables
    double2* z;                // [pairs][len]
    double* part;              // [S][lags]: D(T)
    double* amp;               // spectra: [S][len/2 + 1] amplitudes |X_s(k)|
    int64_t seqs;              // S = B * C
    int64_t n_all, window_stride, channel_stride;
    int64_t len;
    int64_t tw_a, tw_b, tw_lo, tw_hi;
    int32_t num_channels;
    int32_t tmin, tmax, lags;
    int32_t lg, lg1, lg2, lgc, lgr;
    WindowTable tab;
    // Ragged launches (windows of different lengths) transform the pairs of
    // one length class, list[bounds[cls] .. bounds[cls + 1]) (class = log2 of
    // the transform length).  Transform z of pair p sits at z + p * zstride.
    const int32_t* list;
    const int32_t* bounds;
    int64_t zstride;
    int32_t cls;
    // Loads of a transform see samples [seg_start, seg_start + seg_len) of
    // each sequence (seg_len 0: all of it): the heads and tails of the wrap
    // correction.
    int64_t seg_start, seg_len;
    // Wrap correction: the inverse column kernel of the head-tail transform
    // writes the cross-correlations cc(s), s < wm, to wout ([S][wm]); the one
    // of the main transform subtracts wrap[s][Tmax - T] from r(T) for T > wrap_w.
    double* wout;
    const double* wrap;
    int64_t wrap_w;
    int32_t wm;
    // Fused finalisation (one channel, uniform batch): S(T) to s64 and scores.
    double* s64;
    float* scores;
    float w0;
};

// Transform kernels come in two forms: uniform (kRagged false: one workgroup
// per item, grid = items, the loop below runs once) and ragged (a capped grid
// whose workgroups loop over the items of one length class).
template <bool kRagged>
__device__ __forceinline__ int64_t work_items(const FftArgs& a, int64_t per_pair) {
    return kRagged ? (int64_t)(a.bounds[a.cls + 1] - a.bounds[a.cls]) * per_pair
                   : (int64_t)gridDim.x;
}
template <bool kRagged>
__device__ __forceinline__ int64_t pair_at(const FftArgs& a, int64_t k) {
    return kRagged ? (int64_t)a.list[a.bounds[a.cls] + k] : k;
}

__device__ __forceinline__ double2 cadd(double2 a, double2 b) {
    return make_double2(a.x + b.x, a.y + b.y);
}
__device__ __forceinline__ double2 csub(double2 a, double2 b) {
    return make_double2(a.x - b.x, a.y - b.y);
}
__device__ __forceinline__ double2 cmul(double2 a, double2 b) {
    return make_double2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ double2 cmul_conj(double2 a, double2 b) {   // a * conj(b)
    return make_double2(a.x * b.x + a.y * b.y, a.y * b.x - a.x * b.y);
}
__device__ __forceinline__ uint32_t bitrev(uint32_t v, int lg) {
    return lg == 0 ? 0u : (__builtin_bitreverse32(v) >> (32 - lg));
}

// Consecutive workgroups of a launch go round-robin to the 8 XCDs; this maps
// them so that each XCD takes a contiguous range of logical ids (neighbouring
// column groups of one pair then share that XCD's L2).
__device__ __forceinline__ int64_t xcd_remap(int64_t bid, int64_t nblk) {
    if (nblk % 8 != 0) return bid;
    return (bid & 7) * (nblk >> 3) + (bid >> 3);
}

// Transforms of `cols` interleaved sequences of L = 2^lg points, s[i * cols + q],
// as radix-2 butterflies: forward by decimation in frequency (natural order
// in, bit-reversed out), at stage h = 2^st the pair (i, i + h) becomes
// (a + b, (a - b) W_2h^j), j = i mod h; inverse by decimation in time
// (bit-reversed in, natural out), (a + b conj(W_2h^j), a - b conj(W_2h^j)).
// tw[m] = exp(-2 pi i m / L), m < L/2, so W_2h^j = tw[j L / 2h].
//
// A pass runs 2^R-point groups through R consecutive stages in registers (the
// same butterflies, so the same roundings as stage-by-stage): the points of a
// group share every index bit outside the pass's stages.  Passes hold up to 4
// stages, with at least 256 groups when the LDS tile allows (all threads busy).
template <int R, bool kInverse>
__device__ __forceinline__ void fft_pass(double2* s, int lg, int lgc, int st_lo,
                                         const double2* __restrict__ tw) {
    constexpr int kR = 1 << R;
    const int cols = 1 << lgc;
    const int groups = 1 << (lg - R + lgc);
    const int lo_mask = (1 << st_lo) - 1;
    for (int gi = threadIdx.x; gi < groups; gi += kTThreads) {
        const int q = gi & (cols - 1);
        const int g = gi >> lgc;
        const int blo = g & lo_mask;
        const int base = ((g >> st_lo) << (st_lo + R)) | blo;
        // the twiddles of all R stages first: stage k uses 2^k of them,
        // W_2h^(blo + u 2^st_lo) for u < 2^k, at wt[2^k - 1 + u]
        double2 wt[kR - 1];
#pragma unroll
        for (int k = 0; k < R; ++k)
#pragma unroll
            for (int u = 0; u < (1 << k); ++u)
                wt[(1 << k) - 1 + u] = tw[(blo + (u << st_lo)) << (lg - 1 - (st_lo + k))];
        double2 v[kR];
#pragma unroll
        for (int m = 0; m < kR; ++m) v[m] = s[(base + (m << st_lo)) * cols + q];
#pragma unroll
        for (int kk = 0; kk < R; ++kk) {
            const int k = kInverse ? kk : R - 1 - kk;   // stage st_lo + k
#pragma unroll
            for (int m = 0; m < kR; ++m) {
                if (m & (1 << k)) continue;
                const double2 w = wt[(1 << k) - 1 + (m & ((1 << k) - 1))];
                const double2 a = v[m];
                if (kInverse) {
                    const double2 b = cmul_conj(v[m + (1 << k)], w);
                    v[m] = cadd(a, b);
                    v[m + (1 << k)] = csub(a, b);
                } else {
                    const double2 b = v[m + (1 << k)];
                    v[m] = cadd(a, b);
                    v[m + (1 << k)] = cmul(csub(a, b), w);
                }
            }
        }
#pragma unroll
        for (int m = 0; m < kR; ++m) s[(base + (m << st_lo)) * cols + q] = v[m];
    }
}

template <bool kInverse, int kMaxR>
__device__ void lds_fft(double2* s, int lg, int lgc, const double2* __restrict__ tw) {
    int rmax = lg + lgc - kFftThreadsLog2;   // log2 of the points per thread
    rmax = rmax < 1 ? 1 : (rmax > kMaxR ? kMaxR : rmax);
    const int np = (lg + rmax - 1) / rmax;
    const int base = lg / np, extra = lg % np;
    int st = kInverse ? 0 : lg;
    for (int p = 0; p < np; ++p) {
        const int r = base + (p < extra ? 1 : 0);
        const int st_lo = kInverse ? st : st - r;
        if (r == 1) fft_pass<1, kInverse>(s, lg, lgc, st_lo, tw);
        else if (r == 2 || kMaxR < 3) fft_pass<(kMaxR < 2 ? 1 : 2), kInverse>(s, lg, lgc, st_lo, tw);
        else if (r == 3 || kMaxR < 4) fft_pass<(kMaxR < 3 ? 1 : 3), kInverse>(s, lg, lgc, st_lo, tw);
        else fft_pass<(kMaxR < 4 ? 1 : 4), kInverse>(s, lg, lgc, st_lo, tw);
        __syncthreads();
        st = kInverse ? st + r : st_lo;
    }
}

// A workgroup of 2^kFftThreadsLog2 threads on a tile of 2^kTile points holds
// 2^(kTile - kFftThreadsLog2) points per thread: the largest useful pass radix.
template <int kTile>
__device__ __forceinline__ void lds_fft_fwd(double2* s, int lg, int lgc, const double2* tw) {
    lds_fft<false, kTile - kFftThreadsLog2>(s, lg, lgc, tw);
}
template <int kTile>
__device__ __forceinline__ void lds_fft_inv(double2* s, int lg, int lgc, const double2* tw) {
    lds_fft<true, kTile - kFftThreadsLog2>(s, lg, lgc, tw);
}

// W_L^e = exp(-2 pi i e / L) for e < L from two tables split at bit lg2.
__device__ __forceinline__ double2 twiddle(const FftArgs& a, int64_t e) {
    return cmul(a.tw[a.tw_hi + (e >> a.lg2)], a.tw[a.tw_lo + (e & ((int64_t(1) << a.lg2) - 1))]);
}

// The pass twiddles of one 2^lg-point sub-transform (tw[m], m < 2^(lg-1)),
// copied to LDS at twl by the workgroup: load() issues the loads into
// registers (with the caller's data loads, all in flight together), store()
// writes them; the caller's barrier before the transform orders them.
template <int kTile>
struct TwiddleCopy {
    static constexpr int kPer = ((1 << (kTile - 1)) + kTThreads - 1) / kTThreads;
    double2 v[kPer];
    __device__ __forceinline__ void load(const double2* __restrict__ tw, int lg) {
        const int count = 1 << (lg - 1);
#pragma unroll
        for (int r = 0; r < kPer; ++r) {
            const int k = threadIdx.x + r * kTThreads;
            v[r] = k < count ? tw[k] : make_double2(0.0, 0.0);
        }
    }
    __device__ __forceinline__ void store(double2* twl, int lg) const {
        const int count = 1 << (lg - 1);
#pragma unroll
        for (int r = 0; r < kPer; ++r) {
            const int k = threadIdx.x + r * kTThreads;
            if (k < count) twl[k] = v[r];
        }
    }
};

// The four-step twiddle tables (tw_lo, 2^lg2 entries, then tw_hi, 2^lg1) in
// LDS at tl when together they hold at most kFourStepLds entries: copied like
// the pass twiddles, then read by twiddle_at with the same operations as
// twiddle().  (The forward column and row kernels; the wrap correction's row
// kernel keeps the global tables, whose LDS would cost it a workgroup per CU.)
constexpr int kFourStepLds = 1024;
__host__ __device__ inline bool four_step_in_lds(int lg1, int lg2) {
    return (1 << lg1) + (1 << lg2) <= kFourStepLds;
}
struct FourStepCopy {
    static constexpr int kPer = kFourStepLds / kTThreads;
    double2 v[kPer];
    __device__ __forceinline__ void load(const FftArgs& a) {
        const int count = (1 << a.lg1) + (1 << a.lg2);
#pragma unroll
        for (int r = 0; r < kPer; ++r) {
            const int k = threadIdx.x + r * kTThreads;
            v[r] = k < count ? a.tw[a.tw_lo + k] : make_double2(0.0, 0.0);
        }
    }
    __device__ __forceinline__ void store(const FftArgs& a, double2* tl) const {
        const int count = (1 << a.lg1) + (1 << a.lg2);
#pragma unroll
        for (int r = 0; r < kPer; ++r) {
            const int k = threadIdx.x + r * kTThreads;
            if (k < count) tl[k] = v[r];
        }
    }
};
__device__ __forceinline__ double2 twiddle_at(const FftArgs& a, const double2* tl, bool lds4,
                                              int64_t e) {
    if (!lds4) return twiddle(a, e);
    return cmul(tl[(1 << a.lg2) + (e >> a.lg2)], tl[e & ((int64_t(1) << a.lg2) - 1)]);
}

// 4 (|X_a|^2 + i |X_b|^2) at frequency k from Z(k) and Z(L - k).
__device__ __forceinline__ double2 power_pair(double2 zk, double2 zm) {
    const double ux = zk.x + zm.x, uy = zk.y - zm.y;
    const double vx = zk.x - zm.x, vy = zk.y + zm.y;
    return make_double2(ux * ux + uy * uy, vx * vx + vy * vy);
}

struct Seq {
    const float* p;
    int64_t n;
    double mu;
};

__device__ __forceinline__ Seq seq_of(const FftArgs& a, int64_t s) {
    Seq q;
    if (s >= a.seqs) {
        q.p = nullptr;
        q.n = 0;
        q.mu = 0.0;
        return q;
    }
    const int64_t b = s / a.num_channels;
    const int64_t c = s % a.num_channels;
    q.n = table_n(a.tab, b, a.n_all);
    q.p = a.x + table_off(a.tab, b, a.window_stride) + c * a.channel_stride;
    q.mu = a.fstat[4 * s];
    if (a.seg_len > 0) {
        q.p += a.seg_start;
        q.n = min(q.n - a.seg_start, a.seg_len);
    }
    return q;
}

__device__ __forceinline__ double centred(const Seq& q, int64_t i) {
    return i < q.n ? (double)q.p[i] - q.mu : 0.0;
}

// D(T) of sequence s from the scaled inverse transform value w = 4 L r(T).
__device__ __forceinline__ void write_d(const FftArgs& a, int64_t s, int64_t t, double w) {
    if (s >= a.seqs || t < a.tmin || t > a.tmax) return;
    const int64_t b = s / a.num_channels;
    const int64_t n = table_n(a.tab, b, a.n_all);
    const bool live = n > 0 && t <= table_tmax(a.tab, b, a.tmax);
    double d = 0.0;
    if (live) {
        double r = ldexp(w, -(a.lg + 2));
        if (a.wrap && t > a.wrap_w) r -= a.wrap[s * a.wm + (a.tmax - t)];   // circular term
        const double e = a.fstat[4 * s + 1];
        const double* ed = a.edge + s * 2 * (int64_t)(a.tmax + 1);
        d = ((e - ed[a.tmax + 1 + t]) + (e - ed[t])) - 2.0 * r;
    }
    const int64_t k = s * a.lags + (t - a.tmin);
    if (a.s64) {   // the finalisation of a single channel, in its own arithmetic
        if (!live && !a.scores) return;   // past a table window's lags: left unwritten
        const double v = 0.0 + (double)a.w0 * (d / (double)(n - t));
        a.s64[k] = v;
        if (a.scores) a.scores[k] = (float)v;
    } else {
        a.part[k] = d;
    }
}

// Sums of y^2 over the first T samples (head) and the last T samples (tail)
// of a sequence, T = 0..Tmax of its window; one workgroup per (sequence,
// side).  Tiles of 4096 terms are loaded (all of a thread's loads in flight at
// once) and staged in LDS; each thread adds 16 consecutive terms, an
// exclusive scan of the thread totals (lane shuffles within each wavefront,
// then the wavefront totals in order) gives each thread its offset, and the
// running sums go back through LDS for coalesced stores.  (The mean, sum y^2
// and sum |y| come from the window statistics, computed with the same mean.)
constexpr int kEdgeTile = 4096;
constexpr int kEdgePer = kEdgeTile / kThreads;   // 16 terms per thread
constexpr int kEdgeWaves = kThreads / kWave;

__device__ __forceinline__ int edge_slot(int k) { return k + (k >> 4); }   // padded: no bank clash

__global__ __launch_bounds__(kThreads) void fft_edge_kernel(FftArgs a) {
    __shared__ double tile[kEdgeTile + kEdgeTile / 16];
    __shared__ double wsum[kEdgeWaves];
    const int64_t s = blockIdx.x >> 1;
    const int side = blockIdx.x & 1;
    const int64_t b = s / a.num_channels;
    const int64_t c = s % a.num_channels;
    const int64_t n = table_n(a.tab, b, a.n_all);
    const float* __restrict__ p = a.x + table_off(a.tab, b, a.window_stride) + c * a.channel_stride;
    const double mu = a.fstat[4 * s];
    double* __restrict__ out = a.edge + (s * 2 + side) * ((int64_t)a.tmax + 1);   // out[T]
    // T = 0 .. this window's largest lag (nothing for an empty slot)
    const int64_t span = n > 0 ? (int64_t)min(table_tmax(a.tab, b, a.tmax), a.tmax) + 1 : 1;
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    if (threadIdx.x == 0) out[0] = 0.0;
    double carry = 0.0;
    // the next tile's samples are loaded while this tile is scanned
    float nxt[kEdgePer];
    auto load_tile = [&](int64_t k0, float (&v)[kEdgePer]) {
#pragma unroll
        for (int r = 0; r < kEdgePer; ++r) {
            const int64_t kk = k0 + (int)threadIdx.x + r * kThreads;
            const bool in = kk < n && kk < span - 1;
            v[r] = in ? p[side == 0 ? kk : n - 1 - kk] : 0.0f;
        }
    };
    if (span - 1 > 0) load_tile(0, nxt);
    for (int64_t k0 = 0; k0 < span - 1; k0 += kEdgeTile) {   // terms k0 .. k0 + 4095
        {
            float v[kEdgePer];
#pragma unroll
            for (int r = 0; r < kEdgePer; ++r) v[r] = nxt[r];
            if (k0 + kEdgeTile < span - 1) load_tile(k0 + kEdgeTile, nxt);
#pragma unroll
            for (int r = 0; r < kEdgePer; ++r) {
                const int k = (int)threadIdx.x + r * kThreads;
                const int64_t kk = k0 + k;
                const double y = (kk < n && kk < span - 1) ? (double)v[r] - mu : 0.0;
                tile[edge_slot(k)] = y * y;
            }
        }
        __syncthreads();
        double part = 0.0;
        for (int r = 0; r < kEdgePer; ++r) part += tile[edge_slot((int)threadIdx.x * kEdgePer + r)];
        double inc = part;   // inclusive scan within the wavefront
        for (int o = 1; o < kWave; o <<= 1) {
            const double u = __shfl_up(inc, o);
            if (lane >= o) inc += u;
        }
        if (lane == kWave - 1) wsum[wave] = inc;
        __syncthreads();
        double run = carry, total = carry;
        for (int w = 0; w < kEdgeWaves; ++w) {
            if (w < wave) run += wsum[w];
            total += wsum[w];
        }
        run += inc - part;   // this thread's exclusive offset
        for (int r = 0; r < kEdgePer; ++r) {
            const int k = (int)threadIdx.x * kEdgePer + r;
            run += tile[edge_slot(k)];
            tile[edge_slot(k)] = run;   // sum of terms 0 .. k0 + k: the value at T = k0 + k + 1
        }
        __syncthreads();
        for (int r = 0; r < kEdgePer; ++r) {
            const int k = (int)threadIdx.x + r * kThreads;
            const int64_t t = k0 + k + 1;
            if (t < span) out[t] = tile[edge_slot(k)];
        }
        carry = total;
        __syncthreads();
    }
}

// Twiddle tables: A (transforms of 2^lga points), B (2^lgb points, if any),
// and the two halves of W_L^e for the split transform.
__global__ void fft_twiddle_kernel(double2* tw, int lga, int lgb, int lg, int lg2, int64_t nb,
                                   int64_t nlo, int64_t nhi) {
    const int64_t na = int64_t(1) << (lga - 1);
    const int64_t total = na + nb + nlo + nhi;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        int64_t m;
        int lgl;
        if (e < na) {
            m = e;
            lgl = lga;
        } else if (e < na + nb) {
            m = e - na;
            lgl = lgb;
        } else if (e < na + nb + nlo) {
            m = e - na - nb;
            lgl = lg;
        } else {
            m = e - na - nb - nlo;
            lgl = lg - lg2;
        }
        double sn, cs;
        sincospi(ldexp(2.0 * (double)m, -lgl), &sn, &cs);   // exact argument 2m / 2^lgl
        tw[e] = make_double2(cs, -sn);
    }
}

// Whole transform of one pair in one workgroup (L <= 2^12).
template <int kTile, bool kRagged>
__global__ __launch_bounds__(kTThreads) void fft_single_kernel(FftArgs a) {
    constexpr int kRegPoints = (1 << kTile) / kTThreads;
    extern __shared__ double2 lds[];
    const int64_t items = work_items<kRagged>(a, 1);
    for (int64_t base = 0; base < items; base += gridDim.x) {
    const int64_t item = base + blockIdx.x;
    if (item >= items) break;
    const int64_t pair = pair_at<kRagged>(a, item);
    const Seq qa = seq_of(a, 2 * pair), qb = seq_of(a, 2 * pair + 1);
    const int lg = a.lg;
    const int len = 1 << lg;
    const double2* tw = a.tw + a.tw_a;
    {   // all loads of a thread in flight before its LDS writes
        double2 v[kRegPoints];
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int i = threadIdx.x + r * kTThreads;
            v[r] = make_double2(centred(qa, i), centred(qb, i));
        }
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int i = threadIdx.x + r * kTThreads;
            if (i < len) lds[i] = v[r];
        }
    }
    __syncthreads();
    lds_fft_fwd<kTile>(lds, lg, 0, tw);
    double2 wv[kRegPoints];
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int pos = threadIdx.x + r * kTThreads;
        if (pos < len) {
            const uint32_t k = bitrev(pos, lg);
            const uint32_t km = (len - k) & (len - 1);
            wv[r] = power_pair(lds[pos], lds[bitrev(km, lg)]);
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int pos = threadIdx.x + r * kTThreads;
        if (pos < len) lds[pos] = wv[r];
    }
    __syncthreads();
    lds_fft_inv<kTile>(lds, lg, 0, tw);
    const int64_t tend = min((int64_t)a.tmax, (int64_t)len - 1);
    for (int64_t t = a.tmin + threadIdx.x; t <= tend; t += kTThreads) {
        write_d(a, 2 * pair, t, lds[t].x);
        write_d(a, 2 * pair + 1, t, lds[t].y);
    }
    if (!kRagged) break;
    __syncthreads();   // the next pair reuses the LDS
    }
}

// Split transform, step 1: column transforms (L1 points, stride L2) of
// 2^lgc neighbouring columns, then the twiddles W_L^(k1 n2).  Row p of the
// output holds frequency k1 = bitrev(p).
template <int kTile, bool kRagged>
__global__ __launch_bounds__(kTThreads) void fft_cols_fwd_kernel(FftArgs a) {
    constexpr int kRegPoints = (1 << kTile) / kTThreads;
    extern __shared__ double2 lds[];
    const int64_t groups = int64_t(1) << (a.lg2 - a.lgc);
    const int64_t items = work_items<kRagged>(a, groups);
    for (int64_t base = 0; base < items; base += gridDim.x) {
    const int64_t id = base + xcd_remap(blockIdx.x, gridDim.x);
    if (id >= items) break;
    const int64_t pair = pair_at<kRagged>(a, id / groups);
    const int64_t c0 = (id % groups) << a.lgc;
    const int cols = 1 << a.lgc;
    const int npts = (1 << a.lg1) * cols;
    const int64_t l2 = int64_t(1) << a.lg2;
    const Seq qa = seq_of(a, 2 * pair), qb = seq_of(a, 2 * pair + 1);
    double2* twl = lds + npts;   // the pass twiddles, after the tile
    // Tiles of four or more columns whose rows start on 16-byte boundaries: a
    // thread takes runs of four points of a row (their four samples of each
    // sequence in one 16-byte load) instead of single points.
    auto aligned = [&](const Seq& q) {
        return q.n == 0 || ((reinterpret_cast<uintptr_t>(q.p + c0) & 15) == 0);
    };
    const bool rows4 = a.lgc >= 2 && npts == kRegPoints * kTThreads && (l2 & 3) == 0 &&
                       aligned(qa) && aligned(qb);
    const bool lds4 = four_step_in_lds(a.lg1, a.lg2);
    double2* tl = twl + (1 << (a.lg1 - 1));   // the four-step twiddles, after the pass ones
    FourStepCopy fc;
    if (lds4) fc.load(a);
    if (rows4) {   // all loads of a thread in flight before its LDS writes
        constexpr int kRows = kRegPoints / 4;   // runs of four points a thread
        const int quads = cols >> 2;            // runs in a row of the tile
        TwiddleCopy<kTile> tc;
        tc.load(a.tw + a.tw_a, a.lg1);
        auto row_of = [&](const Seq& q, int64_t i) -> float4 {
            if (i + 3 < q.n) return *reinterpret_cast<const float4*>(q.p + i);
            float4 f4 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            if (i < q.n) f4.x = q.p[i];
            if (i + 1 < q.n) f4.y = q.p[i + 1];
            if (i + 2 < q.n) f4.z = q.p[i + 2];
            return f4;
        };
        float4 va[kRows], vb[kRows];
#pragma unroll
        for (int k = 0; k < kRows; ++k) {
            const int qd = threadIdx.x + k * kTThreads;   // points 4 qd .. 4 qd + 3
            const int64_t i = (int64_t)(qd / quads) * l2 + c0 + 4 * (qd % quads);
            va[k] = row_of(qa, i);
            vb[k] = row_of(qb, i);
        }
        tc.store(twl, a.lg1);
        if (lds4) fc.store(a, tl);
#pragma unroll
        for (int k = 0; k < kRows; ++k) {
            const int qd = threadIdx.x + k * kTThreads;
            const int f = 4 * qd;
            const int64_t i = (int64_t)(qd / quads) * l2 + c0 + 4 * (qd % quads);
            // the same values as centred(): (double)x - mu inside the sequence, 0 past it
            auto cv = [&](const Seq& q, float x, int64_t ii) {
                return ii < q.n ? (double)x - q.mu : 0.0;
            };
            lds[f + 0] = make_double2(cv(qa, va[k].x, i), cv(qb, vb[k].x, i));
            lds[f + 1] = make_double2(cv(qa, va[k].y, i + 1), cv(qb, vb[k].y, i + 1));
            lds[f + 2] = make_double2(cv(qa, va[k].z, i + 2), cv(qb, vb[k].z, i + 2));
            lds[f + 3] = make_double2(cv(qa, va[k].w, i + 3), cv(qb, vb[k].w, i + 3));
        }
    } else {   // all loads of a thread in flight before its LDS writes
        TwiddleCopy<kTile> tc;
        tc.load(a.tw + a.tw_a, a.lg1);
        double2 v[kRegPoints];
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            const int64_t i = f < npts ? (int64_t)(f >> a.lgc) * l2 + c0 + (f & (cols - 1)) : a.len;
            v[r] = make_double2(centred(qa, i), centred(qb, i));
        }
        tc.store(twl, a.lg1);
        if (lds4) fc.store(a, tl);
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            if (f < npts) lds[f] = v[r];
        }
    }
    __syncthreads();
    lds_fft_fwd<kTile>(lds, a.lg1, a.lgc, twl);
    double2* __restrict__ zp = a.z + pair * a.zstride;
    double2 w[kRegPoints];
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {   // twiddle loads first
        const int f = threadIdx.x + r * kTThreads;
        const int64_t k1 = bitrev(f >> a.lgc, a.lg1);
        w[r] = f < npts ? twiddle_at(a, tl, lds4, k1 * (c0 + (f & (cols - 1))))
                        : make_double2(1.0, 0.0);
    }
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int f = threadIdx.x + r * kTThreads;
        if (f < npts) zp[(int64_t)(f >> a.lgc) * l2 + c0 + (f & (cols - 1))] = cmul(lds[f], w[r]);
    }
    if (!kRagged) break;
    __syncthreads();   // the next item reuses the LDS
    }
}

// Split transform, step 2: row k1 and its mirror row L1 - k1 (frequencies k
// and L - k pair up between them): forward row transforms, separation into
// the two sequences' power spectra, inverse row transforms, inverse twiddles.
// A workgroup takes 2^lgr consecutive row pairs (4096 points in LDS).
template <int kTile, bool kRagged>
__global__ __launch_bounds__(kTThreads) void fft_rows_kernel(FftArgs a) {
    constexpr int kRegPoints = (1 << kTile) / kTThreads;
    extern __shared__ double2 lds[];   // point i of slot q at i * 2^(lgr+1) + q
    const int64_t per = (int64_t(1) << (a.lg1 - 1)) + 1;   // row pairs per transform
    const int64_t wgs = (per + (1 << a.lgr) - 1) >> a.lgr;
    const int64_t items = work_items<kRagged>(a, wgs);
    for (int64_t base = 0; base < items; base += gridDim.x) {
    const int64_t id = base + xcd_remap(blockIdx.x, gridDim.x);
    if (id >= items) break;
    const int64_t pair = pair_at<kRagged>(a, id / wgs);
    const int64_t g0 = (id % wgs) << a.lgr;
    const uint32_t l1 = 1u << a.lg1;
    const int lgs = a.lgr + 1;                 // log2 of the slots
    const int slots = 1 << lgs;
    const int l2 = 1 << a.lg2;
    const int npts = l2 << lgs;
    double2* __restrict__ zp = a.z + pair * a.zstride;
    // slot q: row pair g0 + (q >> 1), side q & 1 (0: k1 = g, 1: k1 = L1 - g)
    auto k1_of = [&](int q, bool& valid, bool& self) -> uint32_t {
        const int64_t g = g0 + (q >> 1);
        valid = g < per;
        const uint32_t ka = (uint32_t)g, kb = (l1 - (uint32_t)g) & (l1 - 1);
        self = ka == kb;
        return (q & 1) ? kb : ka;
    };
    double2* twl = lds + npts;   // the pass twiddles, after the tile
    const bool lds4 = four_step_in_lds(a.lg1, a.lg2);
    double2* tl = twl + (1 << (a.lg2 - 1));   // the four-step twiddles, after the pass ones
    {   // all loads of a thread in flight before its LDS writes
        TwiddleCopy<kTile> tc;
        tc.load(a.tw + a.tw_b, a.lg2);
        FourStepCopy fc;
        if (lds4) fc.load(a);
        double2 v[kRegPoints];
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            bool valid, self;
            const uint32_t k1 = k1_of(f & (slots - 1), valid, self);
            v[r] = (valid && f < npts) ? zp[(int64_t)bitrev(k1, a.lg1) * l2 + (f >> lgs)]
                                       : make_double2(0.0, 0.0);
        }
        tc.store(twl, a.lg2);
        if (lds4) fc.store(a, tl);
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            if (f < npts) lds[f] = v[r];
        }
    }
    __syncthreads();
    lds_fft_fwd<kTile>(lds, a.lg2, lgs, twl);
    double2 wv[kRegPoints];
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int f = threadIdx.x + r * kTThreads;
        if (f < npts) {
            const int q = f & (slots - 1);
            bool valid, self;
            const uint32_t k1 = k1_of(q, valid, self);
            const uint32_t k2 = bitrev(f >> lgs, a.lg2);
            const uint32_t k2m = k1 == 0 ? ((l2 - k2) & (l2 - 1)) : (l2 - 1 - k2);
            const int qm = self ? q : (q ^ 1);
            wv[r] = power_pair(lds[f], lds[(bitrev(k2m, a.lg2) << lgs) + qm]);
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int f = threadIdx.x + r * kTThreads;
        if (f < npts) lds[f] = wv[r];
    }
    __syncthreads();
    lds_fft_inv<kTile>(lds, a.lg2, lgs, twl);
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {   // twiddle loads first (wv is free again)
        const int f = threadIdx.x + r * kTThreads;
        bool valid, self;
        const uint32_t k1 = k1_of(f & (slots - 1), valid, self);
        wv[r] = (f < npts && valid) ? twiddle_at(a, tl, lds4, (int64_t)k1 * (f >> lgs))
                                    : make_double2(1.0, 0.0);
    }
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int f = threadIdx.x + r * kTThreads;
        const int q = f & (slots - 1);
        bool valid, self;
        const uint32_t k1 = k1_of(q, valid, self);
        if (f >= npts || !valid || ((q & 1) && self)) continue;
        zp[(int64_t)bitrev(k1, a.lg1) * l2 + (f >> lgs)] = cmul_conj(lds[f], wv[r]);
    }
    if (!kRagged) break;
    __syncthreads();   // the next item reuses the LDS
    }
}

// 4 Q(k) of the wrap correction from the head transform Z1 = FFT(h_a + i h_b)
// and the tail transform Z2 = FFT(u_a + i u_b) at k and L - k:
// with H_a = (Z1(k) + conj Z1(L-k)) / 2, H_b = (Z1(k) - conj Z1(L-k)) / 2i and
// U_a, U_b likewise from Z2, Q = U_a conj(H_a) + i U_b conj(H_b), whose
// inverse transform is cc_a + i cc_b, cc(s) = sum_j h_j u_{j+s}.
__device__ __forceinline__ double2 cross_pair(double2 z1k, double2 z1m, double2 z2k, double2 z2m) {
    const double2 ha = make_double2(z1k.x + z1m.x, z1k.y - z1m.y);   // 2 H_a
    const double2 hb = make_double2(z1k.y + z1m.y, z1m.x - z1k.x);   // 2 H_b
    const double2 ua = make_double2(z2k.x + z2m.x, z2k.y - z2m.y);   // 2 U_a
    const double2 ub = make_double2(z2k.y + z2m.y, z2m.x - z2k.x);   // 2 U_b
    const double2 pa = cmul_conj(ua, ha), pb = cmul_conj(ub, hb);
    return make_double2(pa.x - pb.y, pa.y + pb.x);
}

// Wrap correction, step 2: rows k1 and L1 - k1 of both the head transform
// (at z) and the tail transform (at z + zoff2) of 2^lgr consecutive row pairs:
// forward row transforms, the cross spectrum Q of the pair, inverse row
// transforms of Q and the inverse twiddles; Q's rows go over the head
// transform's rows.  LDS: point i of slot q at i * 4 * 2^lgr + q, slot q =
// (row pair, side, transform) from the high bits down; Q then takes the
// layout of two slots per row pair.
template <int kTile>
__global__ __launch_bounds__(kTThreads) void fft_wrap_rows_kernel(FftArgs a, int64_t zoff2) {
    constexpr int kRegPoints = (1 << kTile) / kTThreads;
    extern __shared__ double2 lds[];
    const int64_t per = (int64_t(1) << (a.lg1 - 1)) + 1;
    const int64_t wgs = (per + (1 << a.lgr) - 1) >> a.lgr;
    const int64_t id = xcd_remap(blockIdx.x, gridDim.x);
    const int64_t pair = id / wgs;
    const int64_t g0 = (id % wgs) << a.lgr;
    const uint32_t l1 = 1u << a.lg1;
    const int lgs = a.lgr + 2;
    const int slots = 1 << lgs;
    const int l2 = 1 << a.lg2;
    const int npts = l2 << lgs;
    double2* __restrict__ z1 = a.z + pair * a.zstride;
    const double2* __restrict__ z2 = z1 + zoff2;
    auto k1_of = [&](int64_t g, int side, bool& valid, bool& self) -> uint32_t {
        valid = g < per;
        const uint32_t ka = (uint32_t)g, kb = (l1 - (uint32_t)g) & (l1 - 1);
        self = ka == kb;
        return side ? kb : ka;
    };
    double2* twl = lds + npts;   // the pass twiddles, after the tile
    {
        TwiddleCopy<kTile> tc;
        tc.load(a.tw + a.tw_b, a.lg2);
        double2 v[kRegPoints];
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            const int q = f & (slots - 1);
            bool valid, self;
            const uint32_t k1 = k1_of(g0 + (q >> 2), (q >> 1) & 1, valid, self);
            const double2* src = (q & 1) ? z2 : z1;
            v[r] = (valid && f < npts) ? src[(int64_t)bitrev(k1, a.lg1) * l2 + (f >> lgs)]
                                       : make_double2(0.0, 0.0);
        }
        tc.store(twl, a.lg2);
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            if (f < npts) lds[f] = v[r];
        }
    }
    __syncthreads();
    lds_fft_fwd<kTile>(lds, a.lg2, lgs, twl);
    double2 wv[kRegPoints];
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {   // at the head transform's slots
        const int f = threadIdx.x + r * kTThreads;
        const int q = f & (slots - 1);
        if (f < npts && (q & 1) == 0) {
            bool valid, self;
            const uint32_t k1 = k1_of(g0 + (q >> 2), (q >> 1) & 1, valid, self);
            const uint32_t k2 = bitrev(f >> lgs, a.lg2);
            const uint32_t k2m = k1 == 0 ? ((l2 - k2) & (l2 - 1)) : (l2 - 1 - k2);
            const int qm = self ? q : (q ^ 2);
            const int fm = (int)(bitrev(k2m, a.lg2) << lgs) + qm;
            wv[r] = cross_pair(lds[f], lds[fm], lds[f + 1], lds[fm + 1]);
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {   // Q: point i of slot q >> 1 at i * slots / 2 + (q >> 1)
        const int f = threadIdx.x + r * kTThreads;
        const int q = f & (slots - 1);
        if (f < npts && (q & 1) == 0) lds[(f >> lgs) * (slots >> 1) + (q >> 1)] = wv[r];
    }
    __syncthreads();
    lds_fft_inv<kTile>(lds, a.lg2, lgs - 1, twl);
    const int half = npts >> 1;
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {   // twiddle loads first
        const int f = threadIdx.x + r * kTThreads;
        const int q2 = f & ((slots >> 1) - 1);
        bool valid, self;
        const uint32_t k1 = k1_of(g0 + (q2 >> 1), q2 & 1, valid, self);
        wv[r] = (f < half && valid) ? twiddle(a, (int64_t)k1 * (f >> (lgs - 1)))
                                    : make_double2(1.0, 0.0);
    }
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int f = threadIdx.x + r * kTThreads;
        const int q2 = f & ((slots >> 1) - 1);
        bool valid, self;
        const uint32_t k1 = k1_of(g0 + (q2 >> 1), q2 & 1, valid, self);
        if (f >= half || !valid || ((q2 & 1) && self)) continue;
        z1[(int64_t)bitrev(k1, a.lg1) * l2 + (f >> (lgs - 1))] = cmul_conj(lds[f], wv[r]);
    }
}

// Split transform, step 3: inverse column transforms (row p holds k1 =
// bitrev(p): the bit-reversed input order of the decimation in time), and
// D(T) for the lags T = n1 L2 + n2 in [tmin, tmax].
template <int kTile, bool kRagged>
__global__ __launch_bounds__(kTThreads) void fft_cols_inv_kernel(FftArgs a) {
    constexpr int kRegPoints = (1 << kTile) / kTThreads;
    extern __shared__ double2 lds[];
    const int64_t groups = int64_t(1) << (a.lg2 - a.lgc);
    const int64_t items = work_items<kRagged>(a, groups);
    for (int64_t base = 0; base < items; base += gridDim.x) {
    const int64_t id = base + xcd_remap(blockIdx.x, gridDim.x);
    if (id >= items) break;
    const int64_t pair = pair_at<kRagged>(a, id / groups);
    const int64_t c0 = (id % groups) << a.lgc;
    const int cols = 1 << a.lgc;
    const int npts = (1 << a.lg1) * cols;
    const int64_t l2 = int64_t(1) << a.lg2;
    const double2* __restrict__ zp = a.z + pair * a.zstride;
    double2* twl = lds + npts;   // the pass twiddles, after the tile
    {   // all loads of a thread in flight before its LDS writes
        TwiddleCopy<kTile> tc;
        tc.load(a.tw + a.tw_a, a.lg1);
        double2 v[kRegPoints];
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            v[r] = f < npts ? zp[(int64_t)(f >> a.lgc) * l2 + c0 + (f & (cols - 1))]
                            : make_double2(0.0, 0.0);
        }
        tc.store(twl, a.lg1);
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            if (f < npts) lds[f] = v[r];
        }
    }
    __syncthreads();
    lds_fft_inv<kTile>(lds, a.lg1, a.lgc, twl);
    if (a.wout) {   // head-tail transform: cc_a(s) + i cc_b(s) for shifts s < wm
        const int rows = (int)min((int64_t)((a.wm - 1) / l2) + 1, int64_t(1) << a.lg1);
        for (int f = threadIdx.x; f < rows * cols; f += kTThreads) {
            const int64_t sh = (int64_t)(f >> a.lgc) * l2 + c0 + (f & (cols - 1));
            if (sh >= a.wm) continue;
            a.wout[2 * pair * a.wm + sh] = ldexp(lds[f].x, -(a.lg + 2));
            if (2 * pair + 1 < a.seqs) a.wout[(2 * pair + 1) * a.wm + sh] = ldexp(lds[f].y, -(a.lg + 2));
        }
    } else {
        const int rows = (int)min((int64_t)(a.tmax / l2) + 1, int64_t(1) << a.lg1);
        for (int f = threadIdx.x; f < rows * cols; f += kTThreads) {
            const int64_t t = (int64_t)(f >> a.lgc) * l2 + c0 + (f & (cols - 1));
            write_d(a, 2 * pair, t, lds[f].x);
            write_d(a, 2 * pair + 1, t, lds[f].y);
        }
    }
    if (!kRagged) break;
    __syncthreads();   // the next item reuses the LDS
    }
}

// Amplitudes |X_a(k)| and |X_b(k)| of the two sequences of a pair at
// frequency k <= L/2, from Z(k) and Z(L - k): |Z(k) + conj Z(L-k)| / 2 and
// |Z(k) - conj Z(L-k)| / 2.
__device__ __forceinline__ void write_amplitudes(const FftArgs& a, int64_t pair, int64_t k,
                                                 double2 zk, double2 zm) {
    const double ux = zk.x + zm.x, uy = zk.y - zm.y;
    const double vx = zk.x - zm.x, vy = zk.y + zm.y;
    const int64_t half = a.len / 2 + 1;
    const int64_t sa = 2 * pair, sb = sa + 1;
    a.amp[sa * half + k] = 0.5 * sqrt(ux * ux + uy * uy);
    if (sb < a.seqs) a.amp[sb * half + k] = 0.5 * sqrt(vx * vx + vy * vy);
}

// Spectrum of one pair in one workgroup (L up to one tile).
template <int kTile>
__global__ __launch_bounds__(kTThreads) void spec_single_kernel(FftArgs a) {
    constexpr int kRegPoints = (1 << kTile) / kTThreads;
    extern __shared__ double2 lds[];
    const int64_t pair = blockIdx.x;
    const Seq qa = seq_of(a, 2 * pair), qb = seq_of(a, 2 * pair + 1);
    const int lg = a.lg;
    const int len = 1 << lg;
    {
        double2 v[kRegPoints];
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int i = threadIdx.x + r * kTThreads;
            v[r] = make_double2(centred(qa, i), centred(qb, i));
        }
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int i = threadIdx.x + r * kTThreads;
            if (i < len) lds[i] = v[r];
        }
    }
    __syncthreads();
    lds_fft_fwd<kTile>(lds, lg, 0, a.tw + a.tw_a);
    for (int pos = threadIdx.x; pos < len; pos += kTThreads) {
        const uint32_t k = bitrev(pos, lg);
        if (k > (uint32_t)(len / 2)) continue;
        const uint32_t km = (len - k) & (len - 1);
        write_amplitudes(a, pair, k, lds[pos], lds[bitrev(km, lg)]);
    }
}

// Spectrum of a split transform: after the column kernel, forward row
// transforms of row pairs (k1, L1 - k1), then the amplitudes at every
// frequency k = k1 + L1 k2 <= L/2 (each written once: a self-paired row only
// from its first slot).
template <int kTile>
__global__ __launch_bounds__(kTThreads) void spec_rows_kernel(FftArgs a) {
    constexpr int kRegPoints = (1 << kTile) / kTThreads;
    extern __shared__ double2 lds[];
    const int64_t per = (int64_t(1) << (a.lg1 - 1)) + 1;
    const int64_t wgs = (per + (1 << a.lgr) - 1) >> a.lgr;
    const int64_t id = xcd_remap(blockIdx.x, gridDim.x);
    const int64_t pair = id / wgs;
    const int64_t g0 = (id % wgs) << a.lgr;
    const uint32_t l1 = 1u << a.lg1;
    const int lgs = a.lgr + 1;
    const int slots = 1 << lgs;
    const int l2 = 1 << a.lg2;
    const int npts = l2 << lgs;
    const double2* __restrict__ zp = a.z + pair * a.zstride;
    auto k1_of = [&](int q, bool& valid, bool& self) -> uint32_t {
        const int64_t g = g0 + (q >> 1);
        valid = g < per;
        const uint32_t ka = (uint32_t)g, kb = (l1 - (uint32_t)g) & (l1 - 1);
        self = ka == kb;
        return (q & 1) ? kb : ka;
    };
    {
        double2 v[kRegPoints];
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            bool valid, self;
            const uint32_t k1 = k1_of(f & (slots - 1), valid, self);
            v[r] = (valid && f < npts) ? zp[(int64_t)bitrev(k1, a.lg1) * l2 + (f >> lgs)]
                                       : make_double2(0.0, 0.0);
        }
#pragma unroll
        for (int r = 0; r < kRegPoints; ++r) {
            const int f = threadIdx.x + r * kTThreads;
            if (f < npts) lds[f] = v[r];
        }
    }
    __syncthreads();
    lds_fft_fwd<kTile>(lds, a.lg2, lgs, a.tw + a.tw_b);
    const int64_t half_len = a.len / 2;
    for (int f = threadIdx.x; f < npts; f += kTThreads) {
        const int q = f & (slots - 1);
        bool valid, self;
        const uint32_t k1 = k1_of(q, valid, self);
        if (!valid || ((q & 1) && self)) continue;
        const uint32_t k2 = bitrev(f >> lgs, a.lg2);
        const int64_t k = (int64_t)k1 + (int64_t)l1 * k2;
        if (k > half_len) continue;
        const uint32_t k2m = k1 == 0 ? ((l2 - k2) & (l2 - 1)) : (l2 - 1 - k2);
        const int qm = self ? q : (q ^ 1);
        write_amplitudes(a, pair, k, lds[f], lds[(bitrev(k2m, a.lg2) << lgs) + qm]);
    }
}

// Absolute error bound of the computed D(T) of sequence s (any T), from the
// norms of s and of the sequence it shares the transform with.
//
// A radix-2 transform of L = 2^lg points with twiddles accurate to mu errs by
// at most phi ||exact||_2, phi = k eta / (1 - k eta), eta = mu + g4 (sqrt2 + mu)
// (Higham, Accuracy and Stability of Numerical Algorithms, Thm. 24.2), with k
// = lg + 1 stages (the split form adds the twiddle stage); mu = 16 u covers
// the table entries and the product of two of them.  Then, with zeta^2 =
// E_a + E_b, the spectrum of a errs by e1 sqrt(L) zeta (e1 = phi + 4u, with
// the separation); its power spectrum, summed over all frequencies and divided
// by L, errs by 2 e1 zeta |y_a| + (e1 zeta)^2 + g3 (|y_a| + e1 zeta)^2; the
// inverse transform adds phi (1 + g3) (|y_a|_1 + e1 sqrt(L) zeta)(|y_a| +
// e1 zeta) and the same for b.  Each bounds |r_computed(T) - r(T)|.  The
// energies E - head and E - tail are sums of at most 2N + 2 rounded terms
// (g_{2N+2} E each) plus the additions of the assembly, and centring in fp64
// moves D by at most 4u sqrt(D E) + 4 u^2 E <= 2u D + 3u E.  The result is
// doubled as a margin.
__device__ double fft_bound(const double* fstat, int64_t s, int64_t seqs, int64_t n, int lg) {
    const double u = 1.1102230246251565e-16;
    const double ea = fstat[4 * s + 1], la = fstat[4 * s + 2];
    const int64_t o = s ^ 1;
    const double eb = o < seqs ? fstat[4 * o + 1] : 0.0;
    const double lb = o < seqs ? fstat[4 * o + 2] : 0.0;
    const double ya = sqrt(ea), yb = sqrt(eb), zeta = sqrt(ea + eb);
    const double mu = 16.0 * u;
    const double g3 = 3.0 * u / (1.0 - 3.0 * u);
    const double g4 = 4.0 * u / (1.0 - 4.0 * u);
    const double eta = mu + g4 * (1.4142135623730951 + mu);
    const double keta = (double)(lg + 1) * eta;
    const double phi = keta / (1.0 - keta);
    const double e1 = phi + 4.0 * u;
    const double sl = sqrt(ldexp(1.0, lg));
    const double pa = ya + e1 * zeta, pb = yb + e1 * zeta;
    const double fwd = 2.0 * e1 * zeta * ya + e1 * e1 * zeta * zeta + g3 * pa * pa;
    const double inv = phi * (1.0 + g3) * ((la + e1 * sl * zeta) * pa + (lb + e1 * sl * zeta) * pb);
    const double k = 2.0 * (double)n + 2.0;
    const double ge = k * u / (1.0 - k * u);
    return 2.0 * (2.02 * (fwd + inv) + (2.0 * ge + 17.0 * u) * ea);
}

// Absolute error bound of the wrap term's share of D(T) (any T > W): the
// head-tail transform of 2^lg points takes z1 = h_a + i h_b and z2 = u_a + i u_b
// (the first and last M samples of a and of its partner b), whose norms the
// whole sequences' norms bound.  Each separated spectrum errs by e1 sqrt(L) zeta
// as in fft_bound; the products U conj H, summed over all frequencies and
// divided by L, err by 2 e1 zeta |y_a| + (e1 zeta)^2, their rounding and the
// assembly of Q (a product of two perturbed spectra and one addition each,
// within gamma_4) by g4 ((|y_a| + e1 zeta)^2 + (|y_b| + e1 zeta)^2), and the
// inverse transform by phi (1 + g3) ((|y_a|_1 + e1 sqrt(L) zeta)(|y_a| + e1 zeta)
// + the same for b).  The sum bounds |cc_computed(s) - cc(s)|; D takes it
// twice (D = ... - 2 (r_circ - cc)), with 1% margin, and the result is doubled.
__device__ double fft_bound_wrap(const double* fstat, int64_t s, int64_t seqs, int lg) {
    const double u = 1.1102230246251565e-16;
    const double ea = fstat[4 * s + 1], la = fstat[4 * s + 2];
    const int64_t o = s ^ 1;
    const double eb = o < seqs ? fstat[4 * o + 1] : 0.0;
    const double lb = o < seqs ? fstat[4 * o + 2] : 0.0;
    const double ya = sqrt(ea), yb = sqrt(eb), zeta = sqrt(ea + eb);
    const double mu = 16.0 * u;
    const double g3 = 3.0 * u / (1.0 - 3.0 * u);
    const double g4 = 4.0 * u / (1.0 - 4.0 * u);
    const double eta = mu + g4 * (1.4142135623730951 + mu);
    const double keta = (double)(lg + 1) * eta;
    const double phi = keta / (1.0 - keta);
    const double e1 = phi + 4.0 * u;
    const double sl = sqrt(ldexp(1.0, lg));
    const double pa = ya + e1 * zeta, pb = yb + e1 * zeta;
    const double fwd = 2.0 * e1 * zeta * ya + e1 * e1 * zeta * zeta + g4 * (pa * pa + pb * pb);
    const double inv = phi * (1.0 + g3) * ((la + e1 * sl * zeta) * pa + (lb + e1 * sl * zeta) * pb);
    return 2.0 * (2.02 * (fwd + inv));
}

struct FixArgs {
    const float* x;
    const double* fstat;
    double* s64;
    float* scores;
    uint32_t* tier1;
    WinState* state;
    int64_t seqs;
    int64_t n_all, window_stride, channel_stride;
    int32_t num_channels, tmin, tmax, lags, words, lg;
    double tau0;
    WindowTable tab;
    const int32_t* pair_lg;    // per pair: log2 of its transform length, or null (all lg)
    int32_t wrap_lg;           // log2 of the head-tail transform (wrap correction), or -1
};

// One workgroup per window: lags whose score the FFT bound cannot place within
// tau0 / 2 of itself (the other half covers the rounding of the finalisation
// and of the sequential evaluation) are re-scored by a wavefront in fp64 and
// marked tier 1.  A score of exactly zero always lands here.
__global__ __launch_bounds__(kThreads) void fft_fixup_kernel(FixArgs a, Weights w) {
    __shared__ double abound;
    const int64_t b = blockIdx.x;
    const int64_t n = table_n(a.tab, b, a.n_all);
    if (n == 0) return;
    const int32_t tm = table_tmax(a.tab, b, a.tmax);
    if (threadIdx.x == 0) {
        double acc = 0.0;
        for (int32_t c = 0; c < a.num_channels; ++c) {
            const int64_t sq = b * a.num_channels + c;
            const int lg = a.pair_lg ? a.pair_lg[sq >> 1] : a.lg;
            double e = fft_bound(a.fstat, sq, a.seqs, n, lg);
            if (a.wrap_lg >= 0) e += fft_bound_wrap(a.fstat, sq, a.seqs, a.wrap_lg);
            acc += (double)w.w[c] * e;
        }
        abound = acc * (1.0 + 1e-12);
    }
    __syncthreads();
    const double ab = abound;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x >> 6;
    const float* __restrict__ xw = a.x + table_off(a.tab, b, a.window_stride);
    const int32_t nlags = tm - a.tmin + 1;
    // wavefront w tests lags j0 + lane, j0 = 64 w + 256 k; the scores of
    // kFixBatch consecutive k are loaded together (all in flight), then tested
    constexpr int kFixBatch = 8;
    for (int32_t jb = wave * kWave; jb < nlags; jb += kThreads * kFixBatch) {
    double vb[kFixBatch];
#pragma unroll
    for (int r = 0; r < kFixBatch; ++r) {
        const int32_t j = jb + r * kThreads + lane;
        vb[r] = j < nlags ? a.s64[b * a.lags + j] : 0.0;
    }
#pragma unroll
    for (int r = 0; r < kFixBatch; ++r) {
        const int32_t j0 = jb + r * kThreads;
        const int32_t j = j0 + lane;
        bool fix = false;
        if (j < nlags) {
            const int64_t t = (int64_t)a.tmin + j;
            fix = !(ab / (double)(n - t) <= 0.5 * a.tau0 * vb[r]);
        }
        uint64_t mask = __ballot(fix);
        while (mask) {
            const int k = __builtin_ctzll(mask);
            mask &= mask - 1;
            const int32_t jj = j0 + k;
            const int64_t t = (int64_t)a.tmin + jj;
            const double v =
                exact::wave_score(xw, a.num_channels, a.channel_stride, n, t, w, lane);
            if (lane == 0) {
                a.s64[b * a.lags + jj] = v;
                if (a.scores) a.scores[b * a.lags + jj] = (float)v;
                atomicOr(&a.tier1[b * a.words + (jj >> 5)], 1u << (jj & 31));
                atomicAdd(&a.state[b].rescored, 1);
            }
        }
    }
    }
}

struct SpecSelArgs {
    double* amp;               // [S][half]: per-channel amplitudes, channel 0 overwritten by A
    const double* fstat;       // [S][4]
    gpoeo_pd_spectral_result* out;
    int64_t seqs, half, len;
    int32_t num_channels, tmin, tmax, k_max, lg;
    double c_peak;
};

constexpr int kCandCap = 1024;   // candidates collected per window

// Candidates of one window from its amplitude spectrum A(k) = sum_c w_c |X_c(k)|:
// peaks (2 <= k <= L/2 - 1, A(k) > A(k-1), A(k) >= A(k+1)), the largest peak,
// then the peaks above c_peak times it whose period round(L/k) is in
// [tmin, tmax], strongest first (ties: smaller k).  The window is flagged
// UNRESOLVED when a peak test, the threshold, or the order of the reported
// candidates lies within four times the amplitude error bound (the list a
// correctly rounded spectrum gives could then differ), or when more than
// kCandCap candidates qualify.
template <int kThreads>
__global__ __launch_bounds__(kThreads) void spec_select_kernel(SpecSelArgs a, Weights w) {
    __shared__ double red[kThreads];
    __shared__ int32_t redi[kThreads];
    __shared__ double cand_a[kCandCap];
    __shared__ int32_t cand_k[kCandCap];
    __shared__ int32_t ncand;
    __shared__ int32_t flag;
    const int64_t b = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t half = a.half;               // L/2 + 1 bins
    double* __restrict__ amp = a.amp + b * a.num_channels * half;
    // 1. channel sum in channel order (into channel 0)
    for (int64_t k = tid; k < half; k += kThreads) {
        double acc = 0.0;
        for (int32_t c = 0; c < a.num_channels; ++c) acc += (double)w.w[c] * amp[c * half + k];
        amp[k] = acc;
    }
    if (tid == 0) {
        ncand = 0;
        flag = 0;
    }
    __syncthreads();
    // 2. peaks and the largest one
    double mx = 0.0;
    int32_t npk = 0;
    for (int64_t k = 2 + tid; k <= half - 2; k += kThreads) {
        const double v = amp[k];
        if (v > amp[k - 1] && v >= amp[k + 1]) {
            ++npk;
            mx = fmax(mx, v);
        }
    }
    red[tid] = mx;
    redi[tid] = npk;
    __syncthreads();
    for (int st = kThreads / 2; st > 0; st >>= 1) {
        if (tid < st) {
            red[tid] = fmax(red[tid], red[tid + st]);
            redi[tid] += redi[tid + st];
        }
        __syncthreads();
    }
    const double top = red[0];
    const int32_t n_peaks = redi[0];
    __syncthreads();
    // 3. error bound of A (any k): the transform bound of each channel's pair
    // (as for the FFT scores: phi sqrt(L) zeta, plus the separation), summed
    // with the weights, plus the rounding of the amplitude and the channel sum
    const double u = 1.1102230246251565e-16;
    const double mu = 16.0 * u;
    const double g4 = 4.0 * u / (1.0 - 4.0 * u);
    const double keta = (double)(a.lg + 1) * (mu + g4 * (1.4142135623730951 + mu));
    const double phi = keta / (1.0 - keta);
    double eps = 0.0;
    for (int32_t c = 0; c < a.num_channels; ++c) {
        const int64_t sq = b * a.num_channels + c, o = sq ^ 1;
        const double z2 = a.fstat[4 * sq + 1] + (o < a.seqs ? a.fstat[4 * o + 1] : 0.0);
        eps += (double)w.w[c] * (phi + 4.0 * u) * sqrt((double)a.len) * sqrt(z2);
    }
    eps = 2.0 * (eps + ((double)a.num_channels + 6.0) * u * top);
    const double m = 4.0 * eps;
    const double thr = a.c_peak * top;
    // 4. candidates, and decisions too close to call
    for (int64_t k = 2 + tid; k <= half - 2; k += kThreads) {
        const double v = amp[k];
        if (v + m < a.c_peak * (top - m)) continue;       // cannot matter
        const double l = amp[k - 1], r = amp[k + 1];
        const bool peak = v > l && v >= r;
        if (fabs(v - l) <= m || fabs(v - r) <= m) atomicOr(&flag, 1);
        if (!peak) continue;
        const int64_t t = (2 * a.len + k) / (2 * k);       // round(L / k), halves up
        if (t < a.tmin || t > a.tmax) continue;
        if (fabs(v - thr) <= m * (1.0 + a.c_peak)) atomicOr(&flag, 1);
        if (!(v > thr)) continue;
        const int slot = atomicAdd(&ncand, 1);
        if (slot < kCandCap) {
            cand_a[slot] = v;
            cand_k[slot] = (int32_t)k;
        } else {
            atomicOr(&flag, 2);
        }
    }
    __syncthreads();
    const int nc = min(ncand, kCandCap);
    // 5. the strongest first: rounds of a block-wide arg-max (larger A, then smaller k)
    gpoeo_pd_spectral_result res = {};
    double prev = 0.0;
    int rounds = min(nc, a.k_max + 1);                     // one more to check the order
    for (int r = 0; r < rounds; ++r) {
        double bv = -1.0;
        int32_t bk = INT32_MAX, bi = -1;
        for (int i = tid; i < nc; i += kThreads) {
            const double v = cand_a[i];
            if (v > bv || (v == bv && cand_k[i] < bk)) {
                bv = v;
                bk = cand_k[i];
                bi = i;
            }
        }
        red[tid] = bv;
        redi[tid] = bi;
        __syncthreads();
        for (int st = kThreads / 2; st > 0; st >>= 1) {
            if (tid < st) {
                const int i1 = redi[tid + st], i0 = redi[tid];
                const double v1 = red[tid + st], v0 = red[tid];
                if (i1 >= 0 && (i0 < 0 || v1 > v0 || (v1 == v0 && cand_k[i1] < cand_k[i0]))) {
                    red[tid] = v1;
                    redi[tid] = i1;
                }
            }
            __syncthreads();
        }
        const int best = redi[0];
        const double bvv = red[0];
        __syncthreads();
        if (tid == 0) {
            if (r > 0 && prev - bvv <= m) flag |= 1;
            if (r < a.k_max) {
                const int32_t k = cand_k[best];
                res.periods[r] = (int32_t)((2 * a.len + k) / (2 * (int64_t)k));
                res.bins[r] = k;
                res.amplitudes[r] = bvv;
                res.count = r + 1;
            }
            cand_a[best] = -1.0;                           // taken
        }
        prev = bvv;
        __syncthreads();
    }
    if (tid == 0) {
        res.n_peaks = n_peaks;
        res.max_peak = top;
        res.flags = flag ? GPOEO_PD_UNRESOLVED : 0u;
        a.out[b] = res;
    }
}

// Length classes of a batch of windows of different lengths (a window table):
// the class of a pair is the log2 of the smallest power of two (at least 64)
// holding N + Tmax of each non-empty sequence of the pair, -1 if both are
// empty.  Writes every pair's class, then the pairs sorted by class (ascending
// pair index within a class: a stable counting sort in one workgroup) and the
// start of each class in that list.
constexpr int kClassThreads = 1024;
constexpr int kClassWaves = kClassThreads / kWave;

struct ClassArgs {
    int32_t* pair_lg;          // [pairs]
    int32_t* list;             // [pairs]
    int32_t* bounds;           // [kFftClasses + 1]
    int64_t pairs, seqs, n_all;
    int32_t num_channels, tmax, lg_max;
    WindowTable tab;
};

__device__ int class_of(const ClassArgs& a, int64_t pair) {
    int lg = -1;
    for (int64_t s = 2 * pair; s < 2 * pair + 2 && s < a.seqs; ++s) {
        const int64_t b = s / a.num_channels;
        const int64_t n = table_n(a.tab, b, a.n_all);
        if (n <= 0) continue;
        const int64_t need = n + (int64_t)min(table_tmax(a.tab, b, a.tmax), a.tmax);
        int l = kFftMinLog2;
        while (l < a.lg_max && (int64_t(1) << l) < need) ++l;
        lg = max(lg, l);
    }
    return lg;
}

__global__ __launch_bounds__(kClassThreads) void fft_classify_kernel(ClassArgs a) {
    __shared__ int32_t run[kFftClasses];
    __shared__ int32_t wcount[kClassWaves][kFftClasses];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    if (tid < kFftClasses) run[tid] = 0;
    __syncthreads();
    for (int64_t p = tid; p < a.pairs; p += kClassThreads) {
        const int lg = class_of(a, p);
        a.pair_lg[p] = lg;
        if (lg >= 0) atomicAdd(&run[lg], 1);
    }
    __syncthreads();
    if (tid == 0) {
        int32_t acc = 0;
        for (int c = 0; c < kFftClasses; ++c) {
            const int32_t k = run[c];
            run[c] = acc;
            a.bounds[c] = acc;
            acc += k;
        }
        a.bounds[kFftClasses] = acc;
    }
    for (int64_t p0 = 0; p0 < a.pairs; p0 += kClassThreads) {
        for (int i = tid; i < kClassWaves * kFftClasses; i += kClassThreads)
            wcount[i / kFftClasses][i % kFftClasses] = 0;
        __syncthreads();
        const int64_t p = p0 + tid;
        const int lg = p < a.pairs ? a.pair_lg[p] : -1;   // written by this thread above
        int rank = 0;
        uint64_t todo = __ballot(lg >= 0);
        while (todo) {                                     // one round per class in the wave
            const int c = __shfl(lg, __builtin_ctzll(todo));
            const uint64_t same = __ballot(lg == c);
            if (lg == c) rank = __popcll(same & ((uint64_t(1) << lane) - 1));
            if (lane == 0) wcount[wave][c] = __popcll(same);
            todo &= ~same;
        }
        __syncthreads();
        if (lg >= 0) {
            int32_t off = run[lg] + rank;
            for (int w = 0; w < wave; ++w) off += wcount[w][lg];
            a.list[off] = (int32_t)p;
        }
        __syncthreads();
        if (tid < kFftClasses) {
            int32_t add = 0;
            for (int w = 0; w < kClassWaves; ++w) add += wcount[w][tid];
            run[tid] += add;
        }
        __syncthreads();
    }
}

// Transform geometry of 2^lg points in the launch arguments.
void set_geometry(FftArgs& a, int lg) {
    int32_t m1, m2, cols;
    fft_geometry(lg, &m1, &m2, &cols);
    a.lg = lg;
    a.len = int64_t(1) << lg;
    if (m2 == 1) {   // one workgroup per pair
        a.lg1 = lg;
        a.lg2 = 0;
        a.lgc = 0;
        a.lgr = 0;
        a.tw_a = 0;
        a.tw_b = a.tw_lo = a.tw_hi = 0;
    } else {
        a.lg1 = __builtin_ctz((unsigned)m1);
        a.lg2 = __builtin_ctz((unsigned)m2);
        a.lgc = __builtin_ctz((unsigned)cols);
        const int tile = fft_tile_log2(lg);
        a.lgr = a.lg2 >= tile - 1 ? 0 : tile - 1 - a.lg2;   // row pairs per tile
        a.tw_a = 0;
        a.tw_b = m1 / 2;
        a.tw_lo = a.tw_b + m2 / 2;
        a.tw_hi = a.tw_lo + m2;
    }
}

FftArgs args_of(const Plan& p, const float* x, double* fstat, double* edge, double* tw, double* z,
                double* part) {
    FftArgs a;
    a.x = x;
    a.fstat = fstat;
    a.edge = edge;
    a.tw = reinterpret_cast<const double2*>(tw);
    a.z = reinterpret_cast<double2*>(z);
    a.part = part;
    a.amp = nullptr;
    a.seqs = p.num_windows * (int64_t)p.num_channels;
    a.n_all = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    a.tmin = p.tmin;
    a.tmax = p.tmax;
    a.lags = p.lags;
    a.tab = p.table;
    a.list = nullptr;
    a.bounds = nullptr;
    a.zstride = p.fft_len;
    a.cls = 0;
    a.seg_start = 0;
    a.seg_len = 0;
    a.wout = nullptr;
    a.wrap = nullptr;
    a.wrap_w = 0;
    a.wm = 0;
    a.s64 = nullptr;
    a.scores = nullptr;
    a.w0 = 1.0f;
    set_geometry(a, p.fft_log2);
    return a;
}

// Workgroups of a ragged launch: the pairs of a class are known only on the
// GPU, so each launch gets a fixed grid whose workgroups loop over the class.
constexpr int64_t kRaggedGrid = 4096;

// The transform kernels for the geometry in `a`, over `pairs` pairs (a
// uniform batch: one workgroup per item), or over at most `pairs` pairs of one
// length class (ragged: a capped grid).
template <int kTile, bool kRagged>
void launch_transforms(const FftArgs& a, int64_t pairs, hipStream_t s) {
    auto grid = [&](int64_t items) {
        return dim3((unsigned)(kRagged ? std::min(items, kRaggedGrid) : items));
    };
    if (a.lg2 == 0) {
        const size_t lds = sizeof(double2) * (size_t)a.len;
        hipLaunchKernelGGL((fft_single_kernel<kTile, kRagged>), grid(pairs), dim3(kTThreads), lds,
                           s, a);
        return;
    }
    const int64_t m1 = int64_t(1) << a.lg1, m2 = int64_t(1) << a.lg2, cols = int64_t(1) << a.lgc;
    const int64_t col_groups = pairs * (m2 / cols);
    // tiles, then each kernel's pass twiddles (half a sub-transform), then for
    // the forward columns and the rows the four-step twiddles when they fit
    const size_t fs = four_step_in_lds(a.lg1, a.lg2) ? (size_t)(m1 + m2) : 0;
    const size_t lds_cols = sizeof(double2) * (size_t)(m1 * cols + m1 / 2);
    const size_t lds_cols_fwd = lds_cols + sizeof(double2) * fs;
    const int64_t rp = int64_t(1) << a.lgr;
    const size_t lds_rows = sizeof(double2) * ((size_t)(2 * rp * m2 + m2 / 2) + fs);
    const int64_t row_groups = pairs * ((m1 / 2 + 1 + rp - 1) / rp);
    hipLaunchKernelGGL((fft_cols_fwd_kernel<kTile, kRagged>), grid(col_groups), dim3(kTThreads),
                       lds_cols_fwd, s, a);
    hipLaunchKernelGGL((fft_rows_kernel<kTile, kRagged>), grid(row_groups), dim3(kTThreads),
                       lds_rows, s, a);
    hipLaunchKernelGGL((fft_cols_inv_kernel<kTile, kRagged>), grid(col_groups), dim3(kTThreads),
                       lds_cols, s, a);
}

// Complex fp64 entries of the twiddle tables of one transform of 2^lg points.
int64_t twiddle_count_of(int lg) {
    int32_t m1, m2, cols;
    fft_geometry(lg, &m1, &m2, &cols);
    if (m2 == 1) return (int64_t)m1 / 2;
    return m1 / 2 + m2 / 2 + m2 + m1;
}

}  // namespace

// Complex fp64 entries of the twiddle tables of a plan (a ragged plan: those
// of every length class, one after another).
int64_t fft_twiddle_count(const Plan& p) {
    if (!p.fft_ragged)
        return twiddle_count_of(p.fft_log2) + (p.fft_wrap ? twiddle_count_of(p.fft_wrap_log2) : 0);
    int64_t total = 0;
    for (int lg = kFftMinLog2; lg <= p.fft_log2; ++lg) total += twiddle_count_of(lg);
    return total;
}

// int32 entries of the length-class buffers of a plan.
int64_t fft_class_ints(const Plan& p) {
    return p.fft_ragged ? 2 * p.fft_pairs + kFftClasses + 1 : 0;
}

namespace {

// Twiddle tables of the geometry in `a`, written at `tw`.
void launch_twiddles(const FftArgs& a, double2* tw, hipStream_t s) {
    const int64_t count = twiddle_count_of(a.lg);
    int64_t tg = (count + 255) / 256;
    if (tg > 1024) tg = 1024;
    if (a.lg2 == 0) {
        hipLaunchKernelGGL(fft_twiddle_kernel, dim3((unsigned)tg), dim3(256), 0, s, tw, a.lg, 1,
                           a.lg, 0, (int64_t)0, (int64_t)0, (int64_t)0);
    } else {
        const int64_t m1 = int64_t(1) << a.lg1, m2 = int64_t(1) << a.lg2;
        hipLaunchKernelGGL(fft_twiddle_kernel, dim3((unsigned)tg), dim3(256), 0, s, tw, a.lg1,
                           a.lg2, a.lg, a.lg2, m2 / 2, m2, m1);
    }
}

template <int kTile>
void launch_spectrum(const Plan& p, const FftArgs& a, hipStream_t s) {
    if (p.fft_m2 == 1) {
        const size_t lds = sizeof(double2) * (size_t)p.fft_len;
        hipLaunchKernelGGL(spec_single_kernel<kTile>, dim3((unsigned)p.fft_pairs), dim3(kTThreads),
                           lds, s, a);
        return;
    }
    const int64_t col_groups = p.fft_pairs * (p.fft_m2 / p.fft_cols);
    const size_t lds_cols = sizeof(double2) * ((size_t)p.fft_m1 * p.fft_cols + p.fft_m1 / 2 +
                                               (four_step_in_lds(a.lg1, a.lg2)
                                                    ? (size_t)(p.fft_m1 + p.fft_m2) : 0));
    const int64_t rp = int64_t(1) << a.lgr;
    const size_t lds_rows = sizeof(double2) * 2 * rp * (size_t)p.fft_m2;
    const int64_t row_groups = p.fft_pairs * ((p.fft_m1 / 2 + 1 + rp - 1) / rp);
    hipLaunchKernelGGL((fft_cols_fwd_kernel<kTile, false>), dim3((unsigned)col_groups),
                       dim3(kTThreads), lds_cols, s, a);
    hipLaunchKernelGGL(spec_rows_kernel<kTile>, dim3((unsigned)row_groups), dim3(kTThreads),
                       lds_rows, s, a);
}

}  // namespace

hipError_t launch_spectral(const Plan& p, const Weights& w, const float* x, const double* fstat,
                           double* tw, double* z, double* amp, double c_peak, int32_t k_max,
                           gpoeo_pd_spectral_result* out, hipStream_t s) {
    FftArgs a = args_of(p, x, const_cast<double*>(fstat), nullptr, tw, z, nullptr);
    a.amp = amp;
    launch_twiddles(a, reinterpret_cast<double2*>(tw), s);
    if (fft_tile_log2(a.lg) == kFftSmallTileLog2)
        launch_spectrum<kFftSmallTileLog2>(p, a, s);
    else
        launch_spectrum<kFftTileLog2>(p, a, s);
    SpecSelArgs sa;
    sa.amp = amp;
    sa.fstat = fstat;
    sa.out = out;
    sa.seqs = a.seqs;
    sa.half = p.fft_len / 2 + 1;
    sa.len = p.fft_len;
    sa.num_channels = p.num_channels;
    sa.tmin = p.tmin;
    sa.tmax = p.tmax;
    sa.k_max = k_max;
    sa.lg = p.fft_log2;
    sa.c_peak = c_peak;
    if (sa.half > 16384)   // long spectra: more of each window's bins in flight
        hipLaunchKernelGGL(spec_select_kernel<1024>, dim3((unsigned)p.num_windows), dim3(1024), 0,
                           s, sa, w);
    else
        hipLaunchKernelGGL(spec_select_kernel<kThreads>, dim3((unsigned)p.num_windows),
                           dim3(kThreads), 0, s, sa, w);
    return hipGetLastError();
}

namespace {

// The wrap term of every sequence into `wrap` ([S][M]): head and tail
// transforms (column kernels on the segments), the cross spectrum and its
// inverse rows, then the inverse columns.  Twiddles of the 2^lgw geometry at
// `tw`.
template <int kTile>
void launch_wrap(const Plan& p, FftArgs aw, double2* tw, double2* zw, double* wrap,
                 hipStream_t s) {
    const int64_t lw = int64_t(1) << p.fft_wrap_log2;
    aw.tw = tw;
    aw.zstride = lw;
    aw.len = lw;
    launch_twiddles(aw, tw, s);
    const int64_t m1 = int64_t(1) << aw.lg1, m2 = int64_t(1) << aw.lg2, cols = int64_t(1) << aw.lgc;
    const int64_t col_groups = p.fft_pairs * (m2 / cols);
    const size_t fs = four_step_in_lds(aw.lg1, aw.lg2) ? (size_t)(m1 + m2) : 0;
    const size_t lds_cols = sizeof(double2) * (size_t)(m1 * cols + m1 / 2);
    const size_t lds_cols_fwd = lds_cols + sizeof(double2) * fs;
    aw.seg_len = p.fft_wrap_m;
    aw.seg_start = 0;                                  // heads
    aw.z = zw;
    hipLaunchKernelGGL((fft_cols_fwd_kernel<kTile, false>), dim3((unsigned)col_groups),
                       dim3(kTThreads), lds_cols_fwd, s, aw);
    aw.seg_start = p.n - p.fft_wrap_m;                 // tails
    aw.z = zw + p.fft_pairs * lw;
    hipLaunchKernelGGL((fft_cols_fwd_kernel<kTile, false>), dim3((unsigned)col_groups),
                       dim3(kTThreads), lds_cols_fwd, s, aw);
    aw.seg_len = 0;
    aw.z = zw;
    // a row pair holds four rows of m2 points: its two rows in each transform
    const int rows_tile = 4 * m2 <= (int64_t(1) << kFftSmallTileLog2) ? kFftSmallTileLog2
                                                                       : kFftTileLog2;
    aw.lgr = rows_tile - 2 - aw.lg2;
    if (aw.lgr > aw.lg1 - 1) aw.lgr = aw.lg1 - 1;
    const int64_t rp = int64_t(1) << aw.lgr;
    const int64_t row_groups = p.fft_pairs * ((m1 / 2 + 1 + rp - 1) / rp);
    const size_t lds_rows = sizeof(double2) * (size_t)(4 * rp * m2 + m2 / 2);
    if (rows_tile == kFftSmallTileLog2)
        hipLaunchKernelGGL((fft_wrap_rows_kernel<kFftSmallTileLog2>), dim3((unsigned)row_groups),
                           dim3(kTThreads), lds_rows, s, aw, p.fft_pairs * lw);
    else
        hipLaunchKernelGGL((fft_wrap_rows_kernel<kFftTileLog2>), dim3((unsigned)row_groups),
                           dim3(kTThreads), lds_rows, s, aw, p.fft_pairs * lw);
    aw.wout = wrap;
    aw.wm = p.fft_wrap_m;
    hipLaunchKernelGGL((fft_cols_inv_kernel<kTile, false>), dim3((unsigned)col_groups),
                       dim3(kTThreads), lds_cols, s, aw);
}

}  // namespace

hipError_t launch_fft_scores(const Plan& p, const float* x, double* fstat, double* edge,
                             double* tw, double* z, double* part, int32_t* cls, double* zw,
                             double* wrap, double* s64, float* scores, float w0,
                             hipStream_t s) {
    FftArgs a = args_of(p, x, fstat, edge, tw, z, part);
    double2* const tw2 = reinterpret_cast<double2*>(tw);
    if (fft_fused_finalize(p, scores != nullptr)) {
        a.s64 = s64;
        a.scores = scores;
        a.w0 = w0;
    }
    if (!p.fft_ragged) {
        launch_twiddles(a, tw2, s);
        hipLaunchKernelGGL(fft_edge_kernel, dim3((unsigned)(2 * a.seqs)), dim3(kThreads), 0, s, a);
        if (p.fft_wrap) {
            FftArgs aw = a;
            set_geometry(aw, p.fft_wrap_log2);
            double2* const tww = tw2 + twiddle_count_of(p.fft_log2);
            double2* const zw2 = reinterpret_cast<double2*>(zw);
            if (fft_tile_log2(p.fft_wrap_log2) == kFftSmallTileLog2)
                launch_wrap<kFftSmallTileLog2>(p, aw, tww, zw2, wrap, s);
            else
                launch_wrap<kFftTileLog2>(p, aw, tww, zw2, wrap, s);
            a.wrap = wrap;
            a.wrap_w = p.fft_len - p.n;
            a.wm = p.fft_wrap_m;
        }
        if (fft_tile_log2(a.lg) == kFftSmallTileLog2)
            launch_transforms<kFftSmallTileLog2, false>(a, p.fft_pairs, s);
        else
            launch_transforms<kFftTileLog2, false>(a, p.fft_pairs, s);
        return hipGetLastError();
    }
    // ragged: classify the pairs, then every length class at its own length
    ClassArgs ca;
    ca.pair_lg = cls;
    ca.list = cls + p.fft_pairs;
    ca.bounds = cls + 2 * p.fft_pairs;
    ca.pairs = p.fft_pairs;
    ca.seqs = a.seqs;
    ca.n_all = p.n;
    ca.num_channels = p.num_channels;
    ca.tmax = p.tmax;
    ca.lg_max = p.fft_log2;
    ca.tab = p.table;
    hipLaunchKernelGGL(fft_classify_kernel, dim3(1), dim3(kClassThreads), 0, s, ca);
    hipLaunchKernelGGL(fft_edge_kernel, dim3((unsigned)(2 * a.seqs)), dim3(kThreads), 0, s, a);
    int64_t tw_off = 0;
    for (int lg = kFftMinLog2; lg <= p.fft_log2; ++lg) {
        FftArgs ac = a;
        set_geometry(ac, lg);
        ac.tw = tw2 + tw_off;
        ac.list = ca.list;
        ac.bounds = ca.bounds;
        ac.cls = lg;
        launch_twiddles(ac, tw2 + tw_off, s);
        if (fft_tile_log2(lg) == kFftSmallTileLog2)
            launch_transforms<kFftSmallTileLog2, true>(ac, p.fft_pairs, s);
        else
            launch_transforms<kFftTileLog2, true>(ac, p.fft_pairs, s);
        tw_off += twiddle_count_of(lg);
    }
    return hipGetLastError();
}

hipError_t launch_fft_fixup(const Plan& p, const Weights& w, const float* x, const double* fstat,
                            const int32_t* cls, double* s64, float* scores,
                            const SelectBuffers& sb, hipStream_t s) {
    FixArgs a;
    a.x = x;
    a.fstat = fstat;
    a.s64 = s64;
    a.scores = scores;
    a.tier1 = sb.tier1;
    a.state = sb.state;
    a.seqs = p.num_windows * (int64_t)p.num_channels;
    a.n_all = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    a.tmin = p.tmin;
    a.tmax = p.tmax;
    a.lags = p.lags;
    a.words = p.bitmap_words;
    a.lg = p.fft_log2;
    a.tau0 = kFftRelBound;
    a.tab = p.table;
    a.pair_lg = p.fft_ragged ? cls : nullptr;
    a.wrap_lg = p.fft_wrap ? p.fft_wrap_log2 : -1;
    hipLaunchKernelGGL(fft_fixup_kernel, dim3((unsigned)p.num_windows), dim3(kThreads), 0, s, a,
                       w);
    return hipGetLastError();
}

}  // namespace gpoeo
