// Lag scores from an integer cross-correlation on the matrix cores
// (GPOEO_PD_MFMA_SCORES).
//
// The score of Algorithm 2's point-wise reading, D(T) = sum_{i < N-T}
// (y_i - y_{i+T})^2, equals E1(T) + E2(T) - 2 r(T) with r(T) = sum_i y_i y_{i+T}
// and the energies E1, E2 of the first N-T and the last N-T samples.  Each
// (window, channel) sequence is centred by c = its mean rounded to fp32 and
// scaled by 2^s into integers X_i = rint((x_i - c) 2^s), |X_i| < 2^30.  When
// every x_i - c is a multiple of 2^-s (all of a sequence's samples within a
// few binades, as sampled power is) the X_i represent the samples exactly;
// otherwise the rounding is bounded below.  X splits into four balanced base-256
// digits d_p in [-128, 127], X = sum_p 256^p d_p, and the cross term is the sum
// over digit pairs of 256^(p+q) sum_i d_p(i) d_q(i+T), exact int8 products
// accumulated exactly in int32 by v_mfma_i32_32x32x32_i8.  The three pairs of
// least weight, p + q <= 1, are left out: per sample pair they add at most
// 2^14 + 2 * 256 * 2^14 to a product of up to 2^60, so the cross term they
// drop is within 8404992 (N - T) of r(T), and the fix-up's bound includes it.
//
// Tile of one wavefront: 1024 lags T0 + 32 b + a (a, b < 32) over 32-sample
// steps i0: A[a][k] = d_p(i0 - a + k), B[k][b] = d_q(i0 + T0 + 32 b + k), so
// (A B)[a][b] sums the products of samples i = i0 - a + k and i + T.  Zero
// padding around each digit plane makes every read in range and every pair
// outside [0, N) contribute nothing, so the steps i0 = 0, 32, ... cover each
// lag's pairs exactly once.  The 13 digit-pair products go to 5 shift groups
// p + q = 2 .. 6; every 512 steps the groups are added, scaled by 256^(p+q),
// into fp64.
//
// The fix-up re-scores in fp64 every lag whose error bound (rounding of the
// fp64 sums, the digit pairs left out, and the quantisation of inexact
// sequences) is not within half the
// selection's tier-0 width of its score.
#include <cmath>

#include "exact.h"
#include "internal.h"

namespace gpoeo {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kXcds = 8;   // MI355X: workgroups are dealt to its 8 XCDs in turn
// Shift groups p + q = 2 .. 6 of the 13 digit-pair products kept, and the most
// the three left out (p + q <= 1) add to one sample pair's product, 128^2 (1 + 2 * 256).
constexpr int kGroups = 5;
constexpr double kDroppedPerPair = 8404992.0;
constexpr int kEdgeTile = 4096;
constexpr int kEdgePer = kEdgeTile / kThreads;
constexpr int kEdgeWaves = kThreads / kWave;

struct MfmaArgs {
    const float* x;
    double* qstat;       // [S][4]: centre c, scale exponent s, exact (1 or 0), E = sum X^2
    int8_t* dig;         // [S][4][plane]: digit p of sample i at p * plane + kMfmaPadL + i
    double* edge;        // [S][2][tmax + 1]: head and tail sums of X^2
    double* part;        // [S][lags]: D(T) (unless fused)
    double* rpart;       // chunked tiles: [S][chunks][tiles * 1024] cross terms from lag t0 on
    double* s64;         // fused finalisation (one channel): S(T)
    float* scores;
    float w0;
    int64_t seqs, n, window_stride, channel_stride, plane;
    int32_t num_channels, tmin, tmax, lags, t0, tiles, chunks;
    int64_t chunk_steps;
    WindowTable tab;     // per-window offsets, lengths and Tmax (rolling suffixes), or null
};

__device__ __forceinline__ const float* seq_ptr(const MfmaArgs& a, int64_t s) {
    return a.x + table_off(a.tab, s / a.num_channels, a.window_stride) +
           (s % a.num_channels) * a.channel_stride;
}
// samples of sequence s (0: an empty slot of a window table) and its largest lag
__device__ __forceinline__ int64_t seq_n(const MfmaArgs& a, int64_t s) {
    return table_n(a.tab, s / a.num_channels, a.n);
}
__device__ __forceinline__ int64_t seq_tmax(const MfmaArgs& a, int64_t s) {
    return min((int64_t)table_tmax(a.tab, s / a.num_channels, a.tmax), (int64_t)a.tmax);
}

// The integer sample of x under centre c and scale 2^s (the same expression in
// every kernel, so all of them see the same X).
__device__ __forceinline__ double quantised(float x, double c, double scale) {
    return rint(((double)x - c) * scale);
}

// D(T) = (E - tail(T)) + (E - head(T)) - 2 r(T), scaled back by 2^-2s, into
// part, or with one channel S(T) = w0 D / (N - T) into s64 (and scores), with
// the finalisation's own operations in its order.
__device__ __forceinline__ void write_d(const MfmaArgs& a, int64_t s, int64_t n, int64_t t,
                                        double r) {
    const double e = a.qstat[4 * s + 3];
    const int sc = (int)a.qstat[4 * s + 1];
    const double* __restrict__ ed = a.edge + s * 2 * ((int64_t)a.tmax + 1);
    const double d = ((e - ed[a.tmax + 1 + t]) + (e - ed[t])) - 2.0 * r;
    const double dy = ldexp(d, -2 * sc);
    const int64_t k = s * a.lags + (t - a.tmin);
    if (a.s64) {
        const double v = 0.0 + (double)a.w0 * (dy / (double)(n - t));
        a.s64[k] = v;
        if (a.scores) a.scores[k] = (float)v;
    } else {
        a.part[k] = dy;
    }
}

__device__ double block_sum(double v, double* red) {
    for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_down(v, o);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    double r = 0.0;
    for (int w = 0; w < kThreads / kWave; ++w) r += red[w];
    return r;
}

__device__ float block_min(float v, float* red) {
    for (int o = kWave / 2; o > 0; o >>= 1) v = fminf(v, __shfl_down(v, o));
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float r = red[0];
    for (int w = 1; w < kThreads / kWave; ++w) r = fminf(r, red[w]);
    return r;
}

// One workgroup per sequence.  Pass 1: mean, smallest and largest sample.
// Pass 2: X_i, its digits, E = sum X_i^2, and whether every X_i 2^-s equals
// x_i - c exactly.  Also zeroes the padding of the four digit planes (the
// plane length and kMfmaPadL are multiples of 4 bytes, so are its stores).
__global__ __launch_bounds__(kThreads) void mfma_prep_kernel(MfmaArgs a) {
    __shared__ double red[kThreads / kWave];
    __shared__ float redf[kThreads / kWave];
    const int64_t s = blockIdx.x;
    const float* __restrict__ xs = seq_ptr(a, s);
    const int64_t n = seq_n(a, s);
    if (n == 0) {   // an empty slot: nothing reads its planes
        if (threadIdx.x == 0) {
            a.qstat[4 * s] = a.qstat[4 * s + 1] = a.qstat[4 * s + 3] = 0.0;
            a.qstat[4 * s + 2] = 1.0;
        }
        return;
    }
    // Each thread visits i = tid, tid + kThreads, ... in order; the samples of
    // kPrepBatch consecutive visits are loaded together (all in flight).
    constexpr int kPrepBatch = 8;
    double sum = 0.0;
    float mn = INFINITY, mx = -INFINITY;
    int64_t i1 = threadIdx.x;
    for (; i1 + (kPrepBatch - 1) * kThreads < n; i1 += kPrepBatch * kThreads) {
        float v[kPrepBatch];
#pragma unroll
        for (int r = 0; r < kPrepBatch; ++r) v[r] = xs[i1 + r * kThreads];
#pragma unroll
        for (int r = 0; r < kPrepBatch; ++r) {
            sum += (double)v[r];
            mn = fminf(mn, v[r]);
            mx = fmaxf(mx, v[r]);
        }
    }
    for (; i1 < n; i1 += kThreads) {
        const float v = xs[i1];
        sum += (double)v;
        mn = fminf(mn, v);
        mx = fmaxf(mx, v);
    }
    const double mean = block_sum(sum, red) / (double)n;
    mn = block_min(mn, redf);
    mx = -block_min(-mx, redf);
    const double c = (double)(float)mean;
    const double dev = fmax((double)mx - c, c - (double)mn);   // differences of fp32 values: exact
    int e = 0;
    if (dev > 0.0) frexp(dev, &e);                             // dev < 2^e
    const int sc = 30 - e;                                     // |X| <= dev 2^sc < 2^30
    const double scale = ldexp(1.0, sc);
    int8_t* __restrict__ d0 = a.dig + s * 4 * a.plane + kMfmaPadL;
    double ex = 0.0;
    int exact = 1;
    // four consecutive samples per thread and step: one 32-bit store per digit
    // plane (samples past N, in the padding, get zero digits)
    const int64_t n4 = (n + 3) & ~int64_t(3);
    // the samples of two consecutive steps of a thread are loaded together
    // (zeros past N, which no step below uses)
    float nxt[4];
    auto load4 = [&](int64_t i, float (&v)[4]) {
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = i + k < n ? xs[i + k] : 0.0f;
    };
    if (4 * (int64_t)threadIdx.x < n4) load4(4 * (int64_t)threadIdx.x, nxt);
    for (int64_t i = 4 * (int64_t)threadIdx.x; i < n4; i += 4 * kThreads) {
        float cur[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) cur[k] = nxt[k];
        if (i + 4 * kThreads < n4) load4(i + 4 * kThreads, nxt);
        uint32_t word[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (i + k >= n) break;
            const double xv = (double)cur[k];
            const double y = xv - c;
            const double bb = y - xv;                          // two-sum error of xv + (-c)
            const double err = (xv - (y - bb)) + (-c - bb);
            const double t = y * scale;
            const double q = rint(t);
            exact &= (err == 0.0 && q == t) ? 1 : 0;
            ex += q * q;
            const int32_t v = (int32_t)q;                      // balanced base-256 digits
            const int32_t g0 = (int32_t)(int8_t)(v & 0xff);
            const int32_t r1 = (v - g0) >> 8;
            const int32_t g1 = (int32_t)(int8_t)(r1 & 0xff);
            const int32_t r2 = (r1 - g1) >> 8;
            const int32_t g2 = (int32_t)(int8_t)(r2 & 0xff);
            const int32_t g3 = (r2 - g2) >> 8;
            word[0] |= (uint32_t)(g0 & 0xff) << (8 * k);
            word[1] |= (uint32_t)(g1 & 0xff) << (8 * k);
            word[2] |= (uint32_t)(g2 & 0xff) << (8 * k);
            word[3] |= (uint32_t)(g3 & 0xff) << (8 * k);
        }
#pragma unroll
        for (int p = 0; p < 4; ++p) *reinterpret_cast<uint32_t*>(d0 + p * a.plane + i) = word[p];
    }
    // the rest of the padding, 4 bytes a store: [-kMfmaPadL, 0) and the kMfmaPadR
    // bytes after the samples, all that the tile loop reads of a window of n
    // samples (a window of a table may be shorter than the plane)
    const int64_t pl = kMfmaPadL / 4;
    const int64_t pr = min(a.plane - kMfmaPadL - n4, (int64_t)kMfmaPadR) / 4;
    for (int64_t k = threadIdx.x; k < 4 * (pl + pr); k += kThreads) {
        const int64_t p = k / (pl + pr), j = k % (pl + pr);
        const int64_t i = j < pl ? 4 * (j - pl) : n4 + 4 * (j - pl);
        *reinterpret_cast<uint32_t*>(d0 + p * a.plane + i) = 0u;
    }
    const double etot = block_sum(ex, red);
    const double ex_all = block_sum(exact ? 0.0 : 1.0, red);
    if (threadIdx.x == 0) {
        a.qstat[4 * s] = c;
        a.qstat[4 * s + 1] = (double)sc;
        a.qstat[4 * s + 2] = ex_all == 0.0 ? 1.0 : 0.0;
        a.qstat[4 * s + 3] = etot;
    }
}

// Head and tail sums of X^2 for T = 0 .. Tmax, one workgroup per (sequence,
// side): tiles of 4096 terms staged in LDS, per-thread runs of 16, a scan of
// the thread totals, coalesced stores.
__device__ __forceinline__ int edge_slot(int k) { return k + (k >> 4); }

__global__ __launch_bounds__(kThreads) void mfma_edge_kernel(MfmaArgs a) {
    __shared__ double tile[kEdgeTile + kEdgeTile / 16];
    __shared__ double wsum[kEdgeWaves];
    const int64_t s = blockIdx.x >> 1;
    const int side = blockIdx.x & 1;
    const float* __restrict__ p = seq_ptr(a, s);
    const int64_t n = seq_n(a, s);
    const double c = a.qstat[4 * s];
    const double scale = ldexp(1.0, (int)a.qstat[4 * s + 1]);
    double* __restrict__ out = a.edge + (s * 2 + side) * ((int64_t)a.tmax + 1);
    // T = 0 .. this window's largest lag (nothing for an empty slot)
    const int64_t span = n > 0 ? seq_tmax(a, s) + 1 : 1;
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    if (threadIdx.x == 0) out[0] = 0.0;
    double carry = 0.0;
    // the next tile's samples are loaded while this tile is scanned
    float nxt[kEdgePer];
    auto load_tile = [&](int64_t k0, float (&v)[kEdgePer]) {
#pragma unroll
        for (int r = 0; r < kEdgePer; ++r) {
            const int64_t kk = k0 + (int)threadIdx.x + r * kThreads;
            v[r] = kk < span - 1 ? p[side == 0 ? kk : n - 1 - kk] : 0.0f;
        }
    };
    if (span - 1 > 0) load_tile(0, nxt);
    for (int64_t k0 = 0; k0 < span - 1; k0 += kEdgeTile) {
        {
            float v[kEdgePer];
#pragma unroll
            for (int r = 0; r < kEdgePer; ++r) v[r] = nxt[r];
            if (k0 + kEdgeTile < span - 1) load_tile(k0 + kEdgeTile, nxt);
#pragma unroll
            for (int r = 0; r < kEdgePer; ++r) {
                const int k = (int)threadIdx.x + r * kThreads;
                const double q = k0 + k < span - 1 ? quantised(v[r], c, scale) : 0.0;
                tile[edge_slot(k)] = q * q;
            }
        }
        __syncthreads();
        double part = 0.0;
        for (int r = 0; r < kEdgePer; ++r) part += tile[edge_slot((int)threadIdx.x * kEdgePer + r)];
        double inc = part;
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
        run += inc - part;
        for (int r = 0; r < kEdgePer; ++r) {
            const int k = (int)threadIdx.x * kEdgePer + r;
            run += tile[edge_slot(k)];
            tile[edge_slot(k)] = run;
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

// The workgroup's four tiles read the same A rows and B ranges that overlap
// from one step to the next, so a workgroup stages its digits in LDS a stage
// of kStageSteps steps at a time: per plane, an A block of the samples
// [i0s - 64, i0s + 32 kStageSteps + 96) and a B block of the samples
// [i0s + T0', i0s + T0' + 32 (kStageSteps + 1) + 3072 + 1024), where i0s is the
// stage's first sample and T0' the first lag T0 of the workgroup's first tile
// rounded down to a multiple of 16, so that every staged chunk is 16 aligned
// bytes of a plane.  Samples at or past N are staged as zeros.  The B block is stored as two
// halves, the first and the second 16 bytes of every 32-byte row, so that the
// lanes of a B read (one 16-byte half of 32 consecutive rows) cover 512
// contiguous bytes, free of bank conflicts.
//
// The staging goes straight from memory into LDS (global_load_lds_dwordx4:
// lane l of one instruction writes the 16 bytes at LDS base + 16 l), into the
// other of two stage buffers while this stage's products run; the stage ends
// with a wait for those loads and one barrier.  No staging passes through
// registers, so r(T) stays in registers between flushes, and two workgroups
// share a CU (68 KB of LDS and at most 256 registers a lane each): one wave's
// operand reads overlap the other's products.
constexpr int kStageSteps = 64;
constexpr int kStageA = 32 * kStageSteps + 160;                  // 2208 bytes
constexpr int kStageB = 32 * (kStageSteps + 1) + 4 * kMfmaTileLags;   // 6176 bytes
constexpr int kStageHalf = kStageB / 2;                          // 3088 bytes
constexpr int kStagePlane = kStageA + kStageB;
constexpr int kStageChunks = 4 * kStagePlane / 16;               // 2096 chunks of 16 bytes
constexpr int kStageLoads = (kStageChunks + kWave - 1) / kWave;  // 33 wave-wide loads a stage
constexpr int kStageBytes = kStageLoads * kWave * 16;            // 33792 bytes
static_assert(kStageA % 16 == 0 && kStageB % 32 == 0 && kStageHalf % 16 == 0,
              "16-byte staging chunks, 32-byte B rows");
static_assert(kMfmaFlush % kStageSteps == 0 && kStageSteps % 2 == 0, "stage and flush cadence");

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

// One wavefront per (sequence, tile of 1024 lags, chunk of sample steps); four
// tiles of a sequence per workgroup, sharing the staged digits.  With one chunk
// the wave forms D(T) itself; with several it writes its partial cross terms
// for the combination.
template <bool kChunked>
__global__ __launch_bounds__(kThreads, 2) void mfma_xcorr_kernel(MfmaArgs a) {
    __shared__ __attribute__((aligned(16))) int8_t stage_buf[2 * kStageBytes];
    // the wave index is uniform over the wave: said so, the tile, its step
    // count and the loop control stay scalar
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    // Workgroups go to the 8 XCDs in turn, workgroup b to XCD b % 8.  Every
    // workgroup of sequence s = 8 u + v takes an index with b % 8 == (u + v) % 8:
    // the sequence's digits stay in one XCD's L2, and sequences of any stride
    // (the suffix slots of rolling detection, whose lengths differ) rotate
    // over all XCDs.  The grid is padded to a multiple of 8 sequences.
    const int groups = (a.tiles + 3) / 4;
    const int64_t rest = blockIdx.x / kXcds;
    const int chunk = kChunked ? (int)(rest % a.chunks) : 0;
    const int64_t gi = kChunked ? rest / a.chunks : rest;
    const int64_t su = gi / groups;
    const int64_t s = su * kXcds + (int64_t)((blockIdx.x - su) & (kXcds - 1));
    if (s >= a.seqs) return;   // padding of the grid
    const int tile0 = (int)(gi % groups) * 4;
    const int tile = tile0 + wave;
    const int64_t tg0 = (int64_t)a.t0 + (int64_t)tile0 * kMfmaTileLags;   // the workgroup's first lag
    const int32_t t0 = a.t0 + tile * kMfmaTileLags;
    const int64_t n = seq_n(a, s);
    const int64_t tm = seq_tmax(a, s);
    if (n == 0 || tg0 > tm) return;   // the whole workgroup: no lag of this window in its tiles
    const bool active = tile < a.tiles && t0 <= tm;
    // Steps while some pair (i, i + T) of a tile has i + T < N, rounded up to
    // an even count (a step past that reads only zeros); the chunk's share of
    // them, from its first step kbeg.
    auto steps_of = [&](int64_t first_lag) {
        const int64_t all = ((n - first_lag + 62) / 32 + 1) & ~int64_t(1);
        const int64_t kbeg = kChunked ? min(all, (int64_t)chunk * a.chunk_steps) : 0;
        return kChunked ? min(all - kbeg, a.chunk_steps) : all;
    };
    const int64_t kbeg = kChunked ? (int64_t)chunk * a.chunk_steps : 0;
    const int64_t wg_steps = max((int64_t)0, steps_of(tg0));   // the first tile has the most
    const int64_t my_steps = active ? max((int64_t)0, steps_of(t0)) : 0;
    const int64_t stages = (wg_steps + kStageSteps - 1) / kStageSteps;
    const int8_t* __restrict__ seq = a.dig + s * 4 * a.plane + kMfmaPadL;
    // The steps' samples are moved dl = T0 - T0' (0 .. 15) earlier than i0, so
    // that B starts on the aligned T0': step i0 pairs, for lag T0 + 32 b + a,
    // the samples i = i0 - dl - a + k and i + T (k < 32).  Successive steps
    // still cover every i exactly once, from i = -dl - a <= 0 on.
    const int dl = (int)(tg0 & 15);

    // Staging: the 16-byte chunk c of a stage lands at byte 16 c of its buffer.
    // Per plane p, chunks j < kStageA / 16 are the A block; then the B rows'
    // first halves, then their second halves.  A chunk that starts at or past
    // N is read from the zero padding before the plane's first sample, as is
    // every slot past the last chunk.  Wave w issues the loads w, w + 4, ...
    auto fetch = [&](int64_t st, int buf) {
        const int64_t i0s = 32 * (kbeg + st * kStageSteps);
        for (int r = wave; r < kStageLoads; r += kThreads / kWave) {
            const int c = r * kWave + lane;
            const int p = c / (kStagePlane / 16), j = c % (kStagePlane / 16);
            const int8_t* plane = seq + (int64_t)min(p, 3) * a.plane;
            int64_t i;
            if (j < kStageA / 16) {
                i = i0s - 64 + 16 * j;
            } else {
                const int jb = j - kStageA / 16;
                const int half = jb >= kStageHalf / 16 ? 1 : 0;
                i = i0s + (tg0 - dl) + 32 * (jb - half * (kStageHalf / 16)) + 16 * half;
            }
            const int8_t* src = (c < kStageChunks && i < n) ? plane + i : seq - 64;
            __builtin_amdgcn_global_load_lds((global_void*)src,
                                             (lds_void*)(stage_buf + buf * kStageBytes +
                                                         r * (kWave * 16)),
                                             16, 0, 0);
        }
    };
    // the stage's loads have landed, for every wave of the workgroup
    auto stage_barrier = [&]() {
        __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0); expcnt and lgkmcnt not waited on
        __syncthreads();
    };

    const int m = lane & 31, h = lane >> 5;
    const int off = (-dl - m) & 3;   // byte offset of this lane's A row within its first dword
    v16i acc[kGroups];   // acc[g] holds shift group p + q = g + 2
#pragma unroll
    for (int g = 0; g < kGroups; ++g) acc[g] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    // Per step, from the stage buffer: A row a = m, bytes i0 - dl - m + 16 h
    // .. + 15 (dword-aligned reads shifted into place); B column b = m, bytes
    // i0 + T0' + 32 m + 16 h .. + 15.
    uint32_t w0[4][5], w1[4][5];
    v4i b0[4], b1[4];
    auto load = [&](const int8_t* sb, uint32_t (&w)[4][5], v4i (&bq)[4], int k) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint32_t* src = reinterpret_cast<const uint32_t*>(
                sb + p * kStagePlane + 32 * k + 64 - dl - m + 16 * h - off);
#pragma unroll
            for (int e = 0; e < 5; ++e) w[p][e] = src[e];
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
            bq[q] = *reinterpret_cast<const v4i*>(sb + q * kStagePlane + kStageA + h * kStageHalf +
                                                  16 * (k + wave * (kMfmaTileLags / 32) + m));
    };
    auto step = [&](const uint32_t (&w)[4][5], const v4i (&bq)[4]) {
        v4i A[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            A[p][0] = (int)__builtin_amdgcn_alignbyte(w[p][1], w[p][0], off);
            A[p][1] = (int)__builtin_amdgcn_alignbyte(w[p][2], w[p][1], off);
            A[p][2] = (int)__builtin_amdgcn_alignbyte(w[p][3], w[p][2], off);
            A[p][3] = (int)__builtin_amdgcn_alignbyte(w[p][4], w[p][3], off);
        }
#pragma unroll
        for (int p = 0; p < 4; ++p)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (p + q >= 2)
                    acc[p + q - 2] =
                        __builtin_amdgcn_mfma_i32_32x32x32_i8(A[p], bq[q], acc[p + q - 2], 0, 0, 0);
    };
    // Every kMfmaFlush steps (each group sum stays below 2^31 over that many)
    // the shift groups are added, scaled by 256^(p+q), into r(T) in fp64,
    // which the lane holds in registers.  Register j of lane (m, h) holds row
    // 8 (j / 4) + 4 h + j % 4, column m: lag t0 + 32 m + row.
    double r[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) r[j] = 0.0;
    auto flush = [&]() {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
#pragma unroll
            for (int g = kGroups - 1; g >= 0; --g) r[j] += ldexp((double)acc[g][j], 8 * (g + 2));
        }
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
            acc[g] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    };

    if (stages > 0) fetch(0, 0);
    stage_barrier();
    for (int64_t st = 0; st < stages; ++st) {
        // the next stage's loads, into the other buffer (every wave has left
        // it behind at the last barrier), in flight while this one's products run
        if (st + 1 < stages) fetch(st + 1, (int)((st + 1) & 1));
        const int8_t* sb = stage_buf + (st & 1) * kStageBytes;
        // this wave's steps in the stage (none once its tile's run out)
        const int nk = (int)min((int64_t)kStageSteps, max((int64_t)0, my_steps - st * kStageSteps));
        // two operand sets: the reads of step k + 1 are in flight while the
        // products of step k run (nk is even)
        if (nk > 0) load(sb, w0, b0, 0);
        for (int k = 0; k < nk; k += 2) {
            load(sb, w1, b1, k + 1);
            step(w0, b0);
            if (k + 2 < nk) load(sb, w0, b0, k + 2);
            step(w1, b1);
        }
        if (active && ((st + 1) % (kMfmaFlush / kStageSteps) == 0 || st + 1 == stages)) flush();
        stage_barrier();
    }
    if (!active) return;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int row = 8 * (j >> 2) + 4 * h + (j & 3);
        const int64_t t = (int64_t)t0 + 32 * m + row;
        if (t < a.tmin || t > tm) continue;   // lags past a table window's own: left unwritten
        if (kChunked)   // the partials stay for the combination
            a.rpart[(s * a.chunks + chunk) * ((int64_t)a.tiles * kMfmaTileLags) + (t - a.t0)] = r[j];
        else
            write_d(a, s, n, t, r[j]);
    }
}

// Chunked tiles: r(T) as the sum of the chunks' partial cross terms in chunk
// order, then D(T) as above; one thread per (sequence, lag).
__global__ __launch_bounds__(kThreads) void mfma_combine_kernel(MfmaArgs a) {
    const int64_t lag_groups = ((int64_t)a.lags + kThreads - 1) / kThreads;
    const int64_t s = blockIdx.x / lag_groups;
    const int64_t n = seq_n(a, s);
    const int64_t tm = seq_tmax(a, s);
    const int64_t t = (int64_t)a.tmin + (int64_t)(blockIdx.x % lag_groups) * kThreads + threadIdx.x;
    if (n == 0 || t > tm) return;
    const int64_t tl = (int64_t)a.tiles * kMfmaTileLags;
    const double* __restrict__ rp = a.rpart + s * a.chunks * tl + (t - a.t0);
    double r = 0.0;
    for (int c = 0; c < a.chunks; ++c) r += rp[c * tl];
    write_d(a, s, n, t, r);
}

struct MfixArgs {
    const float* x;
    const double* qstat;
    double* s64;
    float* scores;
    uint32_t* tier1;
    WinState* state;
    int64_t n, window_stride, channel_stride;
    int32_t num_channels, tmin, tmax, lags, words, t0, chunks;
    double tau0;
    WindowTable tab;
};

// One workgroup per window.  Per channel (X units): the rounding of E and of
// the edge sums (each within gamma_{N+1} E), of the three operations forming
// D, and of the fp64 sum of the shift groups into r (5 additions per flush,
// over terms whose magnitudes sum to at most (N - T) 2^62 1.008, because a
// balanced four-digit X has sum_p 256^p |d_p| < 2^31 1.004) give R, lag-
// independent with N - T <= N.  An inexact sequence adds the quantisation:
// with |X_i - 2^s (x_i - c)| <= 1/2 + 2^-23, D_X - 2^2s D is at most
// 4 sqrt(m D_X) + 6 m over m = N - T pairs.  Every sequence adds the digit
// pairs left out of r, L = 2 * 8404992 m in D.  D_X is bounded through the
// computed score: w_c D_c <= m S + sum_c' w_c' (R_c' + L_c').  Lags whose total bound,
// divided by m, exceeds tau0 / 2 of the score (the other half covers the
// finalisation and the fp32 output) are re-scored by a wavefront in fp64 and
// marked tier 1; so is every score of exactly zero.
__global__ __launch_bounds__(kThreads) void mfma_fixup_kernel(MfixArgs a, Weights w) {
    __shared__ double rr[kMaxChannels], qa[kMaxChannels], qb[kMaxChannels], tr[kMaxChannels];
    __shared__ double total_r, total_t;
    const int64_t b = blockIdx.x;
    const int64_t n = table_n(a.tab, b, a.n);
    if (n == 0) return;   // an empty slot of a window table
    const int32_t tm = min(table_tmax(a.tab, b, a.tmax), a.tmax);
    const double u = 1.1102230246251565e-16;
    const double steps = (double)((n + 62) / 32);
    // flushes over all chunks, and the additions of the chunks' partial sums
    const double flushes = floor(steps / (double)kMfmaFlush) + 2.0 + (double)a.chunks;
    for (int32_t c = threadIdx.x; c < a.num_channels; c += kThreads) {
        const int64_t sq = b * a.num_channels + c;
        const double sc = a.qstat[4 * sq + 1];
        const double e = a.qstat[4 * sq + 3];
        const double round_x = u * (4.04 * ((double)n + 1.0) + 12.0) * e +
                               2.0 * (5.0 * flushes + (double)a.chunks) * u * 1.01 * (double)n *
                                   ldexp(1.008, 62);
        rr[c] = 1.01 * ldexp(round_x, -2 * (int)sc);
        tr[c] = 1.01 * ldexp(2.0 * kDroppedPerPair, -2 * (int)sc);   // per pair, times m
        const bool inexact = a.qstat[4 * sq + 2] == 0.0;
        qa[c] = inexact ? 1.01 * 4.0 * ldexp(1.0, -(int)sc) : 0.0;
        qb[c] = inexact ? 1.01 * 6.0 * ldexp(1.0, -2 * (int)sc) : 0.0;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double acc = 0.0, acct = 0.0;
        for (int32_t c = 0; c < a.num_channels; ++c) {
            acc += (double)w.w[c] * rr[c];
            acct += (double)w.w[c] * tr[c];
        }
        total_r = acc * (1.0 + 1e-12);
        total_t = acct * (1.0 + 1e-12);
    }
    __syncthreads();
    const double ar = total_r, at = total_t;
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
            const double m = (double)(n - t);
            const double v = vb[r];
            const double art = (ar + at * m) * (1.0 + 1e-12);   // all channels' R and left-out pairs
            double bound = art;
            for (int32_t c = 0; c < a.num_channels; ++c) {
                if (qa[c] == 0.0) continue;
                const double wc = (double)w.w[c];
                const double dup = (m * fmax(v, 0.0) * (1.0 + 1e-12) + art) / wc + rr[c] + tr[c] * m;
                bound += wc * (qa[c] * sqrt(m * dup) + qb[c] * m);
            }
            fix = !(bound * (1.0 + 1e-12) / m <= 0.5 * a.tau0 * v);
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

MfmaArgs args_of(const Plan& p, const float* x, double* qstat, int8_t* dig, double* edge,
                 double* rpart, double* part) {
    MfmaArgs a;
    a.x = x;
    a.qstat = qstat;
    a.dig = dig;
    a.edge = edge;
    a.part = part;
    a.rpart = rpart;
    a.s64 = nullptr;
    a.scores = nullptr;
    a.w0 = 1.0f;
    a.seqs = p.num_windows * (int64_t)p.num_channels;
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.plane = p.mfma_plane;
    a.num_channels = p.num_channels;
    a.tmin = p.tmin;
    a.tmax = p.tmax;
    a.lags = p.lags;
    a.t0 = p.mfma_t0;
    a.tiles = p.mfma_tiles;
    a.chunks = p.mfma_chunks;
    a.chunk_steps = p.mfma_chunk_steps;
    a.tab = p.table;
    return a;
}

}  // namespace

hipError_t launch_mfma_scores(const Plan& p, const float* x, double* qstat, int8_t* dig,
                              double* edge, double* rpart, double* part, double* s64,
                              float* scores, float w0, hipStream_t s) {
    MfmaArgs a = args_of(p, x, qstat, dig, edge, rpart, part);
    if (mfma_fused_finalize(p, scores != nullptr)) {
        a.s64 = s64;
        a.scores = scores;
        a.w0 = w0;
    }
    hipLaunchKernelGGL(mfma_prep_kernel, dim3((unsigned)a.seqs), dim3(kThreads), 0, s, a);
    hipLaunchKernelGGL(mfma_edge_kernel, dim3((unsigned)(2 * a.seqs)), dim3(kThreads), 0, s, a);
    const int64_t groups = (p.mfma_tiles + 3) / 4;
    const int64_t seqs8 = (a.seqs + kXcds - 1) / kXcds * kXcds;
    if (p.mfma_chunks == 1) {
        hipLaunchKernelGGL(mfma_xcorr_kernel<false>, dim3((unsigned)(seqs8 * groups)),
                           dim3(kThreads), 0, s, a);
    } else {
        hipLaunchKernelGGL(mfma_xcorr_kernel<true>,
                           dim3((unsigned)(seqs8 * groups * p.mfma_chunks)), dim3(kThreads), 0,
                           s, a);
        hipLaunchKernelGGL(mfma_combine_kernel,
                           dim3((unsigned)(a.seqs * ((p.lags + kThreads - 1) / kThreads))),
                           dim3(kThreads), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_mfma_fixup(const Plan& p, const Weights& w, const float* x,
                             const double* qstat, double* s64, float* scores,
                             const SelectBuffers& sb, hipStream_t s) {
    MfixArgs a;
    a.x = x;
    a.qstat = qstat;
    a.s64 = s64;
    a.scores = scores;
    a.tier1 = sb.tier1;
    a.state = sb.state;
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    a.tmin = p.tmin;
    a.tmax = p.tmax;
    a.lags = p.lags;
    a.words = p.bitmap_words;
    a.t0 = p.mfma_t0;
    a.tau0 = kScoreRelBound;
    a.chunks = p.mfma_chunks;
    a.tab = p.table;
    hipLaunchKernelGGL(mfma_fixup_kernel, dim3((unsigned)p.num_windows), dim3(kThreads), 0, s, a,
                       w);
    return hipGetLastError();
}

}  // namespace gpoeo
