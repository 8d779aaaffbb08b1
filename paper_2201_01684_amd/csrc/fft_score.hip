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
#include <cmath>

#include "internal.h"
#include "exact.h"

namespace gpoeo {
namespace {

constexpr int kThreads = 256;
constexpr int kLdsPoints = 4096;           // complex fp64 points per workgroup: 64 KiB
constexpr int kRegPoints = kLdsPoints / kThreads;

struct FftArgs {
    const float* x;
    double* fstat;             // [S][4]: mean, sum y^2, sum |y|, unused
    double* edge;              // [S][2][tmax + 1]: head and tail sums of y^2
    const double2* tw;         // twiddle tables
    double2* z;                // [pairs][len]
    double* part;              // [S][lags]: D(T)
    int64_t seqs;              // S = B * C
    int64_t n_all, window_stride, channel_stride;
    int64_t len;
    int64_t tw_a, tw_b, tw_lo, tw_hi;
    int32_t num_channels;
    int32_t tmin, tmax, lags;
    int32_t lg, lg1, lg2, lgc;
    WindowTable tab;
};

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

// Forward transform (exp(-2 pi i kn/L), L = 2^lg) of `cols` interleaved
// sequences s[i * cols + q], by decimation in frequency: natural order in,
// bit-reversed out.  tw[m] = exp(-2 pi i m / L), m < L/2.
__device__ void lds_fft_fwd(double2* s, int lg, int lgc, const double2* __restrict__ tw) {
    const int cols = 1 << lgc;
    const int nb = 1 << (lg - 1 + lgc);
    for (int st = lg - 1; st >= 0; --st) {
        const int h = 1 << st;
        for (int f = threadIdx.x; f < nb; f += kThreads) {
            const int q = f & (cols - 1);
            const int bf = f >> lgc;
            const int j = bf & (h - 1);
            const int i0 = ((bf >> st) << (st + 1)) + j;
            const int i1 = i0 + h;
            const double2 a = s[i0 * cols + q], b = s[i1 * cols + q];
            const double2 w = tw[j << (lg - 1 - st)];
            s[i0 * cols + q] = cadd(a, b);
            s[i1 * cols + q] = cmul(csub(a, b), w);
        }
        __syncthreads();
    }
}

// Inverse transform (exp(+2 pi i kn/L), no 1/L) by decimation in time:
// bit-reversed order in, natural out.
__device__ void lds_fft_inv(double2* s, int lg, int lgc, const double2* __restrict__ tw) {
    const int cols = 1 << lgc;
    const int nb = 1 << (lg - 1 + lgc);
    for (int st = 0; st < lg; ++st) {
        const int h = 1 << st;
        for (int f = threadIdx.x; f < nb; f += kThreads) {
            const int q = f & (cols - 1);
            const int bf = f >> lgc;
            const int j = bf & (h - 1);
            const int i0 = ((bf >> st) << (st + 1)) + j;
            const int i1 = i0 + h;
            const double2 a = s[i0 * cols + q];
            const double2 b = cmul_conj(s[i1 * cols + q], tw[j << (lg - 1 - st)]);
            s[i0 * cols + q] = cadd(a, b);
            s[i1 * cols + q] = csub(a, b);
        }
        __syncthreads();
    }
}

// W_L^e = exp(-2 pi i e / L) for e < L from two tables split at bit lg2.
__device__ __forceinline__ double2 twiddle(const FftArgs& a, int64_t e) {
    return cmul(a.tw[a.tw_hi + (e >> a.lg2)], a.tw[a.tw_lo + (e & ((int64_t(1) << a.lg2) - 1))]);
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
    double d = 0.0;
    if (n > 0 && t <= table_tmax(a.tab, b, a.tmax)) {
        const double r = ldexp(w, -(a.lg + 2));
        const double e = a.fstat[4 * s + 1];
        const double* ed = a.edge + s * 2 * (int64_t)(a.tmax + 1);
        d = ((e - ed[a.tmax + 1 + t]) + (e - ed[t])) - 2.0 * r;
    }
    a.part[s * a.lags + (t - a.tmin)] = d;
}

__device__ double block_sum(double v, double* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}

// Per sequence: the fp64 mean (the centring constant), sum y^2 and sum |y| of
// the centred samples, and the sums of y^2 over the first and the last T
// samples for T = 0..Tmax (each thread sums a contiguous stretch, then the
// stretch totals are added in thread order).
__global__ __launch_bounds__(kThreads) void fft_prep_kernel(FftArgs a) {
    __shared__ double red[kThreads];
    __shared__ double base[kThreads];
    const int64_t s = blockIdx.x;
    const int64_t b = s / a.num_channels;
    const int64_t c = s % a.num_channels;
    const int64_t n = table_n(a.tab, b, a.n_all);
    const float* __restrict__ p = a.x + table_off(a.tab, b, a.window_stride) + c * a.channel_stride;
    double sum = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += kThreads) sum += (double)p[i];
    const double mu = n > 0 ? block_sum(sum, red) / (double)n : 0.0;
    double e = 0.0, l1 = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += kThreads) {
        const double y = (double)p[i] - mu;
        e += y * y;
        l1 += fabs(y);
    }
    e = block_sum(e, red);
    l1 = block_sum(l1, red);
    if (threadIdx.x == 0) {
        a.fstat[4 * s] = mu;
        a.fstat[4 * s + 1] = e;
        a.fstat[4 * s + 2] = l1;
        a.fstat[4 * s + 3] = 0.0;
    }
    const int64_t span = (int64_t)a.tmax + 1;
    double* __restrict__ head = a.edge + s * 2 * span;
    double* __restrict__ tail = head + span;
    const int64_t per = (span + kThreads - 1) / kThreads;
    const int64_t lo = threadIdx.x * per;
    const int64_t hi = lo + per < span ? lo + per : span;
    for (int side = 0; side < 2; ++side) {
        // term k (k = 0..Tmax-1) of the running sum: y_k (head) or y_{n-1-k} (tail)
        auto term = [&](int64_t k) -> double {
            const int64_t i = side == 0 ? k : n - 1 - k;
            if (k >= n || i < 0) return 0.0;
            const double y = (double)p[i] - mu;
            return y * y;
        };
        double t = 0.0;
        for (int64_t k = lo; k < hi; ++k)
            if (k >= 1) t += term(k - 1);
        base[threadIdx.x] = t;
        __syncthreads();
        if (threadIdx.x == 0) {
            double run = 0.0;
            for (int k = 0; k < kThreads; ++k) {
                const double v = base[k];
                base[k] = run;
                run += v;
            }
        }
        __syncthreads();
        double* __restrict__ out = side == 0 ? head : tail;
        double run = base[threadIdx.x];
        for (int64_t k = lo; k < hi; ++k) {
            if (k >= 1) run += term(k - 1);
            out[k] = run;
        }
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
__global__ __launch_bounds__(kThreads) void fft_single_kernel(FftArgs a) {
    extern __shared__ double2 lds[];
    const int64_t pair = blockIdx.x;
    const Seq qa = seq_of(a, 2 * pair), qb = seq_of(a, 2 * pair + 1);
    const int lg = a.lg;
    const int len = 1 << lg;
    const double2* tw = a.tw + a.tw_a;
    for (int i = threadIdx.x; i < len; i += kThreads)
        lds[i] = make_double2(centred(qa, i), centred(qb, i));
    __syncthreads();
    lds_fft_fwd(lds, lg, 0, tw);
    double2 wv[kRegPoints];
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int pos = threadIdx.x + r * kThreads;
        if (pos < len) {
            const uint32_t k = bitrev(pos, lg);
            const uint32_t km = (len - k) & (len - 1);
            wv[r] = power_pair(lds[pos], lds[bitrev(km, lg)]);
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int pos = threadIdx.x + r * kThreads;
        if (pos < len) lds[pos] = wv[r];
    }
    __syncthreads();
    lds_fft_inv(lds, lg, 0, tw);
    for (int64_t t = a.tmin + threadIdx.x; t <= a.tmax; t += kThreads) {
        write_d(a, 2 * pair, t, lds[t].x);
        write_d(a, 2 * pair + 1, t, lds[t].y);
    }
}

// Split transform, step 1: column transforms (L1 points, stride L2) of
// 2^lgc neighbouring columns, then the twiddles W_L^(k1 n2).  Row p of the
// output holds frequency k1 = bitrev(p).
__global__ __launch_bounds__(kThreads) void fft_cols_fwd_kernel(FftArgs a) {
    extern __shared__ double2 lds[];
    const int64_t groups = int64_t(1) << (a.lg2 - a.lgc);
    const int64_t id = xcd_remap(blockIdx.x, gridDim.x);
    const int64_t pair = id / groups;
    const int64_t c0 = (id % groups) << a.lgc;
    const int cols = 1 << a.lgc;
    const int npts = (1 << a.lg1) * cols;
    const int64_t l2 = int64_t(1) << a.lg2;
    const Seq qa = seq_of(a, 2 * pair), qb = seq_of(a, 2 * pair + 1);
    for (int f = threadIdx.x; f < npts; f += kThreads) {
        const int64_t i = (int64_t)(f >> a.lgc) * l2 + c0 + (f & (cols - 1));
        lds[f] = make_double2(centred(qa, i), centred(qb, i));
    }
    __syncthreads();
    lds_fft_fwd(lds, a.lg1, a.lgc, a.tw + a.tw_a);
    double2* __restrict__ zp = a.z + pair * a.len;
    for (int f = threadIdx.x; f < npts; f += kThreads) {
        const int pos = f >> a.lgc;
        const int64_t n2 = c0 + (f & (cols - 1));
        const int64_t k1 = bitrev(pos, a.lg1);
        zp[pos * l2 + n2] = cmul(lds[f], twiddle(a, k1 * n2));
    }
}

// Split transform, step 2: row k1 and its mirror row L1 - k1 (frequencies k
// and L - k pair up between them): forward row transforms, separation into
// the two sequences' power spectra, inverse row transforms, inverse twiddles.
__global__ __launch_bounds__(kThreads) void fft_rows_kernel(FftArgs a) {
    extern __shared__ double2 lds[];   // [L2][2], slot q of point i at 2 i + q
    const int64_t per = (int64_t(1) << (a.lg1 - 1)) + 1;
    const int64_t id = xcd_remap(blockIdx.x, gridDim.x);
    const int64_t pair = id / per;
    const uint32_t l1 = 1u << a.lg1;
    const uint32_t k1a = (uint32_t)(id % per);
    const uint32_t k1b = (l1 - k1a) & (l1 - 1);
    const bool self = k1a == k1b;
    const int64_t ra = bitrev(k1a, a.lg1), rb = bitrev(k1b, a.lg1);
    const int l2 = 1 << a.lg2;
    double2* __restrict__ zp = a.z + pair * a.len;
    for (int f = threadIdx.x; f < 2 * l2; f += kThreads) {
        const int64_t row = (f & 1) ? rb : ra;
        lds[f] = zp[row * l2 + (f >> 1)];
    }
    __syncthreads();
    lds_fft_fwd(lds, a.lg2, 1, a.tw + a.tw_b);
    double2 wv[kRegPoints];
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int f = threadIdx.x + r * kThreads;
        if (f < 2 * l2) {
            const int q = f & 1;
            const uint32_t k1 = q ? k1b : k1a;
            const uint32_t k2 = bitrev(f >> 1, a.lg2);
            const uint32_t k2m = k1 == 0 ? ((l2 - k2) & (l2 - 1)) : (l2 - 1 - k2);
            const int qm = self ? q : 1 - q;
            wv[r] = power_pair(lds[f], lds[2 * bitrev(k2m, a.lg2) + qm]);
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRegPoints; ++r) {
        const int f = threadIdx.x + r * kThreads;
        if (f < 2 * l2) lds[f] = wv[r];
    }
    __syncthreads();
    lds_fft_inv(lds, a.lg2, 1, a.tw + a.tw_b);
    for (int f = threadIdx.x; f < 2 * l2; f += kThreads) {
        const int q = f & 1;
        if (q && self) continue;
        const int64_t n2 = f >> 1;
        const int64_t k1 = q ? k1b : k1a;
        zp[(q ? rb : ra) * l2 + n2] = cmul_conj(lds[f], twiddle(a, k1 * n2));
    }
}

// Split transform, step 3: inverse column transforms (row p holds k1 =
// bitrev(p): the bit-reversed input order of the decimation in time), and
// D(T) for the lags T = n1 L2 + n2 in [tmin, tmax].
__global__ __launch_bounds__(kThreads) void fft_cols_inv_kernel(FftArgs a) {
    extern __shared__ double2 lds[];
    const int64_t groups = int64_t(1) << (a.lg2 - a.lgc);
    const int64_t id = xcd_remap(blockIdx.x, gridDim.x);
    const int64_t pair = id / groups;
    const int64_t c0 = (id % groups) << a.lgc;
    const int cols = 1 << a.lgc;
    const int npts = (1 << a.lg1) * cols;
    const int64_t l2 = int64_t(1) << a.lg2;
    const double2* __restrict__ zp = a.z + pair * a.len;
    for (int f = threadIdx.x; f < npts; f += kThreads)
        lds[f] = zp[(int64_t)(f >> a.lgc) * l2 + c0 + (f & (cols - 1))];
    __syncthreads();
    lds_fft_inv(lds, a.lg1, a.lgc, a.tw + a.tw_a);
    const int rows = (int)(a.tmax / l2) + 1;
    for (int f = threadIdx.x; f < rows * cols; f += kThreads) {
        const int64_t t = (int64_t)(f >> a.lgc) * l2 + c0 + (f & (cols - 1));
        write_d(a, 2 * pair, t, lds[f].x);
        write_d(a, 2 * pair + 1, t, lds[f].y);
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
        for (int32_t c = 0; c < a.num_channels; ++c)
            acc += (double)w.w[c] * fft_bound(a.fstat, b * a.num_channels + c, a.seqs, n, a.lg);
        abound = acc * (1.0 + 1e-12);
    }
    __syncthreads();
    const double ab = abound;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x >> 6;
    const float* __restrict__ xw = a.x + table_off(a.tab, b, a.window_stride);
    const int32_t nlags = tm - a.tmin + 1;
    for (int32_t j0 = wave * kWave; j0 < nlags; j0 += kThreads) {
        const int32_t j = j0 + lane;
        bool fix = false;
        if (j < nlags) {
            const int64_t t = (int64_t)a.tmin + j;
            const double v = a.s64[b * a.lags + j];
            fix = !(ab / (double)(n - t) <= 0.5 * a.tau0 * v);
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

FftArgs args_of(const Plan& p, const float* x, double* fstat, double* edge, double* tw, double* z,
                double* part) {
    FftArgs a;
    a.x = x;
    a.fstat = fstat;
    a.edge = edge;
    a.tw = reinterpret_cast<const double2*>(tw);
    a.z = reinterpret_cast<double2*>(z);
    a.part = part;
    a.seqs = p.num_windows * (int64_t)p.num_channels;
    a.n_all = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.len = p.fft_len;
    a.num_channels = p.num_channels;
    a.tmin = p.tmin;
    a.tmax = p.tmax;
    a.lags = p.lags;
    a.lg = p.fft_log2;
    a.tab = p.table;
    if (p.fft_m2 == 1) {   // one workgroup per pair
        a.lg1 = p.fft_log2;
        a.lg2 = 0;
        a.lgc = 0;
        a.tw_a = 0;
        a.tw_b = a.tw_lo = a.tw_hi = 0;
    } else {
        a.lg1 = __builtin_ctz((unsigned)p.fft_m1);
        a.lg2 = __builtin_ctz((unsigned)p.fft_m2);
        a.lgc = __builtin_ctz((unsigned)p.fft_cols);
        a.tw_a = 0;
        a.tw_b = p.fft_m1 / 2;
        a.tw_lo = a.tw_b + p.fft_m2 / 2;
        a.tw_hi = a.tw_lo + p.fft_m2;
    }
    return a;
}

}  // namespace

// Complex fp64 entries of the twiddle tables of a plan.
int64_t fft_twiddle_count(const Plan& p) {
    if (p.fft_m2 == 1) return p.fft_len / 2;
    return p.fft_m1 / 2 + p.fft_m2 / 2 + p.fft_m2 + p.fft_m1;
}

hipError_t launch_fft_scores(const Plan& p, const float* x, double* fstat, double* edge,
                             double* tw, double* z, double* part, hipStream_t s) {
    const FftArgs a = args_of(p, x, fstat, edge, tw, z, part);
    const int64_t count = fft_twiddle_count(p);
    int64_t tg = (count + 255) / 256;
    if (tg > 1024) tg = 1024;
    if (p.fft_m2 == 1) {
        hipLaunchKernelGGL(fft_twiddle_kernel, dim3((unsigned)tg), dim3(256), 0, s,
                           reinterpret_cast<double2*>(tw), a.lg, 1, a.lg, 0, (int64_t)0,
                           (int64_t)0, (int64_t)0);
    } else {
        hipLaunchKernelGGL(fft_twiddle_kernel, dim3((unsigned)tg), dim3(256), 0, s,
                           reinterpret_cast<double2*>(tw), a.lg1, a.lg2, a.lg, a.lg2,
                           (int64_t)(p.fft_m2 / 2), (int64_t)p.fft_m2, (int64_t)p.fft_m1);
    }
    hipLaunchKernelGGL(fft_prep_kernel, dim3((unsigned)a.seqs), dim3(kThreads), 0, s, a);
    if (p.fft_m2 == 1) {
        const size_t lds = sizeof(double2) * (size_t)p.fft_len;
        hipLaunchKernelGGL(fft_single_kernel, dim3((unsigned)p.fft_pairs), dim3(kThreads), lds, s,
                           a);
        return hipGetLastError();
    }
    const int64_t col_groups = p.fft_pairs * (p.fft_m2 / p.fft_cols);
    const size_t lds_cols = sizeof(double2) * (size_t)p.fft_m1 * p.fft_cols;
    const size_t lds_rows = sizeof(double2) * 2 * (size_t)p.fft_m2;
    const int64_t row_groups = p.fft_pairs * (p.fft_m1 / 2 + 1);
    hipLaunchKernelGGL(fft_cols_fwd_kernel, dim3((unsigned)col_groups), dim3(kThreads), lds_cols,
                       s, a);
    hipLaunchKernelGGL(fft_rows_kernel, dim3((unsigned)row_groups), dim3(kThreads), lds_rows, s, a);
    hipLaunchKernelGGL(fft_cols_inv_kernel, dim3((unsigned)col_groups), dim3(kThreads), lds_cols,
                       s, a);
    return hipGetLastError();
}

hipError_t launch_fft_fixup(const Plan& p, const Weights& w, const float* x, const double* fstat,
                            double* s64, float* scores, const SelectBuffers& sb, hipStream_t s) {
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
    hipLaunchKernelGGL(fft_fixup_kernel, dim3((unsigned)p.num_windows), dim3(kThreads), 0, s, a,
                       w);
    return hipGetLastError();
}

}  // namespace gpoeo
