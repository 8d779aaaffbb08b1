// Mean-removed score S_c(T) at finalist periods (Sec. 4.1.2, Algorithm 2's
// relative values with one group per sample).
//
// For a window and a candidate period T the trace is cut into Num_T =
// floor(N/T) whole sub-curves of T samples; every adjacent pair (i, i+1) is
// compared point by point after each sub-curve's own mean is removed:
//   D_c = sum_{i < Num_T - 1} sum_{j<T} ((x[iT+j] - mu_i) - (x[(i+1)T+j] - mu_{i+1}))^2
//   S_c(T) = sum_c w_c D_c / ((Num_T - 1) T).
// Equivalently SSD - T sum_i (mu_i - mu_{i+1})^2 over the whole-sub-curve
// pairs: a linear drift adds the same amount to every difference of a pair and
// leaves S_c unchanged.  Because removing the means also removes most of a
// short lag's differences, S_c suits re-scoring candidate periods (as
// Algorithm 1 applies Algorithm 2 to its candidates), not an exhaustive scan.
//
// Evaluation.  The centred difference of point j of pair (a, b) is
// d_j - mean(d) with d_j = a_j - b_j (mean(d) = mu_a - mu_b), so a pair's sum is
// the sum of squared deviations of d from its mean.  Each lane takes one pass
// over its points, in blocks whose moments are merged with the pairwise
// formula of Chan, Golub and LeVeque (as are the lanes' partial results): no
// sub-curve is read twice for a pair, there is no cancellation under drift,
// and a pair whose differences are all equal (a drift of a whole number of
// periods) gives exactly 0.
//
// Work mapping.  One workgroup of kThreads lanes per (window, lag) query.  The
// lanes form segments of S lanes (S a power of two, 1..64, chosen per query):
// segment g takes the pairs g, g + kThreads/S, ...; its lanes stride over the
// T points of a pair and merge their partial results by a butterfly of lane
// shuffles inside the segment (each merge ordered by lane, so both partners
// compute the same bits).  Each segment adds its pair sums in pair order and
// the segments' sums are added in segment order, so the result does not depend
// on scheduling.  Queries are dealt to the XCDs in contiguous ranges, so the
// queries of one window (which callers list together) read it through the same
// L2.  All arithmetic is fp64.
#include "internal.h"

namespace gpoeo {
namespace {

constexpr int kThreads = 256;

// Count, mean and sum of squared deviations of a run of points.
struct Moments {
    double n, mean, m2;
};

// Merge of two runs (Chan, Golub and LeVeque's pairwise update); `lo` is the
// run of the lower lane (or the earlier points), so both lanes of a butterfly
// step get the same bits.
__device__ __forceinline__ Moments merge(const Moments& lo, const Moments& hi) {
    if (hi.n == 0.0) return lo;
    if (lo.n == 0.0) return hi;
    const double n = lo.n + hi.n;
    const double f = hi.n / n;
    const double d = hi.mean - lo.mean;
    Moments r;
    r.n = n;
    r.mean = lo.mean + d * f;
    r.m2 = (lo.m2 + hi.m2) + d * d * (lo.n * f);
    return r;
}

__device__ __forceinline__ Moments seg_merge(Moments m, int s, int ls) {
    for (int o = s >> 1; o > 0; o >>= 1) {
        Moments p;
        p.n = __shfl_xor(m.n, o);
        p.mean = __shfl_xor(m.mean, o);
        p.m2 = __shfl_xor(m.m2, o);
        m = (ls & o) ? merge(p, m) : merge(m, p);
    }
    return m;
}

struct CentredArgs {
    const float* x;
    const int32_t* windows;
    const int32_t* lags;
    double* out;
    int64_t num_windows;
    int64_t n;
    int64_t window_stride;
    int64_t channel_stride;
    int32_t num_channels;
};

// Segment width: the S minimising pair rounds times the cost of a round, which
// is its sample steps (each step two loads; below 16 lanes a load instruction
// touches 64 / S separate 64-byte pieces, which the address unit serialises)
// plus the merge steps.
__device__ __forceinline__ int choose_segment(int64_t pairs, int64_t t) {
    int best_s = 1;
    double best = INFINITY;
    for (int s = 1, lg = 0; s <= kWave; s <<= 1, ++lg) {
        const int64_t per_round = kThreads / s;
        const int64_t rounds = (pairs + per_round - 1) / per_round;
        const double step = 4.0 + (s < 16 ? 16.0 / (double)s : 1.0);
        const double cost = (double)rounds * ((double)((t + s - 1) / s) * step + 6.0 * lg);
        if (cost < best) {
            best = cost;
            best_s = s;
        }
    }
    return best_s;
}

// Sum over j < t of the squared difference of the mean-removed points of the
// sub-curves a and b, computed by the s lanes of a segment (this lane is ls).
// A lane takes its points in blocks of kBlock: a block's moments come from
// sums of the differences shifted by the block's first one, a member of the
// block, so the sum of squares exceeds the block's squared deviations by at
// most a factor kBlock + 1 and its subtraction loses at most that much; the
// blocks, then the last few points one by one, are merged in order.
constexpr int kBlock = 8;

__device__ double pair_sum(const float* __restrict__ a, const float* __restrict__ b, int64_t t,
                           int s, int ls) {
    Moments m = {0.0, 0.0, 0.0};
    int64_t j = ls;
    for (; j + (kBlock - 1) * (int64_t)s < t; j += kBlock * (int64_t)s) {
        double d[kBlock];
#pragma unroll
        for (int u = 0; u < kBlock; ++u)
            d[u] = (double)a[j + u * (int64_t)s] - (double)b[j + u * (int64_t)s];
        double s1 = 0.0, s2 = 0.0;
#pragma unroll
        for (int u = 1; u < kBlock; ++u) {
            const double e = d[u] - d[0];
            s1 += e;
            s2 = fma(e, e, s2);
        }
        const double q = s1 * (1.0 / kBlock);
        Moments blk;
        blk.n = (double)kBlock;
        blk.mean = d[0] + q;
        blk.m2 = fmax(s2 - s1 * q, 0.0);
        m = merge(m, blk);
    }
    for (; j < t; j += s) {
        Moments one;
        one.n = 1.0;
        one.mean = (double)a[j] - (double)b[j];
        one.m2 = 0.0;
        m = merge(m, one);
    }
    return seg_merge(m, s, ls).m2;
}

__global__ __launch_bounds__(kThreads) void centred_kernel(CentredArgs a, Weights w) {
    __shared__ double part[kThreads];
    const int tid = threadIdx.x;
    const int64_t groups = gridDim.x;
    int64_t q = blockIdx.x;
    const int64_t full = groups - groups % 8;
    if (q < full) q = (q % 8) * (full / 8) + q / 8;
    const int64_t win = a.windows[q];
    const int64_t t = a.lags[q];
    if (win < 0 || win >= a.num_windows || t < 1 || t > a.n) {
        if (tid == 0) a.out[q] = NAN;
        return;
    }
    const int64_t pairs = a.n / t - 1;
    if (pairs < 1) {
        if (tid == 0) a.out[q] = -1.0;
        return;
    }
    const int s = choose_segment(pairs, t);
    const int seg = tid / s, ls = tid % s, nseg = kThreads / s;
    double acc = 0.0;
    for (int32_t c = 0; c < a.num_channels; ++c) {
        const float* xc = a.x + win * a.window_stride + (int64_t)c * a.channel_stride;
        double mine = 0.0;
        for (int64_t i = seg; i < pairs; i += nseg)
            mine += pair_sum(xc + i * t, xc + (i + 1) * t, t, s, ls);
        __syncthreads();
        if (ls == 0) part[seg] = mine;
        __syncthreads();
        double total = 0.0;
        for (int g = 0; g < nseg; ++g) total += part[g];
        acc += (double)w.w[c] * (total / (double)(pairs * t));
    }
    if (tid == 0) a.out[q] = acc;
}

}  // namespace

hipError_t launch_centred(const Plan& p, const Weights& w, const float* x, const int32_t* windows,
                          const int32_t* lags, int64_t count, double* out, hipStream_t s) {
    CentredArgs a;
    a.x = x;
    a.windows = windows;
    a.lags = lags;
    a.out = out;
    a.num_windows = p.num_windows;
    a.n = p.n;
    a.window_stride = p.window_stride;
    a.channel_stride = p.channel_stride;
    a.num_channels = p.num_channels;
    hipLaunchKernelGGL(centred_kernel, dim3((unsigned)count), dim3(kThreads), 0, s, a, w);
    return hipGetLastError();
}

}  // namespace gpoeo
