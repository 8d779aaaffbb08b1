// fp64 helpers of the Gaussian-mixture grouping (Algorithm 2): 2^z for z <= 0
// and a reciprocal, both cheaper than the general library routines.
//
// gmm_exp2_nonpos(z) = 2^z for z <= 0: the responsibilities of the E-step are
// 2^(l_k - max_j l_j) with base-2 log-densities l_k, so the argument is never
// positive.  Method: the exact range reduction z = k + f, k = rint(z), f = z - k
// in [-1/2, 1/2] (exact for |z| < 2^52), 2^f from its Taylor series
// sum_{n <= 13} (f ln 2)^n / n! evaluated by Horner's rule with fused
// multiply-adds (truncation below 4.2e-18 relative on |f ln 2| <= 0.347), and
// the scaling by 2^k with ldexp.  Arguments below -1022 are clamped there, so
// the result never leaves the normal range (2^-1022 instead of a subnormal or
// 0, a difference far below any value a normalised sum of responsibilities
// can resolve).  The function is exact at 0 (returns 1).  Compiled for the host
// as well, where the same IEEE operations give the same bits, so it is checked
// against libm on the CPU.
#pragma once

#include <math.h>

#if defined(__HIPCC__)
#define GPOEO_HD __host__ __device__
#else
#define GPOEO_HD
#endif

namespace gpoeo {

GPOEO_HD inline double gmm_exp2_nonpos(double z) {
    // (ln 2)^n / n!, n = 0..13, each the double nearest the exact value
    constexpr double c0 = 1.0, c1 = 0.6931471805599453, c2 = 0.24022650695910072,
                     c3 = 0.05550410866482158, c4 = 0.009618129107628477,
                     c5 = 0.0013333558146428443, c6 = 0.0001540353039338161,
                     c7 = 1.5252733804059841e-05, c8 = 1.321548679014431e-06,
                     c9 = 1.01780860092397e-07, c10 = 7.054911620801123e-09,
                     c11 = 4.4455382718708116e-10, c12 = 2.5678435993488206e-11,
                     c13 = 1.3691488853904128e-12;
    z = fmax(z, -1022.0);
    const double k = rint(z);
    const double f = z - k;
    double p = c13;
    p = fma(p, f, c12);
    p = fma(p, f, c11);
    p = fma(p, f, c10);
    p = fma(p, f, c9);
    p = fma(p, f, c8);
    p = fma(p, f, c7);
    p = fma(p, f, c6);
    p = fma(p, f, c5);
    p = fma(p, f, c4);
    p = fma(p, f, c3);
    p = fma(p, f, c2);
    p = fma(p, f, c1);
    p = fma(p, f, c0);
    return ldexp(p, (int)k);
}

}  // namespace gpoeo
