"""The EM's fp64 2^z (csrc/gmm_math.h), compiled for the host, against libm.

gmm_exp2_nonpos uses only IEEE operations (rint, subtraction, fused
multiply-add, ldexp), so the host build computes the same bits as the GPU
build.  Its error against the long-double exp2l must stay within libm's own
1-ulp bound for exp2 on the whole argument range the E-step uses (z <= 0,
clamped at -1022), and it must be exact at 0 and at negative integers.
"""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

DRIVER = r"""
#include <cstdio>
#include <cmath>
#include <cstdint>
#include "gmm_math.h"
int main() {
    double worst = 0.0;
    uint64_t s = 88172645463325252ull;
    auto ulp = [](double ref) { int e; frexp(ref, &e); return ldexp(1.0, e - 53); };
    for (long i = 0; i < 2000000; ++i) {
        s ^= s << 13; s ^= s >> 7; s ^= s << 17;
        const double u = (double)(s >> 11) / 9007199254740992.0;
        const double z = (i % 2) ? -u * 1022.0 : -u * 2.0;
        const long double ref = exp2l((long double)z);
        const double g = gpoeo::gmm_exp2_nonpos(z);
        const double err = (double)(fabsl((long double)g - ref) / ulp((double)ref));
        if (err > worst) worst = err;
    }
    int exact = gpoeo::gmm_exp2_nonpos(0.0) == 1.0;
    for (int k = 1; k <= 1022; ++k) exact &= gpoeo::gmm_exp2_nonpos(-(double)k) == ldexp(1.0, -k);
    printf("%.6f %d %.17g %.17g\n", worst, exact, gpoeo::gmm_exp2_nonpos(-2000.0),
           gpoeo::gmm_exp2_nonpos(-0.5));
    return 0;
}
"""


def test_exp2_within_one_ulp_of_libm(tmp_path):
    src = tmp_path / "exp2.cpp"
    src.write_text(DRIVER)
    exe = tmp_path / "exp2"
    subprocess.run(["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-I",
                    os.path.join(ROOT, "paper_2201_01684_amd", "csrc"), str(src), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()
    worst, exact, clamped, half = float(out[0]), int(out[1]), float(out[2]), float(out[3])
    assert worst <= 1.0, f"max error {worst} ulp"
    assert exact == 1
    assert clamped == 2.0 ** -1022          # below -1022 the argument is clamped
    assert abs(half - 2 ** -0.5) <= 2 ** -53
