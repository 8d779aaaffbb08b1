"""Exact-rational evaluations for tiny inputs (TEST INFRASTRUCTURE ONLY).

Every fp32 sample is an exact binary fraction, so ``fractions.Fraction`` gives
the score S(T) (paper Sec. 4.1.2, Algorithm 2 read as the mean squared
point-wise difference of adjacent sub-curves over all N-T pairs) and the
reference R with no rounding at all.  Pure-Python loops: only for N of a few
dozen samples.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np


def exact_score(xw, t: int, weights=None) -> Fraction:
    """S(T) of one window [C][N] as an exact rational."""
    xw = np.atleast_2d(np.asarray(xw, dtype=np.float32))
    c_count, n = xw.shape
    total = Fraction(0)
    for c in range(c_count):
        xs = [Fraction(float(v)) for v in xw[c]]
        d = sum(((xs[i] - xs[i + t]) ** 2 for i in range(n - t)), Fraction(0))
        w = Fraction(1) if weights is None else Fraction(float(np.float32(weights[c])))
        total += w * d / (n - t)
    return total


def exact_reference(xw, weights=None) -> Fraction:
    """R = 2 * sum_c w_c * population variance, exactly."""
    xw = np.atleast_2d(np.asarray(xw, dtype=np.float32))
    c_count, n = xw.shape
    acc = Fraction(0)
    for c in range(c_count):
        xs = [Fraction(float(v)) for v in xw[c]]
        mean = sum(xs, Fraction(0)) / n
        var = sum(((v - mean) ** 2 for v in xs), Fraction(0)) / n
        w = Fraction(1) if weights is None else Fraction(float(np.float32(weights[c])))
        acc += w * var
    return 2 * acc


def exact_score_centred(xw, t: int, weights=None) -> Fraction:
    """S_c(T) of one window [C][N] as an exact rational: floor(N/T) whole
    sub-curves, each pair of neighbours compared point by point after removing
    each sub-curve's own mean (Algorithm 2's relative values, one group per
    sample)."""
    xw = np.atleast_2d(np.asarray(xw, dtype=np.float32))
    c_count, n = xw.shape
    pairs = n // t - 1
    total = Fraction(0)
    for c in range(c_count):
        xs = [Fraction(float(v)) for v in xw[c]]
        d = Fraction(0)
        for i in range(pairs):
            a, b = xs[i * t:(i + 1) * t], xs[(i + 1) * t:(i + 2) * t]
            ma, mb = sum(a, Fraction(0)) / t, sum(b, Fraction(0)) / t
            d += sum((((u - ma) - (v - mb)) ** 2 for u, v in zip(a, b)), Fraction(0))
        w = Fraction(1) if weights is None else Fraction(float(np.float32(weights[c])))
        total += w * d / (pairs * t)
    return total
