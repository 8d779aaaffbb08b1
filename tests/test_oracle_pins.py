"""Pins of the fp64 CPU oracle against facts fixed by the mathematics, not by itself.

Score S(T) (Sec. 4.1.2, Algorithm 2 read as the mean squared point-wise
difference of adjacent sub-curves over all N-T pairs):
  * exact rational brute force on tiny inputs (single and weighted multi-channel);
  * closed forms: unit step, sinusoid over whole periods, integer-valued inputs;
  * the energy / cross-correlation identity with numpy.correlate;
  * invariants: offset, power-of-two scale, time reversal, zeros at multiples
    of an exact integer period, white-noise expectation.
Reference R: exact rational brute force.
"""
from fractions import Fraction
import math

import numpy as np
import pytest

import oracle
from oracle import brute


def _rng(seed):
    return np.random.default_rng(seed)


# ----------------------------------------------------------------------------
# Brute force
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("n", [4, 9, 17, 32])
def test_score_matches_exact_rational(seed, n):
    x = (_rng(seed).normal(0, 1, size=n) * 10 ** _rng(seed + 99).uniform(-2, 3)).astype(np.float32)
    for t in range(0, n // 2 + 1):
        exact = brute.exact_score(x, t)
        got = oracle.score(x, t)
        if exact == 0:
            assert got == 0.0
        else:
            rel = abs(Fraction(got) - exact) / exact
            assert rel <= n * 2.0 ** -53, (t, float(rel))


@pytest.mark.parametrize("seed", range(4))
def test_weighted_multichannel_score_and_reference_exact(seed):
    rng = _rng(seed)
    c, n = 3, 20
    x = np.stack([rng.normal(m, s, size=n) for m, s in [(100, 5), (0.5, 0.2), (1e4, 3e3)]])
    x = x.astype(np.float32)
    w = np.array([0.5, 2.0, 1e-6], dtype=np.float32)
    for t in range(1, n // 2 + 1):
        exact = brute.exact_score(x, t, w)
        got = oracle.score(x, t, w)
        assert abs(Fraction(got) - exact) / exact <= 4 * n * 2.0 ** -53
    r_exact = brute.exact_reference(x, w)
    assert abs(Fraction(oracle.reference(x, w)) - r_exact) / r_exact <= 4 * n * 2.0 ** -53


def test_reference_exact_single_channel():
    x = _rng(7).uniform(80, 400, size=31).astype(np.float32)
    r_exact = brute.exact_reference(x)
    assert abs(Fraction(oracle.reference(x)) - r_exact) / r_exact <= 31 * 2.0 ** -53
    # R is twice the population (not the sample) variance
    assert oracle.reference(x) == pytest.approx(2 * np.var(x.astype(np.float64)), rel=1e-13)


# ----------------------------------------------------------------------------
# Closed forms
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("n,m", [(64, 32), (100, 30), (257, 200), (4096, 1000)])
def test_unit_step_closed_form(n, m):
    # x = 0 before m, 1 from m on: exactly T of the N-T pairs straddle the step
    x = np.zeros(n, dtype=np.float32)
    x[m:] = 1.0
    for t in range(1, min(m, n - m, n // 2) + 1):
        assert oracle.score(x, t) == float(Fraction(t, n - t))


@pytest.mark.parametrize("period,t", [(7, 1), (7, 3), (12, 5), (50, 17), (3, 1), (64, 32)])
def test_sinusoid_closed_form(period, t):
    # N - T a whole number of periods: S(T) = 2 A^2 sin^2(pi T / P)
    a, phi = 3.0, 0.4
    n = t + period * 40
    i = np.arange(n)
    x = (a * np.sin(2 * np.pi * i / period + phi)).astype(np.float32)
    want = 2 * a * a * math.sin(math.pi * t / period) ** 2
    assert oracle.score(x, t) == pytest.approx(want, rel=2e-6, abs=1e-9)


@pytest.mark.parametrize("seed", range(3))
def test_integer_inputs_sum_exactly(seed):
    x = _rng(seed).integers(-1000, 1000, size=257).astype(np.float32)
    for t in (1, 2, 50, 128):
        exact = brute.exact_score(x, t)
        assert oracle.score(x, t) == float(exact)


# ----------------------------------------------------------------------------
# Identity with the cross-correlation
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(3))
def test_energy_minus_correlation_identity(seed):
    n = 600
    x = (_rng(seed).normal(0, 1, size=n) + 0.5 * np.sin(np.arange(n) / 7.0)).astype(np.float32)
    y = x.astype(np.float64) - x.astype(np.float64).mean()
    r = np.correlate(y, y, mode="full")[n - 1:]            # r[T] = sum_i y[i] y[i+T]
    for t in (1, 2, 3, 44, 150, 300):
        e1 = np.sum(y[: n - t] ** 2)
        e2 = np.sum(y[t:] ** 2)
        want = (e1 + e2 - 2 * r[t]) / (n - t)
        assert oracle.score(x, t) == pytest.approx(want, rel=1e-9)


# ----------------------------------------------------------------------------
# Invariants
# ----------------------------------------------------------------------------

def test_lag_zero_and_nonnegative():
    x = _rng(3).normal(200, 30, size=500).astype(np.float32)
    assert oracle.score(x, 0) == 0.0
    assert all(oracle.score(x, t) >= 0.0 for t in range(1, 251))


def test_offset_invariance_exact_for_integer_data():
    x = _rng(4).integers(0, 500, size=300).astype(np.float32)
    for t in (1, 9, 77, 150):
        assert oracle.score(x + np.float32(1234), t) == oracle.score(x, t)


def test_power_of_two_scaling_is_exact():
    x = _rng(5).normal(0, 3, size=400).astype(np.float32)
    for t in (1, 13, 200):
        assert oracle.score(x * np.float32(8), t) == 64.0 * oracle.score(x, t)
        assert oracle.reference(x * np.float32(0.25)) == oracle.reference(x) / 16.0


def test_time_reversal():
    xi = _rng(6).integers(-50, 50, size=333).astype(np.float32)
    xr = _rng(6).normal(5, 2, size=333).astype(np.float32)
    for t in (1, 5, 100, 166):
        assert oracle.score(xi[::-1].copy(), t) == oracle.score(xi, t)
        assert oracle.score(xr[::-1].copy(), t) == pytest.approx(oracle.score(xr, t), rel=1e-13)


@pytest.mark.parametrize("period", [5, 37, 137])
def test_zero_at_every_multiple_of_an_exact_period(period):
    from gen import planted_trace
    x = planted_trace(4096, period, 4, seed=period, sigma=0.0)
    for k in range(1, 2048 // period + 1):
        assert oracle.score(x, k * period) == 0.0
    assert oracle.score(x, period + 1) > 0.0


def test_white_noise_expectation():
    sigma = 2.0
    x = _rng(8).normal(0, sigma, size=200_000).astype(np.float32)
    for t in (1, 10, 1000):
        assert oracle.score(x, t) == pytest.approx(2 * sigma ** 2, rel=0.02)


# ----------------------------------------------------------------------------
# Batch entry points agree with the single-lag definition
# ----------------------------------------------------------------------------

def test_batch_and_list_entry_points_use_the_same_definition():
    rng = _rng(9)
    b, c, n = 3, 2, 256
    x = rng.normal(0, 1, size=(b, c, n)).astype(np.float32)
    w = np.array([1.0, 0.25], dtype=np.float32)
    lay = oracle.Layout(b, c, n, c * n, n, 2, 128, weights=w)
    scores, out = oracle.detect(x, lay)
    for bb in range(b):
        for t in (2, 3, 64, 128):
            assert scores[bb, t - 2] == oracle.score(x[bb], t, w)
        assert out["r"][bb] == oracle.reference(x[bb], w)
    ws = np.array([0, 2, 1]); ts = np.array([2, 128, 77])
    got = oracle.score_list(x, lay, ws, ts)
    for k in range(3):
        assert got[k] == oracle.score(x[ws[k]], ts[k], w)


def test_overlapping_windows_read_in_place():
    x = _rng(10).normal(0, 1, size=1000).astype(np.float32)
    lay = oracle.Layout(num_windows=5, num_channels=1, n=512, window_stride=100,
                        channel_stride=512, tmin=1, tmax=256)
    scores, _ = oracle.detect(x, lay)
    for b in range(5):
        assert scores[b, 9] == oracle.score(x[100 * b: 100 * b + 512], 10)


def test_invalid_parameters_rejected():
    x = np.zeros(100, dtype=np.float32)
    with pytest.raises(ValueError):
        oracle.detect(x, oracle.Layout(1, 1, 100, 100, 100, 1, 51))   # tmax > n/2
    with pytest.raises(ValueError):
        oracle.detect(x, oracle.Layout(1, 1, 100, 100, 100, 5, 6))    # tmin + 2 > tmax
    with pytest.raises(ValueError):
        oracle.detect(x, oracle.Layout(1, 1, 100, 100, 100, 0, 10))   # tmin < 1
