"""Pins of the oracle's mean-removed score S_c(T) (Algorithm 2's relative values
with one group per sample: each sub-curve's own mean is removed before
corresponding points of adjacent whole sub-curves are compared).

Pinned against: exact rationals on tiny inputs, the closed form
SSD - T sum_i (mu_i - mu_{i+1})^2 evaluated independently with numpy, exact
zeros of a periodic trace under integer linear drift, invariance under any
added linear ramp at every lag, and its ordering against the uncentred sum
over the same pairs.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle.brute import exact_score_centred
from gen import planted_trace


def closed_form(x, t):
    """SSD over whole sub-curve pairs minus T sum (mu_i - mu_{i+1})^2, by numpy."""
    x = np.asarray(x, dtype=np.float64)
    k = x.size // t
    blocks = x[:k * t].reshape(k, t)
    ssd = np.sum((blocks[:-1] - blocks[1:]) ** 2)
    mu = blocks.mean(axis=1)
    return (ssd - t * np.sum((mu[:-1] - mu[1:]) ** 2)) / ((k - 1) * t)


@pytest.mark.parametrize("n,seed", [(12, 0), (17, 1), (24, 2)])
def test_exact_rationals_on_tiny_inputs(n, seed):
    rng = np.random.default_rng(seed)
    x = rng.normal(10, 3, size=n).astype(np.float32)
    for t in range(1, n // 2 + 1):
        exact = exact_score_centred(x, t)
        got = oracle.score_centred(x, t)
        if exact == 0:
            assert got == 0.0
        else:
            assert abs(Fraction(got) - exact) <= Fraction(1, 10**12) * exact, t


def test_exact_rationals_weighted_channels():
    rng = np.random.default_rng(9)
    x = rng.normal(0, 1, size=(2, 20)).astype(np.float32)
    w = np.array([0.5, 3.0], dtype=np.float32)
    for t in (2, 3, 7, 10):
        exact = exact_score_centred(x, t, w)
        got = oracle.score_centred(x, t, w)
        assert abs(Fraction(got) - exact) <= Fraction(1, 10**12) * exact


@pytest.mark.parametrize("t", [7, 64, 100, 333])
def test_closed_form(t):
    x = planted_trace(5000, 250, 6, seed=t, sigma=3.0)
    assert oracle.score_centred(x, t) == pytest.approx(closed_form(x, t), rel=1e-9)


@pytest.mark.parametrize("period,slope", [(64, 1), (128, 3), (256, -2)])
def test_integer_drift_leaves_exact_zeros(period, slope):
    # integer levels plus an integer ramp: every value exact; a power-of-two
    # period makes every sub-curve mean exact, so the relative values of
    # neighbouring sub-curves coincide
    base = planted_trace(40 * period, period, 5, seed=period, integer=True).astype(np.int64)
    x = (base + slope * np.arange(base.size)).astype(np.float32)
    for k in (1, 2, 3):
        assert oracle.score_centred(x, k * period) == 0.0
        assert oracle.score(x, k * period) == pytest.approx((slope * k * period) ** 2)
    assert oracle.score_centred(x, period + 1) > 0.0


def test_any_linear_ramp_changes_no_score():
    x = planted_trace(6000, 321, 7, seed=5, sigma=2.0)
    ramp = (x.astype(np.float64) + 0.37 * np.arange(x.size)).astype(np.float32)
    for t in (5, 50, 321, 500, 2999):
        a, b = oracle.score_centred(x, t), oracle.score_centred(ramp, t)
        # the fp32 rounding of the ramped samples moves the score by ~1e-6 at most
        assert b == pytest.approx(a, rel=1e-5), t


def test_centring_never_increases_the_whole_pair_sum():
    rng = np.random.default_rng(4)
    x = (rng.normal(0, 1, 3000) + np.linspace(0, 40, 3000)).astype(np.float32)
    xd = x.astype(np.float64)
    for t in (3, 30, 300, 1500):
        k = x.size // t
        ssd = np.sum((xd[:(k - 1) * t] - xd[t:k * t]) ** 2) / ((k - 1) * t)
        c = oracle.score_centred(x, t)
        assert 0.0 <= c <= ssd * (1 + 1e-12)


def test_score_list_and_rejected_lags():
    x = planted_trace(4000, 137, 5, seed=1)
    lay = oracle.Layout(1, 1, 4000, 4000, 4000, 2, 2000, centred=True)
    got = oracle.score_list(x, lay, [0, 0], [137, 400])
    assert got[0] == oracle.score_centred(x, 137) and got[1] == oracle.score_centred(x, 400)
    with pytest.raises(ValueError):
        oracle.score_list(x, lay, [0], [2001])      # one whole sub-curve only
    with pytest.raises(ValueError):
        oracle.score_list(x, lay, [0], [0])
