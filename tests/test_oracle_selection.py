"""Pins of the oracle's selection rule (Algorithm 1 read in the lag domain).

Hand-built score rows whose answers follow from the rule by inspection, the
exact integer local-search window against the paper's own formula for it, and
planted periods in generated traces.
"""
from fractions import Fraction
import math

import numpy as np
import pytest

import oracle
from gen import make_workload, planted_trace


def row(tmin, values):
    s = np.asarray(values, dtype=np.float64)
    return s, tmin, tmin + len(values) - 1


def test_constant_window():
    s, tmin, tmax = row(2, [0.0] * 20)
    o = oracle.select(s, 100, tmin, tmax, 0.0)
    assert o["verdict"] == oracle.CONSTANT and o["period"] == 0


def test_monotone_scores_have_no_peak():
    # a boundary minimum at Tmin is not a peak
    s, tmin, tmax = row(2, list(range(10, 30)))
    o = oracle.select(s, 100, tmin, tmax, 100.0)
    assert o["verdict"] == oracle.APERIODIC and o["period"] == 0 and o["n_peaks"] == 0
    # nor is one at Tmax
    s, tmin, tmax = row(2, list(range(30, 10, -1)))
    o = oracle.select(s, 100, tmin, tmax, 100.0)
    assert o["verdict"] == oracle.APERIODIC and o["n_peaks"] == 0


def test_plateau_contributes_its_first_lag():
    vals = [9, 8, 5, 3, 3, 3, 6, 9, 9, 9, 9, 9]
    s, tmin, tmax = row(10, vals)
    o = oracle.select(s, 1000, tmin, tmax, 20.0)
    assert o["n_peaks"] == 1
    assert o["t_cand"] == 13            # first lag of the flat bottom
    assert o["s_pk"] == 3.0


def test_rising_plateau_edge_is_not_a_peak():
    # S(T) == S(T-1) fails the strict left test
    vals = [5, 4, 4, 6, 7]
    s, tmin, tmax = row(2, vals)
    o = oracle.select(s, 1000, tmin, tmax, 20.0)
    assert o["n_peaks"] == 1 and o["t_cand"] == 3


def test_threshold_filters_shallow_peaks():
    r = 100.0
    vals = [90.0] * 60
    vals[10] = 50.0                    # T = 12: height 0.5
    vals[30] = 5.0                     # T = 32: height 0.95 -> S_pk
    s, tmin, tmax = row(2, vals)
    o = oracle.select(s, 10_000, tmin, tmax, r, c_lag=0.9)
    # thr = R - 0.9 (R - S_pk) = 100 - 0.9 * 95 = 14.5: only T = 32 passes
    assert o["s_pk"] == 5.0 and o["n_peaks"] == 2 and o["n_candidates"] == 1
    assert o["t_cand"] == 32 and o["period"] == 32
    # with a looser c_lag both pass and the smaller one is the fundamental
    o = oracle.select(s, 10_000, tmin, tmax, r, c_lag=0.4)
    assert o["n_candidates"] == 2 and o["t_cand"] == 12


def test_candidate_must_be_strictly_below_threshold():
    r = 10.0
    vals = [9.0] * 30
    vals[5] = 1.0                      # S_pk
    # value exactly at thr = 10 - 0.5 * 9 = 5.5 does not pass
    vals[15] = 5.5
    s, tmin, tmax = row(2, vals)
    o = oracle.select(s, 10_000, tmin, tmax, r, c_lag=0.5)
    assert o["n_candidates"] == 1 and o["t_cand"] == 7


def test_no_positive_peak_is_aperiodic():
    # every peak at or above R: thr <= S_pk, so nothing passes
    vals = [12.0, 11.0, 10.0, 11.0, 12.0]
    s, tmin, tmax = row(2, vals)
    o = oracle.select(s, 1000, tmin, tmax, 10.0)
    assert o["n_peaks"] == 1 and o["n_candidates"] == 0
    assert o["verdict"] == oracle.APERIODIC and o["period"] == 0


def test_equal_multiples_pick_the_fundamental():
    vals = [50.0] * 200
    for k in (1, 2, 3, 4):
        vals[25 * k - 2] = 1.0         # T = 25, 50, 75, 100 equally deep
    s, tmin, tmax = row(2, vals)
    o = oracle.select(s, 100_000, tmin, tmax, 100.0)
    assert o["n_candidates"] == 4 and o["t_cand"] == 25 and o["period"] == 25


def test_local_search_moves_to_lower_neighbour_and_ties_go_low():
    n = 1001                           # D = N - 1 = 1000
    vals = [80.0] * 199
    tmin = 2
    vals[100 - tmin] = 10.0            # T_c = 100 (a peak)
    vals[104 - tmin] = 9.0             # not a peak? 9 < 80 and 9 <= 80: also a peak, deeper
    s = np.asarray(vals)
    o = oracle.select(s, n, tmin, tmin + len(vals) - 1, 100.0)
    # peaks at 100 and 104; S_pk = 9 -> thr = 100 - 0.9*91 = 18.1: both pass, T_c = 100
    assert o["t_cand"] == 100
    # window for T_c = 100, D = 1000 (k = 10): [ceil(1000/11), floor(1000/9)] = [91, 111]
    assert (o["t_low"], o["t_up"]) == (91, 111)
    assert o["period"] == 104
    # tie inside the window goes to the smaller lag
    s2 = s.copy()
    s2[95 - tmin] = 9.0
    o2 = oracle.select(s2, n, tmin, tmin + len(vals) - 1, 100.0)
    assert o2["period"] == 95


def test_err_and_err_max_verdict():
    vals = [80.0] * 50
    vals[20] = 20.0
    s, tmin, tmax = row(2, vals)
    o = oracle.select(s, 10_000, tmin, tmax, 100.0)
    assert o["period"] == 22 and o["err"] == 0.2 and o["verdict"] == oracle.PERIODIC
    o = oracle.select(s, 10_000, tmin, tmax, 100.0, err_max=0.2)
    assert o["verdict"] == oracle.APERIODIC and o["period"] == 22


def _paper_window(t_c, n):
    """Algorithm 1's local-search bounds with T_s = 1, in the paper's own form."""
    n_t = Fraction(n - 1, t_c)
    lo = t_c * (1 - 1 / (n_t + 1))
    hi = t_c * (1 + 1 / (n_t - 1))
    return math.ceil(lo), math.floor(hi)


@pytest.mark.parametrize("n,t_c", [(1001, 100), (1001, 200), (1001, 250), (4096, 137),
                                   (65536, 4999), (262144, 20000), (16384, 900), (16384, 4095),
                                   (101, 49), (1001, 7), (16384, 2)])
def test_window_bounds_match_paper_formula(n, t_c):
    tmin, tmax = 1, n // 2
    vals = np.full(tmax - tmin + 1, 50.0)
    vals[t_c - tmin] = 1.0
    if t_c == tmin:
        pytest.skip("a peak cannot sit on Tmin")
    o = oracle.select(vals, n, tmin, tmax, 100.0)
    lo, hi = _paper_window(t_c, n)
    assert o["t_cand"] == t_c
    assert (o["t_low"], o["t_up"]) == (max(lo, tmin), min(hi, tmax))


@pytest.mark.parametrize("k", [3, 4, 5, 8, 10, 20, 40])
def test_window_is_the_neighbouring_fourier_bins(k):
    # T_c = D/k exactly: the window is [D/(k+1), D/(k-1)] rounded inwards
    d = 840 * 7                        # divisible by every k above
    n = d + 1
    t_c = d // k
    vals = np.full(n // 2, 50.0)
    vals[t_c - 1] = 1.0
    o = oracle.select(vals, n, 1, n // 2, 100.0)
    assert o["t_low"] == -(-d // (k + 1))
    assert o["t_up"] == min(d // (k - 1), n // 2)


# ----------------------------------------------------------------------------
# Planted periods through the whole oracle
# ----------------------------------------------------------------------------

def test_first_workload_selects_the_planted_period():
    wl = make_workload("w1")
    _, out = oracle.detect(wl.x, oracle.Layout.of(wl))
    assert out["period"][0] == 137 and out["verdict"][0] == oracle.PERIODIC


@pytest.mark.parametrize("period,k", [(5, 3), (64, 4), (301, 9)])
def test_noise_free_integer_period_selected_exactly(period, k):
    x = planted_trace(8192, period, k, seed=period, integer=True)
    lay = oracle.Layout(1, 1, 8192, 8192, 8192, 2, 2048)
    scores, out = oracle.detect(x, lay)
    assert out["period"][0] == period
    assert scores[0, period - 2] == 0.0


def test_small_spiky_workload_selects_planted_periods():
    wl = make_workload("w3", traces=6, n=16384, tmax=2048, pmax=1500)
    _, out = oracle.detect(wl.x, oracle.Layout.of(wl))
    assert np.array_equal(out["period"], wl.truth)


def test_small_multichannel_workload_selects_planted_periods():
    wl = make_workload("w5", traces=4, n=8192, tmax=1024, pmax=800)
    _, out = oracle.detect(wl.x, oracle.Layout.of(wl))
    assert np.array_equal(out["period"], wl.truth)


def test_small_jittered_workload_within_two_percent():
    wl = make_workload("w2", traces=8, n=16384, tmax=2048, pmax=1500)
    _, out = oracle.detect(wl.x, oracle.Layout.of(wl))
    assert np.all(np.abs(out["period"] - wl.truth) <= np.ceil(0.02 * wl.truth))


def test_small_sliding_window_workload():
    wl = make_workload("w4", total=65536, n=8192, stride=2048, tmax=2048, p1=300, p2=460)
    _, out = oracle.detect(wl.x, oracle.Layout.of(wl))
    defined = wl.truth > 0
    assert np.array_equal(out["period"][defined], wl.truth[defined])
