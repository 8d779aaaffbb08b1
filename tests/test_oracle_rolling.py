"""Pins of the oracle's Algorithm 3 (rolling detection over suffix windows)."""
import math
import os

import numpy as np
import pytest

import oracle
from gen import planted_trace

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "rolling_schedule.txt")


def golden_rows():
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        f = line.split()
        yield int(f[0]), int(f[1]), f[2:]


@pytest.mark.parametrize("n,t_init,want", list(golden_rows()))
def test_schedule_matches_hand_derivation(n, t_init, want):
    starts, short_next = oracle.rolling_schedule(n, t_init)
    if want and want[0].startswith("short:"):
        assert starts == [] and short_next == float(want[0].split(":")[1])
    else:
        assert starts == [int(v) for v in want] and short_next == 0.0


def test_default_schedule_has_seven_windows():
    # 5.25, 4.75, ..., 2.25 periods: the loop stops below c_measure = 2
    starts, _ = oracle.rolling_schedule(1_000_001, 1000)
    assert len(starts) == 7
    durations = [(1_000_000 - s) / 1000 for s in starts]
    assert durations == [5.25, 4.75, 4.25, 3.75, 3.25, 2.75, 2.25]


def brute_schedule(n, t_init, c_measure, step, c_eval):
    """Algorithm 3's suffix starts by enumeration in exact rationals: start at
    (2 + c_eval step) periods before the end (at least sample 0) and move on by
    step periods while at least c_measure periods remain."""
    from fractions import Fraction as F
    d, t = F(n - 1), F(t_init)
    cm, st, ce = F(c_measure), F(step), F(c_eval)
    if d < cm * t:
        return [], float(cm * t - d)
    s = max(F(0), d - (2 + ce * st) * t)
    out = []
    while d - s >= cm * t:
        out.append(math.floor(s))
        s += st * t
    return out, 0.0


def test_schedule_matches_enumeration_for_other_constants():
    # dyadic constants: every quantity of the schedule is exact in fp64, so
    # the oracle must equal the rational enumeration exactly
    rng = np.random.default_rng(11)
    for _ in range(3000):
        n = int(rng.integers(2, 2_000_000))
        t_init = int(rng.integers(1, max(2, n // 2)))
        cm = float(rng.choice([1.0, 1.5, 2.0, 3.0]))
        st = float(rng.choice([0.25, 0.5, 0.75, 1.0, 1.5]))
        ce = float(rng.choice([0.0, 2.5, 6.5, 12.0]))
        want = brute_schedule(n, t_init, cm, st, ce)
        if len(want[0]) > oracle.ROLLING_MAX:
            continue
        assert oracle.rolling_schedule(n, t_init, cm, st, ce) == want, (n, t_init, cm, st, ce)


def lay1(n, tmax, tmin=2):
    return oracle.Layout(1, 1, n, n, n, tmin, tmax)


@pytest.mark.parametrize("period,n", [(100, 10001), (37, 1001), (64, 131)])
def test_stable_exact_period(period, n):
    x = planted_trace(n, period, 4, seed=period, integer=True)
    o = oracle.rolling(x, lay1(n, n // 2))[0]
    starts, _ = oracle.rolling_schedule(n, period)
    assert o["t_init"] == period and o["verdict"] == oracle.PERIODIC
    assert o["n_windows"] == len(starts)
    assert list(o["starts"][: o["n_windows"]]) == starts
    assert np.all(o["periods"][: o["n_windows"]] == period)
    assert o["stable"] == 1 and o["smpdur_next"] == -1.0 and o["diff"] == 0.0
    assert o["period"] == period


def test_best_window_has_the_smallest_err():
    x = planted_trace(20000, 250, 7, seed=3, sigma=4.0)
    o = oracle.rolling(x, lay1(20000, 4000))[0]
    k = o["n_windows"]
    assert k == 7
    periodic = o["verdicts"][:k] == oracle.PERIODIC
    errs = np.where(periodic, o["errs"][:k], np.inf)
    assert o["best"] == int(np.argmin(errs))          # first minimum on ties
    assert o["period"] == o["periods"][o["best"]] and o["err"] == errs.min()


def test_regime_switch_is_not_stable():
    # 200-sample iterations, then 290-sample iterations over the last 1200 samples
    head = planted_trace(6000, 200, 6, seed=5, sigma=1.0)
    tail = planted_trace(1200, 290, 6, seed=6, sigma=1.0)
    x = np.concatenate([head, tail]).astype(np.float32)
    n = x.size
    o = oracle.rolling(x, lay1(n, n // 2))[0]
    k = o["n_windows"]
    p = o["periods"][:k][o["verdicts"][:k] == oracle.PERIODIC]
    assert p.min() != p.max()
    diff = abs((p.max() - p.min()) / p.mean())
    assert o["diff"] == pytest.approx(diff, rel=1e-12) and diff >= 0.05
    d = n - 1
    assert o["stable"] == 0
    assert o["smpdur_next"] == math.ceil(d / p.max()) * p.max() - d


def test_aperiodic_first_pass_has_no_windows():
    x = np.full(4000, 7.0, dtype=np.float32)
    o = oracle.rolling(x, lay1(4000, 2000))[0]
    assert o["verdict"] == oracle.CONSTANT and o["n_windows"] == 0 and o["period"] == 0


def test_threshold_parameter_decides_stability():
    head = planted_trace(6000, 200, 6, seed=5, sigma=1.0)
    tail = planted_trace(1200, 290, 6, seed=6, sigma=1.0)
    x = np.concatenate([head, tail]).astype(np.float32)
    o = oracle.rolling(x, lay1(x.size, x.size // 2), diff_threshold=10.0)[0]
    assert o["stable"] == 1 and o["smpdur_next"] == -1.0
