"""Property-based pins of the oracle (hypothesis, random tiny inputs).

Checked against what the definition fixes rather than against the oracle's own
formula:
- the score against the exact rational value (fractions) of the definition,
  within n * 2^-53 relative, and exact zeros;
- invariances that hold exactly: a constant offset on integer-valued data,
  scaling by a power of two (scores by its square), time reversal of
  integer-valued data;
- the selection rule's invariance under scaling all scores and R by a power
  of two (every comparison and threshold scales exactly while the values stay
  normal numbers).
"""
from fractions import Fraction

import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
from oracle import brute

SETTINGS = settings(max_examples=60, deadline=None)

floats32 = st.floats(min_value=-1e3, max_value=1e3, allow_nan=False, allow_infinity=False,
                     width=32)


@SETTINGS
@given(st.lists(floats32, min_size=4, max_size=24))
def test_score_is_the_exact_definition(values):
    x = np.asarray(values, dtype=np.float32)
    n = x.size
    for t in range(0, n // 2 + 1):
        exact = brute.exact_score(x, t)
        got = oracle.score(x, t)
        if exact == 0:
            assert got == 0.0
        else:
            assert abs(Fraction(got) - exact) / exact <= n * 2.0 ** -53


@SETTINGS
@given(st.lists(st.integers(-500, 500), min_size=6, max_size=40), st.integers(-1000, 1000),
       st.integers(-3, 3))
def test_exact_invariances_on_integer_data(values, offset, k):
    x = np.asarray(values, dtype=np.float32)
    shifted = (x.astype(np.float64) + offset).astype(np.float32)
    scaled = (x.astype(np.float64) * 2.0 ** k).astype(np.float32)
    reversed_ = x[::-1].copy()
    for t in range(0, x.size // 2 + 1):
        s = oracle.score(x, t)
        assert oracle.score(shifted, t) == s
        assert oracle.score(scaled, t) == s * 4.0 ** k
        assert oracle.score(reversed_, t) == s


# scores of zero or well inside the normal range, where scaling by 2^k is exact
scores = st.one_of(st.just(0.0), st.floats(min_value=1e-200, max_value=100.0))


@SETTINGS
@given(st.lists(scores, min_size=5, max_size=60),
       st.floats(min_value=1.0, max_value=300.0), st.integers(-20, 20),
       st.sampled_from([0.5, 0.65, 0.9]))
def test_selection_scales_with_the_scores(values, r, k, c_lag):
    s = np.asarray(values, dtype=np.float64)
    tmin = 2
    tmax = tmin + s.size - 1
    n = 4 * tmax
    a = oracle.select(s, n, tmin, tmax, r, c_lag)
    b = oracle.select(s * 2.0 ** k, n, tmin, tmax, r * 2.0 ** k, c_lag)
    for f in ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates", "n_peaks"):
        assert a[f] == b[f], f
    assert a["err"] == b["err"]
