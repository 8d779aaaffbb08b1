"""Pins of the oracle's Algorithm 2 similarity error (GMM groups + SMAPE).

The paper prints no worked example, and the EM details of the Gaussian mixture
(initialisation, iterations) are not given there and are fixed here.  Pinned: cases whose
answer does not depend on those details (well-separated clusters, which any
mixture fit recovers; a single group; exact periods; the invariances of the
definition), and the EM trajectory itself on overlapping clusters against
scikit-learn's GaussianMixture started from the same parameters.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from gen import planted_trace


def lay(n, channels=1, weights=None):
    return oracle.Layout(1, channels, n, channels * n, n, 1, n // 2, weights=weights)


def err(x, t, **kw):
    x = np.atleast_2d(np.asarray(x, dtype=np.float32))
    c, n = x.shape
    w = kw.pop("weights", None)
    return oracle.similarity(x, lay(n, c, w), [0], [t], **kw)[0]


def test_hand_worked_three_cluster_example():
    # sub-curve 1 = [0 0 10 10 20 20], sub-curve 2 = [0 1 10 12 20 20]
    # means 10 and 10.5; groups {0,1} {2,3} {4,5}:
    #   RelVal  (-10, -10)  (0, 0.5)  (10, 9.5)
    #   SMAPE    0           2         0.5 / 9.75
    # Err = (2 * 0 + 2 * 2 + 2 * 0.5 / 9.75) / 6 = 80 / 117
    x = [0, 0, 10, 10, 20, 20, 0, 1, 10, 12, 20, 20]
    assert err(x, 6) == pytest.approx(float(Fraction(80, 117)), rel=1e-12)


def test_smape_zero_over_zero_and_single_group():
    x = np.random.default_rng(1).normal(5, 2, size=600).astype(np.float32)
    # one group: group mean == sub-curve mean on both sides, SMAPE(0, 0) := 0
    assert err(x, 100, num_groups=1) == 0.0


@pytest.mark.parametrize("period", [7, 50, 137])
def test_exact_period_has_zero_error(period):
    x = planted_trace(40 * period + 3, period, 5, seed=period, integer=True)
    assert err(x, period) == 0.0
    assert err(x, period + 1) > 0.0


def test_too_few_sub_curves_is_undefined():
    x = np.arange(100, dtype=np.float32)
    assert err(x, 51) == -1.0
    assert err(x, 50) >= 0.0


def test_constant_sub_curves():
    x = np.full(300, 4.0, dtype=np.float32)
    assert err(x, 60) == 0.0


def test_offset_and_scale_invariance_on_clustered_data():
    rng = np.random.default_rng(2)
    levels = np.array([0.0, 10.0, 20.0])
    base = np.tile(np.repeat(levels, [5, 7, 8]), 12) + rng.normal(0, 0.3, size=240)
    x = (np.round(base * 64) / 64).astype(np.float32)   # on a 1/64 grid: x + 1000 is exact
    e = err(x, 20)
    assert err(x + np.float32(1000), 20) == pytest.approx(e, rel=1e-9)
    assert err(x * np.float32(4), 20) == pytest.approx(e, rel=1e-9)


def test_channel_weighting():
    a = np.array([0, 0, 10, 10, 20, 20, 0, 1, 10, 12, 20, 20], dtype=np.float32)
    b = np.array([3, 4, 5, 6, 7, 8] * 2, dtype=np.float32)     # identical sub-curves: 0
    w = np.array([2.0, 6.0], dtype=np.float32)
    got = err(np.stack([a, b]), 6, weights=w)
    assert got == pytest.approx(2.0 / 8.0 * 80 / 117, rel=1e-12)


def test_paper_reason_for_groups_noise_robustness():
    # High-frequency noise on an exact period: grouped means average it out,
    # so the true period still scores far better than a wrong one.
    x = planted_trace(8000, 200, 6, seed=9, sigma=8.0)
    assert err(x, 200) < 0.5 * err(x, 230)


def _err_via_sklearn(x, t, groups=3, iters=20):
    """Algorithm 2's Err_T with the mixture fitted by scikit-learn's EM from the
    same initial parameters (means evenly spread over [min, max], variances
    ((max-min)/G)^2, weights 1/G; no regularisation, no early stop), then hard
    labels, relative group means and SMAPE written out here."""
    from sklearn.mixture import GaussianMixture
    v = x.astype(np.float64)
    pairs = v.size // t - 1
    total = 0.0
    for i in range(pairs):
        a, b = v[i * t:(i + 1) * t], v[(i + 1) * t:(i + 2) * t]
        lo, hi = a.min(), a.max()
        width = (hi - lo) / groups
        gm = GaussianMixture(n_components=groups, covariance_type="full", max_iter=iters, tol=0.0,
                             reg_covar=0.0, weights_init=np.full(groups, 1.0 / groups),
                             means_init=(lo + (np.arange(groups) + 0.5) * width).reshape(-1, 1),
                             precisions_init=np.full((groups, 1, 1), 1.0 / width ** 2))
        gm.fit(a.reshape(-1, 1))
        labels = gm.predict(a.reshape(-1, 1))
        err = 0.0
        for k in range(groups):
            sel = labels == k
            if not sel.any():
                continue
            ra, rb = a[sel].mean() - a.mean(), b[sel].mean() - b.mean()
            den = (abs(ra) + abs(rb)) / 2
            err += sel.sum() * (0.0 if den == 0 else abs(ra - rb) / den)
        total += err / t
    return total / pairs


@pytest.mark.filterwarnings("ignore::sklearn.exceptions.ConvergenceWarning")
@pytest.mark.parametrize("t,seed", [(40, 1), (75, 2), (150, 3)])
def test_em_trajectory_matches_scikit_learn(t, seed):
    # overlapping clusters (levels 0, 3, 7 with sigma 1.2): twenty EM iterations
    # that move the mixture far from its initialisation; the variance floor
    # (1e-6 of the initial variance) never binds here
    rng = np.random.default_rng(seed)
    levels = np.repeat([0.0, 3.0, 7.0], [t // 3, t // 3, t - 2 * (t // 3)])
    x = (np.tile(levels, 12) + rng.normal(0, 1.2, size=12 * t)).astype(np.float32)
    want = _err_via_sklearn(x, t)
    assert err(x, t) == pytest.approx(want, rel=1e-9)
