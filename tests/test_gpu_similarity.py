"""GPU parity of Algorithm 2's grouped similarity against the oracle.

Tolerance: 1e-6 relative.  Both sides evaluate the mixture in fp64, but with
their own exp/log and different summation orders, so the fitted parameters
differ in the last bits; the hard groups (and so the errors) agree unless a
sample sits within that distance of a group boundary.  -1 (fewer than two
sub-curves) and exact zeros must match exactly.
"""
from fractions import Fraction

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from gen import make_workload, planted_trace  # noqa: E402


def gpu_similarity(x_np, lay, windows, lags, **kw):
    import paper_2201_01684_amd as pkg
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    x = torch.from_numpy(np.ascontiguousarray(x_np).reshape(-1)).to("cuda:0")
    desc, _keep = pkg.make_desc(lay.num_windows, lay.num_channels, lay.n, lay.window_stride,
                                lay.channel_stride, lay.tmin, lay.tmax, weights=lay.weights)
    w = torch.tensor(np.asarray(windows, dtype=np.int32), device="cuda:0")
    t = torch.tensor(np.asarray(lags, dtype=np.int32), device="cuda:0")
    out = pkg.similarity(x, desc, w, t, **kw)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check(g, o, where):
    assert np.array_equal(g == -1.0, o == -1.0), where
    assert np.array_equal(g == 0.0, o == 0.0), where
    nz = o > 0
    rel = np.abs(g[nz] - o[nz]) / o[nz]
    assert rel.size == 0 or rel.max() <= 1e-6, f"{where}: rel {rel.max():.3e}"


def test_hand_worked_example():
    x = np.array([0, 0, 10, 10, 20, 20, 0, 1, 10, 12, 20, 20], dtype=np.float32)
    lay = oracle.Layout(1, 1, 12, 12, 12, 1, 6)
    g = gpu_similarity(x, lay, [0, 0, 0], [6, 7, 3])
    assert g[0] == pytest.approx(float(Fraction(80, 117)), rel=1e-12)
    assert g[1] == -1.0
    check(g, oracle.similarity(x, lay, [0, 0, 0], [6, 7, 3]), "hand")


@pytest.mark.parametrize("name,kw", [
    ("w1", {}),
    ("w3", dict(traces=3, n=32768, tmax=4096, pmax=3000)),
    ("w5", dict(traces=2, n=8192, tmax=1024, pmax=800)),
])
@pytest.mark.parametrize("groups,iters", [(3, 20), (1, 5), (5, 30)])
def test_finalists_match_oracle(name, kw, groups, iters):
    wl = make_workload(name, **kw)
    lay = oracle.Layout.of(wl)
    rng = np.random.default_rng(7)
    ws, ts = [], []
    for b in range(wl.num_windows):
        p = int(wl.truth[b])
        for t in (p, p - 1, p + 1, 2 * p, max(1, p // 2), int(rng.integers(2, wl.tmax))):
            ws.append(b)
            ts.append(t)
    ws.append(0)
    ts.append(wl.n // 2 + 1)          # one sub-curve only: -1
    g = gpu_similarity(wl.x, lay, ws, ts, num_groups=groups, em_iters=iters)
    o = oracle.similarity(wl.x, lay, ws, ts, num_groups=groups, em_iters=iters)
    check(g, o, f"{name} G={groups} it={iters}")
    if groups == 1:
        assert np.all(o[:-1] == 0.0)      # one group: relative group values are all 0
        return
    # the planted period scores best among its neighbours
    k = 0
    for b in range(wl.num_windows):
        assert o[k] < o[k + 1] and o[k] < o[k + 2]
        k += 6


def test_exact_period_zero_and_out_of_range():
    x = planted_trace(4000, 125, 5, seed=1, integer=True)
    lay = oracle.Layout(1, 1, 4000, 4000, 4000, 2, 2000)
    g = gpu_similarity(x, lay, [0, 0, 1, 0, 0], [125, 250, 125, 0, 4001])
    assert g[0] == 0.0 and g[1] == 0.0
    assert np.isnan(g[2]) and np.isnan(g[3]) and np.isnan(g[4])


def test_weighted_channels():
    a = planted_trace(3000, 100, 6, seed=2, sigma=2.0)
    b = planted_trace(3000, 100, 4, seed=3, sigma=0.1)
    x = np.stack([a, b]).astype(np.float32)
    lay = oracle.Layout(1, 2, 3000, 6000, 3000, 2, 1500,
                        weights=np.array([0.25, 3.0], dtype=np.float32))
    ts = [100, 101, 150, 300, 7]
    check(gpu_similarity(x, lay, [0] * 5, ts), oracle.similarity(x, lay, [0] * 5, ts), "weights")


def gpu_similarity_flagged(x_np, lay, windows, lags, **kw):
    import paper_2201_01684_amd as pkg
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    x = torch.from_numpy(np.ascontiguousarray(x_np).reshape(-1)).to("cuda:0")
    desc, _keep = pkg.make_desc(lay.num_windows, lay.num_channels, lay.n, lay.window_stride,
                                lay.channel_stride, lay.tmin, lay.tmax, weights=lay.weights)
    w = torch.tensor(np.asarray(windows, dtype=np.int32), device="cuda:0")
    t = torch.tensor(np.asarray(lags, dtype=np.int32), device="cuda:0")
    err, flags = pkg.similarity(x, desc, w, t, with_flags=True, **kw)
    plain = pkg.similarity(x, desc, w, t, **kw)
    torch.cuda.synchronize()
    assert torch.equal(err, plain)          # the flags change nothing else
    return err.cpu().numpy(), flags.cpu().numpy()


def test_sample_on_a_group_boundary_is_flagged():
    """A sub-curve symmetric about 5 (eight samples at 0, eight at 10, one at 5)
    keeps a two-component fit symmetric, so the sample at 5 sits exactly on the
    boundary: its label is a tie that rounding decides, and the query is
    flagged.  Moving that sample off the middle clears the flag."""
    import paper_2201_01684_amd as pkg
    sub = [0.0] * 8 + [5.0] + [10.0] * 8
    for mid, want in ((5.0, pkg.UNRESOLVED), (3.0, 0)):
        a = np.array(sub, dtype=np.float32)
        a[8] = mid
        x = np.concatenate([a, a + 1.0]).astype(np.float32)
        lay = oracle.Layout(1, 1, x.size, x.size, x.size, 1, x.size // 2)
        err, flags = gpu_similarity_flagged(x, lay, [0], [a.size], num_groups=2, em_iters=20)
        assert flags[0] == want, (mid, flags)
        check(err, oracle.similarity(x, lay, [0], [a.size], num_groups=2, em_iters=20),
              f"boundary {mid}")


@pytest.mark.parametrize("name,kw", [
    ("w1", {}),
    ("w2", dict(traces=8, n=65536, tmax=8192)),
    ("w3", dict(traces=6, n=262144, tmax=32768)),
    ("w5", dict(traces=3, n=131072, tmax=16384)),
])
def test_workload_finalists_unflagged_and_equal(name, kw):
    """The five finalists of each window (the planted period, its neighbours,
    its double and half) at full window length: no query flagged, every Err
    equal to the oracle's within 1e-6."""
    wl = make_workload(name, **kw)
    lay = oracle.Layout.of(wl)
    ws, ts = [], []
    for b in range(wl.num_windows):
        p = int(wl.truth[b])
        for t in (p, p - 1, p + 1, 2 * p, max(1, p // 2)):
            ws.append(b)
            ts.append(t)
    err, flags = gpu_similarity_flagged(wl.x, lay, ws, ts)
    assert not flags.any(), f"{name}: flagged queries {np.nonzero(flags)[0][:10]}"
    check(err, oracle.similarity(wl.x, lay, ws, ts), name)
