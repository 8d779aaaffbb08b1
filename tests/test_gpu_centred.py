"""GPU parity of the mean-removed score S_c(T) (gpoeo_pd_score_centred) against
the oracle.

Tolerance: 1e-9 relative.  Both sides evaluate the definition in fp64, the
oracle with sequential sums and the GPU with per-lane partial sums; the two
orders differ by a few ulps of each sub-curve mean and of each pair sum,
which is far below 1e-9 of a score unless the score is itself within ~1e-7 of
cancelling to zero.  Exact zeros (identical or drift-shifted sub-curves whose
means are exact) and the -1 / NaN markers must match exactly.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from gen import make_workload, planted_trace  # noqa: E402

RTOL = 1e-9


def gpu_centred(x_np, lay, windows, lags):
    import paper_2201_01684_amd as pkg
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    x = torch.from_numpy(np.ascontiguousarray(x_np).reshape(-1)).to("cuda:0")
    desc, _keep = pkg.make_desc(lay.num_windows, lay.num_channels, lay.n, lay.window_stride,
                                lay.channel_stride, lay.tmin, lay.tmax, weights=lay.weights)
    w = torch.tensor(np.asarray(windows, dtype=np.int32), device="cuda:0")
    t = torch.tensor(np.asarray(lags, dtype=np.int32), device="cuda:0")
    out = pkg.score_centred(x, desc, w, t)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check(g, o, where):
    assert np.array_equal(g == 0.0, o == 0.0), where
    nz = o != 0
    rel = np.abs(g[nz] - o[nz]) / np.abs(o[nz])
    assert rel.size == 0 or rel.max() <= RTOL, f"{where}: rel {rel.max():.3e}"


def test_every_lag_of_small_windows():
    rng = np.random.default_rng(0)
    x = rng.normal(50, 7, size=(2, 257)).astype(np.float32)
    lay = oracle.Layout(2, 1, 257, 257, 257, 1, 128, centred=True)
    ws = [b for b in range(2) for _ in range(1, 129)]
    ts = [t for _ in range(2) for t in range(1, 129)]
    check(gpu_centred(x, lay, ws, ts), oracle.score_list(x, lay, ws, ts), "small")


def test_markers_for_short_and_invalid_queries():
    x = planted_trace(1000, 37, 4, seed=3)
    lay = oracle.Layout(1, 1, 1000, 1000, 1000, 2, 500, centred=True)
    g = gpu_centred(x, lay, [0, 0, 0, 1, 0, -1], [500, 501, 1000, 37, 0, 37])
    assert g[0] >= 0.0 and g[1] == -1.0 and g[2] == -1.0
    assert np.isnan(g[3]) and np.isnan(g[4]) and np.isnan(g[5])


@pytest.mark.parametrize("period,slope", [(64, 1), (256, -3)])
def test_integer_drift_gives_exact_zeros(period, slope):
    base = planted_trace(50 * period, period, 5, seed=period, integer=True).astype(np.int64)
    x = (base + slope * np.arange(base.size)).astype(np.float32)
    n = x.size
    lay = oracle.Layout(1, 1, n, n, n, 2, n // 2, centred=True)
    ts = [period, 2 * period, 3 * period, period + 1, period - 1, 7]
    g = gpu_centred(x, lay, [0] * len(ts), ts)
    assert np.all(g[:3] == 0.0) and np.all(g[3:] > 0.0)
    check(g, oracle.score_list(x, lay, [0] * len(ts), ts), "drift")


@pytest.mark.parametrize("name,kw", [
    ("w1", {}),
    ("w2", dict(traces=4, n=16384, tmax=2048, pmax=1500)),
    ("w3", dict(traces=3, n=32768, tmax=4096, pmax=3000)),
    ("w5", dict(traces=2, n=8192, tmax=1024, pmax=800)),
])
def test_finalists_match_oracle(name, kw):
    wl = make_workload(name, **kw)
    lay = oracle.Layout.of(wl, centred=True)
    rng = np.random.default_rng(5)
    ws, ts = [], []
    for b in range(wl.num_windows):
        p = int(wl.truth[b])
        for t in (p, p - 1, p + 1, 2 * p, max(1, p // 2), int(rng.integers(1, wl.n // 2))):
            ws.append(b)
            ts.append(t)
    check(gpu_centred(wl.x, lay, ws, ts), oracle.score_list(wl.x, lay, ws, ts), name)


def test_drifting_windows_rank_the_true_period_first():
    # the centred score re-ranks candidate periods of drifting traces: at the
    # planted period the drift vanishes, at its neighbours it does not
    n, p = 16384, 400
    rows = []
    for k, slope in enumerate((0.0, 0.02, 0.1)):
        base = planted_trace(n, p, 6, seed=20 + k, sigma=1.0).astype(np.float64)
        rows.append((base + slope * np.arange(n)).astype(np.float32))
    x = np.stack(rows)
    lay = oracle.Layout(3, 1, n, n, n, 2, n // 2, centred=True)
    cands = [p - 2, p - 1, p, p + 1, p + 2]
    ws = [b for b in range(3) for _ in cands]
    ts = [t for _ in range(3) for t in cands]
    g = gpu_centred(x, lay, ws, ts).reshape(3, len(cands))
    check(g.reshape(-1), oracle.score_list(x, lay, ws, ts), "drifting")
    assert np.all(np.argmin(g, axis=1) == 2)


@pytest.mark.parametrize("name", ["w3", "w5"])
def test_full_size_finalists(name):
    wl = make_workload(name)
    lay = oracle.Layout.of(wl, centred=True)
    ws, ts = [], []
    for b in range(wl.num_windows):
        p = int(wl.truth[b])
        for t in (p, p - 1, p + 1, 2 * p, max(1, p // 2)):
            ws.append(b)
            ts.append(t)
    g = gpu_centred(wl.x, lay, ws, ts)
    assert np.all(np.isfinite(g)) and np.all(g >= 0.0)
    pick = np.random.default_rng(3).choice(len(ws), size=40, replace=False)
    o = oracle.score_list(wl.x, lay, np.asarray(ws)[pick], np.asarray(ts)[pick])
    check(g[pick], o, f"{name} sample")
