"""GPU parity of the FFT scores (GPOEO_PD_FFT_SCORES) against the fp64 oracle.

The FFT path promises every score within 1e-6 relative of the exact value
(lags its error bound cannot certify are re-scored in fp64 first), exact
zeros where the oracle has them, and selections identical to the oracle's.
Covered: the one-workgroup transform (up to 2048 points), the split one with
2048-point tiles and, beyond 2^20 points, with 4096-point tiles,
an odd number of sequences (one transform carries a single sequence),
weighted channels, exactly periodic windows (every multiple of the period
re-scored), a window table (rolling detection), scores only, determinism, and
the five workloads at full size (sampled windows against the oracle, every
window against the direct path).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from gen import make_workload, planted_trace  # noqa: E402

from test_gpu_parity import check_results, gpu_run  # noqa: E402

FFT_RTOL = 1e-6


def fft_flag():
    import paper_2201_01684_amd as pkg
    return pkg.FFT_SCORES


def check_fft_scores(g, o, where=""):
    assert g.shape == o.shape
    zero = o == 0
    assert np.all(g[zero] == 0), f"{where}: zero scores not reproduced"
    # g is the fp32 output: its own rounding (2^-24) on top of the 1e-6 bound
    rel = np.abs(g - o)[~zero] / np.abs(o[~zero])
    assert rel.size == 0 or rel.max() <= FFT_RTOL + 2.0 ** -24, f"{where}: rel {rel.max():.3e}"
    return float(rel.max()) if rel.size else 0.0


def fft_parity(x, lay, where="", flags=0):
    g, res = gpu_run(x, lay, flags=fft_flag() | flags)
    o, out = oracle.detect(x, lay)
    check_fft_scores(g, o, where)
    if res is not None:
        check_results(res, out, where)
    return g, res, out


def test_plan_modes():
    import paper_2201_01684_amd as pkg
    for n, tmax, mode in [(1500, 500, "single"), (4096, 1024, "split")]:
        desc, _ = pkg.make_desc(1, 1, n, n, n, 2, tmax, flags=fft_flag())
        assert pkg.describe_plan(desc)["mode"] == 2, mode


@pytest.mark.parametrize("n,tmin,tmax", [
    (8, 1, 4),            # smallest window: 64-point transform
    (1500, 2, 500),       # 2048 points: the largest one-workgroup transform
    (2000, 2, 1000),      # 4096 points: the smallest split transform
    (4096, 1, 2048),      # 8192 points
    (4099, 3, 2049),      # ragged N
    (3000, 1021, 1500),   # lag range far from zero
    (20000, 6, 3333),
])
def test_edge_shapes(n, tmin, tmax):
    x = planted_trace(n, max(3, min(97, n // 3)), 3, seed=n + tmin, sigma=1.0)
    fft_parity(x, oracle.Layout(1, 1, n, n, n, tmin, tmax), f"n={n} T=[{tmin},{tmax}]")


@pytest.mark.parametrize("name,kw", [
    ("w1", {}),
    ("w2", dict(traces=5, n=16384, tmax=2048, pmax=1500)),      # odd: one lone sequence
    ("w3", dict(traces=4, n=32768, tmax=4096, pmax=3000)),
    ("w4", dict(total=131072, n=16384, stride=2048, tmax=4096)),
    ("w5", dict(traces=3, n=16384, tmax=2048, pmax=1500)),
])
def test_reduced_workloads(name, kw):
    wl = make_workload(name, **kw)
    fft_parity(wl.x, oracle.Layout.of(wl), f"fft {name}{kw}")


def test_weighted_channels():
    rng = np.random.default_rng(3)
    b, c, n = 3, 3, 6000
    base = np.stack([planted_trace(n, 300 + 17 * k, 6, seed=k, sigma=0.5) for k in range(b)])
    x = np.stack([base * s + rng.normal(0, 0.3, size=(b, n)) for s in (1.0, 0.01, 30.0)], axis=1)
    lay = oracle.Layout(b, c, n, c * n, n, 2, 3000,
                        weights=np.array([1.0, 250.0, 0.003], dtype=np.float32))
    fft_parity(x.astype(np.float32), lay, "fft weighted")


def test_exact_periods_are_rescored_to_exact_zeros():
    n = 8192
    rows = [np.full(n, 123.25, dtype=np.float32),                         # CONSTANT
            planted_trace(n, 64, 4, seed=1, integer=True),                  # zeros at 64 k
            planted_trace(n, 301, 9, seed=2, sigma=0.0),                    # real-valued repeats
            np.random.default_rng(4).normal(0, 1, n).astype(np.float32),
            np.zeros(n, dtype=np.float32)]
    x = np.stack(rows)
    lay = oracle.Layout(len(rows), 1, n, n, n, 2, 4096)
    g, res, out = fft_parity(x, lay, "fft special windows")
    assert res["period"][1] == 64 and res["period"][2] == 301
    assert np.all(g[1, np.arange(64, 4097, 64) - 2] == 0)
    assert res["n_rescored"][1] >= 4096 // 64 and res["n_rescored"][2] >= 4096 // 301


def test_scores_only_and_no_rescue():
    import paper_2201_01684_amd as pkg
    wl = make_workload("w2", traces=4, n=16384, tmax=2048, pmax=1500)
    lay = oracle.Layout.of(wl)
    g, _ = gpu_run(wl.x, lay, flags=fft_flag() | pkg.SCORES_ONLY)
    o, out = oracle.detect(wl.x, lay)
    check_fft_scores(g, o, "fft scores only")
    _, res = gpu_run(wl.x, lay, flags=fft_flag() | pkg.NO_RESCUE)
    assert np.all(np.abs(res["period"] - out["period"]) <= 2)


def test_rolling_with_fft_scores():
    import paper_2201_01684_amd as pkg
    from test_gpu_rolling import check
    n = 12000
    rows = [planted_trace(n, 250, 7, seed=3, sigma=4.0),
            planted_trace(n, 137, 5, seed=4, integer=True),
            np.concatenate([planted_trace(11500, 200, 6, seed=5, sigma=1.0),
                            planted_trace(500, 290, 6, seed=6, sigma=1.0)]),
            planted_trace(n, 1900, 9, seed=7, sigma=2.0)]
    x = np.stack(rows).astype(np.float32)
    lay = oracle.Layout(len(rows), 1, n, n, n, 2, n // 2)
    xt = torch.from_numpy(x.reshape(-1)).to("cuda:0")
    desc, keep = pkg.make_desc(lay.num_windows, 1, n, n, n, 2, n // 2, flags=fft_flag())
    det = pkg.RollingDetector(xt, desc, pkg.rolling_params(), keep)
    det.run()
    torch.cuda.synchronize()
    check(det.results_numpy(), oracle.rolling(x, lay), "rolling fft")


def test_deterministic_bitwise():
    wl = make_workload("w3", traces=3, n=32768, tmax=4096, pmax=3000)
    lay = oracle.Layout.of(wl)
    a, ra = gpu_run(wl.x, lay, flags=fft_flag())
    b, rb = gpu_run(wl.x, lay, flags=fft_flag())
    assert np.array_equal(a, b) and np.array_equal(ra, rb)


@pytest.mark.parametrize("name", ["w1", "w2", "w3", "w4", "w5"])
def test_full_size(name):
    import paper_2201_01684_amd as pkg
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wl = make_workload(name)
    print(f"\n[fft {name}] {wl.num_windows} windows x {wl.num_channels} ch x {wl.n}", flush=True)
    x = torch.from_numpy(wl.x).to("cuda:0")
    out = {}
    for mode, flags in (("fft", fft_flag()), ("direct", 0)):
        desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                                   wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights,
                                   flags=flags)
        det = pkg.Detector(x, desc, keep)
        det.run()
        torch.cuda.synchronize()
        out[mode] = (det.scores.cpu().numpy(), det.results_numpy())
        del det
        torch.cuda.empty_cache()
    del x
    torch.cuda.empty_cache()
    gf, rf = out["fft"]
    gd, rd = out["direct"]
    assert np.all(rf["flags"] & pkg.UNRESOLVED == 0)
    for f in ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates"):
        assert np.array_equal(rf[f], rd[f]), f"{name}: {f} differs from the direct path"
    # both within their bounds of the exact scores: 2.5e-5 + 1e-6 (+ fp32 rounding)
    nz = gd != 0
    assert np.all(gf[~nz] == 0)
    assert np.all(np.abs(gf[nz].astype(np.float64) - gd[nz]) <= 2.7e-5 * np.abs(gd[nz]))
    rng = np.random.default_rng(99)
    lay1 = oracle.Layout.of(wl, num_windows=1)
    span = (wl.num_channels - 1) * wl.channel_stride + wl.n
    for b in sorted({0, int(rng.integers(0, wl.num_windows))}):
        sub = wl.x[b * wl.window_stride: b * wl.window_stride + span]
        o_scores, o_out = oracle.detect(sub, lay1)
        check_fft_scores(gf[b:b + 1].astype(np.float64), o_scores, f"fft {name} window {b}")
        check_results(rf[b:b + 1], o_out, f"fft {name} window {b}")


def plan_of(lay):
    import paper_2201_01684_amd as pkg
    desc, _ = pkg.make_desc(lay.num_windows, lay.num_channels, lay.n, lay.window_stride,
                            lay.channel_stride, lay.tmin, lay.tmax, weights=lay.weights,
                            flags=pkg.FFT_SCORES)
    info = pkg.describe_plan(desc)
    return info["fft_len"], info["fft_wrap_len"], info["fft_wrap_lags"]


@pytest.mark.parametrize("n,tmin,tmax,plan", [
    (16284, 2, 1000, (16384, 4096, 900)),      # lags 2..100 plain, 101..1000 wrapped
    (16384, 2001, 3000, (16384, 8192, 3000)),  # every lag wrapped
    (30000, 2, 2769, (32768, 4096, 1)),        # only Tmax wrapped
    (65536, 2, 16384, (65536, 32768, 16384)),  # wrap term of L / 4 lags: still taken
    (65536, 2, 16385, (131072, 0, 0)),         # one more lag: the padded transform
])
def test_wrap_correction_shapes(n, tmin, tmax, plan):
    x = planted_trace(n, 1013, 7, seed=n + tmax, sigma=1.5)
    lay = oracle.Layout(1, 1, n, n, n, tmin, tmax)
    assert plan_of(lay) == plan
    fft_parity(x, lay, f"wrap n={n} T=[{tmin},{tmax}]")


def test_wrap_correction_odd_channel_count():
    # three weighted channels: the last sequence has no partner in its transforms
    n = 8192
    x = np.stack([planted_trace(n, 700, 6, seed=31, sigma=1.0),
                  planted_trace(n, 700, 4, seed=32, sigma=0.1) * 40,
                  planted_trace(n, 350, 5, seed=33, sigma=2.0)])
    lay = oracle.Layout(1, 3, n, 3 * n, n, 2, 2048,
                        weights=np.array([1.0, 0.05, 3.0], dtype=np.float32))
    assert plan_of(lay) == (8192, 4096, 2048)
    fft_parity(x, lay, "wrap, 3 channels")


@pytest.mark.parametrize("n,tmax,plan", [
    # N + Tmax = 1,100,000 > 2^20 with N <= 2^20: a 2^20-point transform and a
    # wrap term of 51,424 lags from a 2^17-point head-tail transform
    (1_000_000, 100_000, (1 << 20, 1 << 17, 51_424)),
    # N > 2^20: a 2^21-point transform, row pairs of 2^11 points in 4096-point tiles
    (1_100_000, 100_000, (1 << 21, 0, 0)),
    # a 2^19-point head-tail transform: four rows of 2^10 points in a 4096-point tile
    (1 << 21, 200_000, (1 << 21, 1 << 19, 200_000)),
])
def test_large_transforms(n, tmax, plan):
    import paper_2201_01684_amd as pkg
    x = planted_trace(n, 3001, 9, seed=21, sigma=2.0)
    lay = oracle.Layout(1, 1, n, n, n, 2, tmax)
    assert plan_of(lay) == plan
    g, res = gpu_run(x, lay, flags=fft_flag())
    gd, rd = gpu_run(x, lay)
    for f in ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates"):
        assert np.array_equal(res[f], rd[f]), f
    assert res["period"][0] == 3001
    rng = np.random.default_rng(2)
    ts = np.concatenate([rng.integers(2, tmax + 1, size=48), [2, 3001, 6002, tmax]])
    w = plan[0] - n
    if plan[1]:   # the last plain lag and the first wrapped one (those in range)
        ts = np.concatenate([ts, np.array([t for t in (w, w + 1) if 2 <= t <= tmax],
                                          dtype=ts.dtype)])
    o = oracle.score_list(x, lay, np.zeros(ts.size, dtype=np.int64), ts)
    check_fft_scores(g[0, ts - 2], o, f"n={n} Tmax={tmax}")
