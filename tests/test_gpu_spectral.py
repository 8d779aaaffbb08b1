"""GPU parity of the FFT front end (gpoeo_pd_spectral_candidates) against the oracle.

Every window the GPU leaves unflagged must list exactly the oracle's
candidates: same bins, same periods, same order, and amplitudes within 1e-9
relative (both are fp64 transforms; the oracle uses numpy's FFT).  The test
inputs must leave no window flagged.  Covered: one-workgroup and split
transforms, an odd number of sequences, several channels with weights, pure
tones, the lag range, the threshold and the candidate limit, the five
workloads (reduced) and the 1024-trace workload at full size on sampled
windows.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from gen import make_workload, planted_trace  # noqa: E402


def gpu_spectral(x_np, num_windows, num_channels, n, window_stride, channel_stride, tmin, tmax,
                 weights=None, c_peak=0.65, k_max=16):
    import paper_2201_01684_amd as pkg
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    x = torch.from_numpy(np.ascontiguousarray(x_np, dtype=np.float32).reshape(-1)).to("cuda:0")
    desc, keep = pkg.make_desc(num_windows, num_channels, n, window_stride, channel_stride, tmin,
                               tmax, weights=weights)
    det = pkg.SpectralDetector(x, desc, pkg.spectral_params(c_peak, k_max), keep)
    det.run()
    torch.cuda.synchronize()
    return det.results_numpy()


def check(res, x_np, windows, num_channels, n, window_stride, channel_stride, tmin, tmax,
          weights=None, c_peak=0.65, k_max=16, where=""):
    x_np = np.ascontiguousarray(x_np, dtype=np.float32).reshape(-1)
    flagged = int(np.count_nonzero(res["flags"]))
    assert flagged == 0, f"{where}: {flagged} windows flagged"
    for b in windows:
        base = b * window_stride
        xw = np.stack([x_np[base + c * channel_stride: base + c * channel_stride + n]
                       for c in range(num_channels)])
        o = oracle.spectral_candidates(xw, tmin, tmax, c_peak, k_max, weights)
        r = res[b]
        cnt = int(r["count"])
        assert cnt == len(o["periods"]), f"{where} window {b}: {cnt} vs {len(o['periods'])}"
        assert list(r["bins"][:cnt]) == o["bins"], f"{where} window {b}"
        assert list(r["periods"][:cnt]) == o["periods"], f"{where} window {b}"
        assert np.allclose(r["amplitudes"][:cnt], o["amplitudes"], rtol=1e-9, atol=0), where
        # (the count of all peaks is not compared: peaks of rounding-noise bins
        # far below the threshold depend on the rounding and decide nothing)
        assert r["max_peak"] == pytest.approx(o["max_peak"], rel=1e-9), where


@pytest.mark.parametrize("n", [100, 2048, 4096, 65536])
def test_tones_and_planted_traces(n):
    rows = [planted_trace(n, max(5, n // 37), 5, seed=n, sigma=1.0),
            (100 + 20 * np.sin(2 * np.pi * np.arange(n) / (n / 8) + 0.1)).astype(np.float32),
            planted_trace(n, max(3, n // 11), 3, seed=n + 1, integer=True)]
    x = np.stack(rows)
    res = gpu_spectral(x, 3, 1, n, n, n, 2, n // 2)
    check(res, x, range(3), 1, n, n, n, 2, n // 2, where=f"n={n}")


def test_channels_weights_range_and_limit():
    n = 8192
    chans = [planted_trace(n, 300, 6, seed=1, sigma=2.0), planted_trace(n, 300, 4, seed=2),
             planted_trace(n, 75, 5, seed=3, sigma=0.5)]
    x = np.stack([np.stack(chans), np.stack(chans[::-1])])      # 2 windows x 3 channels
    w = np.array([1.0, 0.3, 2.5], dtype=np.float32)
    for tmin, tmax, c_peak, k_max in [(2, 4096, 0.65, 16), (50, 1000, 0.3, 4), (2, 100, 0.2, 16)]:
        res = gpu_spectral(x, 2, 3, n, 3 * n, n, tmin, tmax, w, c_peak, k_max)
        check(res, x, range(2), 3, n, 3 * n, n, tmin, tmax, w, c_peak, k_max,
              where=f"T=[{tmin},{tmax}] c={c_peak} K={k_max}")


def test_maximum_channel_count():
    rng = np.random.default_rng(12)
    b, c, n = 2, 256, 3000
    x = np.empty((b, c, n), dtype=np.float32)
    for k in range(c):
        x[0, k] = planted_trace(n, 150, 4, seed=200 + k, sigma=1.0) * (1 + k % 5)
        x[1, k] = rng.normal(0, 1, n) + np.sin(2 * np.pi * np.arange(n) / 40.0) * (k % 3)
    w = (0.2 + rng.random(c)).astype(np.float32)
    res = gpu_spectral(x, b, c, n, c * n, n, 2, n // 2, w)
    check(res, x, range(b), c, n, c * n, n, 2, n // 2, w, where="256 channels")


@pytest.mark.parametrize("name,kw", [
    ("w1", {}),
    ("w2", dict(traces=5, n=16384, tmax=2048, pmax=1500)),
    ("w3", dict(traces=4, n=32768, tmax=4096, pmax=3000)),
    ("w4", dict(total=65536, n=16384, stride=2048, tmax=4096)),
    ("w5", dict(traces=3, n=16384, tmax=2048, pmax=1500)),
])
def test_reduced_workloads(name, kw):
    wl = make_workload(name, **kw)
    res = gpu_spectral(wl.x, wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                       wl.channel_stride, wl.tmin, wl.tmax, wl.weights)
    check(res, wl.x, range(wl.num_windows), wl.num_channels, wl.n, wl.window_stride,
          wl.channel_stride, wl.tmin, wl.tmax, wl.weights, where=name)


def test_full_size_sampled_windows():
    wl = make_workload("w3")
    res = gpu_spectral(wl.x, wl.num_windows, 1, wl.n, wl.window_stride, wl.channel_stride,
                       wl.tmin, wl.tmax)
    picks = sorted({0, wl.num_windows - 1, *np.random.default_rng(5).integers(0, 1024, 6).tolist()})
    check(res, wl.x, picks, 1, wl.n, wl.window_stride, wl.channel_stride, wl.tmin, wl.tmax,
          where="w3 full")
    # the planted period's fundamental bin (L / P rounded) is among the candidates
    hits = 0
    for b in range(wl.num_windows):
        cnt = int(res["count"][b])
        if any(abs(int(t) - int(wl.truth[b])) <= max(1, wl.truth[b] // 50)
               for t in res["periods"][b][:cnt]):
            hits += 1
    assert hits >= 0.5 * wl.num_windows
