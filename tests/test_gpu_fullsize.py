"""GPU parity at the five workloads' full sizes, in the launch configuration the
bench times (one gpoeo_pd_detect over the whole batch).

Every window of w1, w2 and w4 is checked against the oracle (every lag's score
and the full selection: the oracle needs seconds for these batches).  The
oracle cannot score every window of w3 and w5 in test time, so for them it
checks whole windows sampled from the batch (first, last and seeded random
ones).  On every batch it also checks seeded random (window, lag) scores.
Properties that hold at any size are checked on every window: the planted
period is selected (within 2% for the length-jittered batch), no window is
flagged UNRESOLVED, and every score is finite and non-negative.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from gen import make_workload  # noqa: E402

from test_gpu_parity import check_results, check_scores  # noqa: E402

WHOLE_WINDOWS = {"w3": 8, "w5": 4}   # sampled whole windows; the others: all


@pytest.fixture(scope="module")
def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.mark.parametrize("name", ["w1", "w2", "w3", "w4", "w5"])
def test_full_size(name, device):
    import paper_2201_01684_amd as pkg
    wl = make_workload(name)
    print(f"\n[{name}] {wl.num_windows} windows x {wl.num_channels} ch x {wl.n}, "
          f"T {wl.tmin}..{wl.tmax}, sha256 {wl.sha256[:16]}", flush=True)
    x = torch.from_numpy(wl.x).to(device)
    desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                               wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights)
    det = pkg.Detector(x, desc, keep)
    det.run()
    torch.cuda.synchronize()
    res = det.results_numpy()
    scores = det.scores.cpu().numpy()
    del x, det
    torch.cuda.empty_cache()

    # properties on every window
    assert np.all(np.isfinite(scores)) and np.all(scores >= 0)
    assert np.all(res["flags"] & pkg.UNRESOLVED == 0), "windows flagged UNRESOLVED"
    d = wl.truth > 0
    if wl.jitter:
        assert np.all(np.abs(res["period"][d] - wl.truth[d]) <= np.ceil(0.02 * wl.truth[d]))
    else:
        assert np.array_equal(res["period"][d], wl.truth[d])

    rng = np.random.default_rng(1234)
    if name not in WHOLE_WINDOWS:   # every window against the oracle
        o_scores, o_out = oracle.detect(wl.x, oracle.Layout.of(wl))
        check_scores(scores.astype(np.float64), o_scores, f"{name} (all windows)")
        check_results(res, o_out, f"{name} (all windows)")
        del o_scores
    else:                           # whole sampled windows against the oracle
        k = WHOLE_WINDOWS[name]
        picks = sorted({0, wl.num_windows - 1,
                        *rng.integers(0, wl.num_windows, size=k).tolist()})
        lay1 = oracle.Layout.of(wl, num_windows=1)
        span = (wl.num_channels - 1) * wl.channel_stride + wl.n
        for b in picks:
            sub = wl.x[b * wl.window_stride: b * wl.window_stride + span]
            o_scores, o_out = oracle.detect(sub, lay1)
            check_scores(scores[b:b + 1].astype(np.float64), o_scores, f"{name} window {b}")
            check_results(res[b:b + 1], o_out, f"{name} window {b}")

    # random single scores against the oracle
    lay = oracle.Layout.of(wl)
    ws = rng.integers(0, wl.num_windows, size=64)
    ts = rng.integers(wl.tmin, wl.tmax + 1, size=64)
    o = oracle.score_list(wl.x, lay, ws, ts)
    g = scores[ws, ts - wl.tmin].astype(np.float64)
    assert np.all((o != 0) | (g == 0))
    nz = o != 0
    assert np.all(np.abs(g[nz] - o[nz]) <= 1e-4 * o[nz])
