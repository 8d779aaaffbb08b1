"""The detection enqueues only kernels (no allocation, memset, copy or host
synchronisation), so one call can be captured into a HIP graph and replayed.

Each case captures one call, then replays it several times with eager work
(input swaps, eager calls, synchronisations) between the replays, and checks
every replay bitwise against the eager result for the input it saw.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from gen import make_workload, planted_trace  # noqa: E402


def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def _snapshot(det):
    torch.cuda.synchronize()
    s = None if det.scores is None else det.scores.clone()
    return s, det.results.clone()


def _check(det, ref, where):
    s, r = _snapshot(det)
    assert torch.equal(r, ref[1]), f"{where}: results differ"
    if s is not None:
        assert torch.equal(s, ref[0]), f"{where}: scores differ"


@pytest.mark.parametrize("mode", ["direct", "fft", "mfma"])
@pytest.mark.parametrize("name,kw", [("w1", {}), ("w3", dict(traces=4, n=32768, tmax=4096,
                                                              pmax=3000))])
def test_detect_captured_and_replayed(name, kw, mode):
    import paper_2201_01684_amd as pkg
    dev = _device()
    wl = make_workload(name, **kw)
    xa = torch.from_numpy(wl.x.reshape(-1)).to(dev)
    xb = torch.flip(xa, dims=[0]).contiguous()          # a different input of the same layout
    x = xa.clone()
    desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                               wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights,
                               flags={"direct": 0, "fft": pkg.FFT_SCORES,
                                      "mfma": pkg.MFMA_SCORES}[mode])
    det = pkg.Detector(x, desc, keep)
    det.run()
    ref_a = _snapshot(det)
    x.copy_(xb)
    det.run()
    ref_b = _snapshot(det)
    x.copy_(xa)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        det.run()                                        # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        det.run()
    torch.cuda.synchronize()

    for k, (src, ref) in enumerate([(xa, ref_a), (xb, ref_b), (xa, ref_a), (xb, ref_b)]):
        x.copy_(src)
        if k == 2:
            det.run()                                    # eager call between replays
            torch.cuda.synchronize()
        det.results.zero_()
        if det.scores is not None:
            det.scores.zero_()
        g.replay()
        _check(det, ref, f"{name} {mode} replay {k}")


def test_rolling_captured_and_replayed():
    import paper_2201_01684_amd as pkg
    dev = _device()
    n = 12000
    rows = [planted_trace(n, 250, 7, seed=3, sigma=4.0), planted_trace(n, 137, 5, seed=4),
            np.concatenate([planted_trace(11500, 200, 6, seed=5, sigma=1.0),
                            planted_trace(500, 290, 6, seed=6, sigma=1.0)])]
    x = torch.from_numpy(np.stack(rows).astype(np.float32).reshape(-1)).to(dev)
    desc, keep = pkg.make_desc(3, 1, n, n, n, 2, n // 2, flags=pkg.FFT_SCORES)
    det = pkg.RollingDetector(x, desc, pkg.rolling_params(), keep)
    det.run()
    torch.cuda.synchronize()
    ref = det.results.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        det.run()
    for _ in range(3):
        det.results.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(det.results, ref)
        det.run()
        torch.cuda.synchronize()
