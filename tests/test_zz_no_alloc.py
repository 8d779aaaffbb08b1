"""gpoeo_pd_detect_noalloc against gpoeo_pd_detect, through the C ABI.

The no-allocation entry point runs the same kernels with its workspace in the
library's static device array, so its scores and results must equal those of
gpoeo_pd_detect with a caller workspace bit for bit (both are deterministic),
and hence meet the oracle parity bar that gpoeo_pd_detect meets.  Two calls in
a row, the second on a smaller input, check that nothing left in the shared
array by the first call leaks into the second.
"""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from gen import make_workload  # noqa: E402


def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def _run_both(wl, flags=0):
    import paper_2201_01684_amd as pkg
    from paper_2201_01684_amd import _binding as B
    dev = _device()
    lib = pkg.load_library()
    x = torch.from_numpy(np.ascontiguousarray(wl.x).reshape(-1)).to(dev)
    desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                               wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights,
                               flags=flags)
    need = pkg.workspace_bytes(desc)
    assert need <= B.NOALLOC_MAX_WORKSPACE
    lags = wl.tmax - wl.tmin + 1
    stream = torch.cuda.current_stream().cuda_stream
    out = []
    for noalloc in (False, True):
        scores = torch.full((wl.num_windows, lags), -1.0, dtype=torch.float32, device=dev)
        results = torch.full((wl.num_windows, B.RESULT_WORDS), -7, dtype=torch.int32, device=dev)
        if noalloc:
            rc = lib.gpoeo_pd_detect_noalloc(ctypes.byref(desc), x.data_ptr(), scores.data_ptr(),
                                             results.data_ptr(), stream)
        else:
            ws = torch.empty(need, dtype=torch.uint8, device=dev)
            rc = lib.gpoeo_pd_detect(ctypes.byref(desc), x.data_ptr(), scores.data_ptr(),
                                     results.data_ptr(), ws.data_ptr(), need, stream)
        assert rc == B.OK, B.strerror(rc)
        torch.cuda.synchronize()
        out.append((scores.cpu().numpy(), B.results_to_numpy(results)))
    del keep
    return out


def _check_equal_and_oracle(wl, pair, where):
    (s_ref, r_ref), (s_na, r_na) = pair
    assert np.array_equal(s_ref.view(np.uint32), s_na.view(np.uint32)), f"{where}: scores differ"
    assert r_ref.tobytes() == r_na.tobytes(), f"{where}: results differ"
    o, out = oracle.detect(wl.x, oracle.Layout.of(wl))
    zero = o == 0
    assert np.all(s_na[zero] == 0)
    rel = np.abs(s_na.astype(np.float64) - o)[~zero] / o[~zero]
    assert rel.max() <= 1e-4, f"{where}: score rel err {rel.max():.3e}"
    for f in ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates"):
        assert np.array_equal(r_na[f], out[f]), f"{where}: {f}"


def test_noalloc_matches_detect_twice_second_smaller():
    big = make_workload("w2", traces=4, n=32768, tmax=4096, pmax=3000)
    small = make_workload("w1")
    _check_equal_and_oracle(big, _run_both(big), "first call (4 x 32768)")
    _check_equal_and_oracle(small, _run_both(small), "second call (1 x 4096)")


def test_noalloc_rejects_oversized_work_before_launching():
    import paper_2201_01684_amd as pkg
    from paper_2201_01684_amd import _binding as B
    _device()
    lib = pkg.load_library()
    desc, _ = pkg.make_desc(1024, 1, 262144, 262144, 262144, 2, 32768)
    assert pkg.workspace_bytes(desc) > B.NOALLOC_MAX_WORKSPACE
    x = torch.zeros(16, dtype=torch.float32, device="cuda:0")
    res = torch.zeros(16, dtype=torch.int32, device="cuda:0")
    rc = lib.gpoeo_pd_detect_noalloc(ctypes.byref(desc), x.data_ptr(), None, res.data_ptr(),
                                     torch.cuda.current_stream().cuda_stream)
    assert rc == B.ETOOBIG
