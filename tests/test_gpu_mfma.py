"""GPU parity of the matrix-core scores (GPOEO_PD_MFMA_SCORES) against the fp64 oracle.

The path promises every score within 1.25e-5 relative of the exact value
(half the direct path's tier-0 width; lags its bound cannot certify are
re-scored in fp64 first), exact zeros where the oracle has them, and
selections identical to the oracle's.  On sequences whose samples the
integer scaling represents exactly (every workload here but the normalised
counters of w5) the only errors left are the fp64 combination and the three
digit pairs of least weight left out of the products (at most 2^24 per sample
pair in D against samples scaled to 2^30, and of random sign), so their scores
are held to the fp32 output rounding.  Covered: the smallest windows, ragged
N, lag ranges that start inside a tile and end on, before and after a tile
boundary, weighted channels at different scales, samples spanning many
binades (inexact, bounded), exactly periodic and constant windows, scores
only, determinism, 256 channels, windows and channels at odd sample offsets,
one window of 2^22 samples (sampled lags), small batches whose tiles split
their samples into chunks (a ragged last chunk, chunks left empty for the
later tiles), and the five workloads at full size (sampled windows against
the oracle, every window against the direct path).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from gen import make_workload, planted_trace  # noqa: E402

from test_gpu_parity import check_results, gpu_run  # noqa: E402

MFMA_RTOL = 1.25e-5 + 2.0 ** -24     # the fix-up's bound plus the fp32 output rounding
EXACT_RTOL = 1e-7                    # exactly represented samples: fp64 combination, left-out pairs, fp32 output


def mfma_flag():
    import paper_2201_01684_amd as pkg
    return pkg.MFMA_SCORES


def check_mfma_scores(g, o, where="", rtol=MFMA_RTOL):
    assert g.shape == o.shape
    zero = o == 0
    assert np.all(g[zero] == 0), f"{where}: zero scores not reproduced"
    rel = np.abs(g - o)[~zero] / np.abs(o[~zero])
    assert rel.size == 0 or rel.max() <= rtol, f"{where}: rel {rel.max():.3e}"
    return float(rel.max()) if rel.size else 0.0


def mfma_parity(x, lay, where="", flags=0, rtol=MFMA_RTOL):
    g, res = gpu_run(x, lay, flags=mfma_flag() | flags)
    o, out = oracle.detect(x, lay)
    check_mfma_scores(g, o, where, rtol)
    if res is not None:
        check_results(res, out, where)
    return g, res, out


@pytest.mark.parametrize("n,tmin,tmax", [
    (8, 1, 4),            # the smallest window: one tile, two steps
    (100, 2, 50),
    (1500, 2, 500),
    (4099, 3, 2049),      # ragged N, three tiles
    (3000, 1021, 1500),   # tiles from Tmin: B staged 13 bytes past a 16-byte boundary
    (5000, 2, 1024),      # Tmax below the last lag of the first tile
    (5000, 2, 1025),      # Tmax on the last lag of the first tile
    (5000, 2, 1026),      # Tmax the first lag of a second tile
    (5000, 9, 2047),      # B offset 9: the third dword of the aligned pair
    (5000, 17, 2047),
    (20000, 6, 3333),
    (20000, 4106, 9000),  # offset 10, workgroups of four tiles from lag 4106
])
def test_edge_shapes(n, tmin, tmax):
    x = planted_trace(n, max(3, min(97, n // 3)), 3, seed=n + tmin, sigma=1.0)
    mfma_parity(x, oracle.Layout(1, 1, n, n, n, tmin, tmax), f"n={n} T=[{tmin},{tmax}]",
                rtol=EXACT_RTOL)


@pytest.mark.parametrize("name,kw,rtol", [
    ("w1", {}, EXACT_RTOL),
    ("w2", dict(traces=5, n=16384, tmax=2048, pmax=1500), EXACT_RTOL),
    ("w3", dict(traces=4, n=32768, tmax=4096, pmax=3000), EXACT_RTOL),
    ("w4", dict(total=131072, n=16384, stride=2048, tmax=4096), EXACT_RTOL),
    ("w5", dict(traces=3, n=16384, tmax=2048, pmax=1500), MFMA_RTOL),   # normalised counters
])
def test_reduced_workloads(name, kw, rtol):
    wl = make_workload(name, **kw)
    mfma_parity(wl.x, oracle.Layout.of(wl), f"mfma {name}{kw}", rtol=rtol)


def test_weighted_channels_at_different_scales():
    rng = np.random.default_rng(3)
    b, c, n = 3, 3, 6000
    base = np.stack([planted_trace(n, 300 + 17 * k, 6, seed=k, sigma=0.5) for k in range(b)])
    x = np.stack([base * s + rng.normal(0, 0.3, size=(b, n)) for s in (1.0, 0.01, 30.0)], axis=1)
    lay = oracle.Layout(b, c, n, c * n, n, 2, 3000,
                        weights=np.array([1.0, 250.0, 0.003], dtype=np.float32))
    mfma_parity(x.astype(np.float32), lay, "mfma weighted")


def test_samples_over_many_binades():
    # magnitudes from 1e-6 to 1e3 in one sequence: no power-of-two scaling
    # represents them in 31 bits, so the quantisation bound decides which lags
    # are re-scored
    n = 8192
    rng = np.random.default_rng(11)
    p = planted_trace(n, 211, 5, seed=12, sigma=0.5).astype(np.float64)
    tiny = rng.normal(0, 1e-6, n)
    x = np.stack([(p + tiny).astype(np.float32),
                  (p * 10.0 ** rng.uniform(-6, 0, n)).astype(np.float32),
                  (1e3 + rng.normal(0, 1e-3, n)).astype(np.float32)])
    g, res, out = mfma_parity(x, oracle.Layout(3, 1, n, n, n, 2, 4096), "mfma binades")
    assert res["period"][0] == 211


def test_left_out_pairs_decide_the_fix_up():
    # Levels below 2^20 in steps of 1/8 (exact in fp32) under noise of 390: the
    # scale is 2^10, so the lowest digit is not zero, and at multiples of the
    # period S is about 3e5 against 7e11 elsewhere.  The bound of the three
    # digit pairs left out of the products, 2 * 8404992 per pair in X units or
    # about 16 per pair in samples, exceeds 1.25e-5 of the score there (the
    # fp64 rounding terms alone would not, below about 4e4), so the fix-up
    # re-scores those lags in fp64; every other lag keeps its certified value.
    n, period = 8192, 97
    rng = np.random.default_rng(31)
    template = rng.integers(-2**20 + 8192, 2**20 - 8192, size=period) + rng.integers(0, 8, period) / 8
    noise = np.round(rng.normal(0.0, 390.0, n) * 8) / 8
    x64 = np.tile(template, n // period + 1)[:n] + noise
    x64[0] -= np.sum(x64) % (n / 8)   # a mean on the 1/8 grid: every x - c exact at scale 2^10
    x = x64.astype(np.float32)
    assert np.array_equal(x.astype(np.float64), x64)
    lay = oracle.Layout(1, 1, n, n, n, 2, 2048)
    g, res, out = mfma_parity(x[None], lay, "mfma left-out pairs", rtol=EXACT_RTOL)
    assert res["period"][0] == period
    at_period = np.arange(period, 2049, period)
    s_at = g[0, at_period - 2]
    assert np.all((s_at > 1e5) & (s_at < 1e6))
    assert res["n_rescored"][0] >= len(at_period)


def test_exact_periods_and_constant_windows():
    n = 8192
    rows = [np.full(n, 123.25, dtype=np.float32),                         # CONSTANT
            planted_trace(n, 64, 4, seed=1, integer=True),                  # zeros at 64 k
            planted_trace(n, 301, 9, seed=2, sigma=0.0),                    # real-valued repeats
            np.random.default_rng(4).normal(0, 1, n).astype(np.float32),
            np.zeros(n, dtype=np.float32)]
    x = np.stack(rows)
    lay = oracle.Layout(len(rows), 1, n, n, n, 2, 4096)
    g, res, out = mfma_parity(x, lay, "mfma special windows")
    assert res["period"][1] == 64 and res["period"][2] == 301
    assert res["verdict"][0] == 2 and res["verdict"][4] == 2
    assert np.all(g[1, np.arange(64, 4097, 64) - 2] == 0)
    assert np.all(g[0] == 0) and np.all(g[4] == 0)


def test_scores_only_and_no_rescue():
    import paper_2201_01684_amd as pkg
    wl = make_workload("w2", traces=4, n=16384, tmax=2048, pmax=1500)
    lay = oracle.Layout.of(wl)
    g, _ = gpu_run(wl.x, lay, flags=mfma_flag() | pkg.SCORES_ONLY)
    o, out = oracle.detect(wl.x, lay)
    check_mfma_scores(g, o, "mfma scores only", EXACT_RTOL)
    _, res = gpu_run(wl.x, lay, flags=mfma_flag() | pkg.NO_RESCUE)
    assert np.all(np.abs(res["period"] - out["period"]) <= 2)


def test_deterministic_bitwise():
    wl = make_workload("w5", traces=2, n=16384, tmax=2048, pmax=1500)
    lay = oracle.Layout.of(wl)
    a, ra = gpu_run(wl.x, lay, flags=mfma_flag())
    b, rb = gpu_run(wl.x, lay, flags=mfma_flag())
    assert np.array_equal(a, b) and np.array_equal(ra, rb)


@pytest.mark.parametrize("name", ["w1", "w2", "w3", "w4", "w5"])
def test_full_size(name):
    import paper_2201_01684_amd as pkg
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    wl = make_workload(name)
    print(f"\n[mfma {name}] {wl.num_windows} windows x {wl.num_channels} ch x {wl.n}", flush=True)
    x = torch.from_numpy(wl.x).to("cuda:0")
    out = {}
    for mode, flags in (("mfma", mfma_flag()), ("direct", 0)):
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
    gm, rm = out["mfma"]
    gd, rd = out["direct"]
    assert np.all(rm["flags"] & pkg.UNRESOLVED == 0)
    for f in ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates"):
        assert np.array_equal(rm[f], rd[f]), f"{name}: {f} differs from the direct path"
    # both within their bounds of the exact scores: 2.5e-5 + 1.25e-5 (+ fp32 rounding)
    nz = gd != 0
    assert np.all(gm[~nz] == 0)
    assert np.all(np.abs(gm[nz].astype(np.float64) - gd[nz]) <= 3.8e-5 * np.abs(gd[nz]))
    rng = np.random.default_rng(99)
    lay1 = oracle.Layout.of(wl, num_windows=1)
    span = (wl.num_channels - 1) * wl.channel_stride + wl.n
    rtol = MFMA_RTOL if name == "w5" else EXACT_RTOL
    for b in sorted({0, wl.num_windows - 1, int(rng.integers(0, wl.num_windows))}):
        sub = wl.x[b * wl.window_stride: b * wl.window_stride + span]
        o_scores, o_out = oracle.detect(sub, lay1)
        check_mfma_scores(gm[b:b + 1].astype(np.float64), o_scores, f"mfma {name} window {b}",
                          rtol)
        check_results(rm[b:b + 1], o_out, f"mfma {name} window {b}")


def test_maximum_channel_count():
    # 256 channels, each with its own weight and scale (several of them inexact)
    rng = np.random.default_rng(11)
    b, c, n = 2, 256, 1500
    x = np.empty((b, c, n), dtype=np.float32)
    for k in range(c):
        x[0, k] = planted_trace(n, 97, 5, seed=100 + k, sigma=0.5) * (0.01 + k % 7)
        x[1, k] = rng.normal(0, 1 + k % 3, n)
    w = (0.1 + rng.random(c)).astype(np.float32)
    lay = oracle.Layout(b, c, n, c * n, n, 2, 700, weights=w)
    g, res, out = mfma_parity(x, lay, "mfma 256 channels")
    assert res["period"][0] == 97


def test_unaligned_strides():
    # windows and channels at odd sample offsets: the samples are read one by
    # one, the digit planes stay aligned in the workspace
    rng = np.random.default_rng(21)
    n, c, b = 5001, 2, 3
    cs, ws = n + 3, 2 * (n + 3) + 7
    x = rng.normal(0, 0.2, size=(b - 1) * ws + (c - 1) * cs + n + 5).astype(np.float32)
    for k in range(b):
        for ch in range(c):
            o = k * ws + ch * cs
            x[o:o + n] += planted_trace(n, 123 + 40 * k, 6, seed=7 * k + ch, sigma=0.0)
    lay = oracle.Layout(b, c, n, ws, cs, 3, 2400)
    g, res, out = mfma_parity(x, lay, "mfma odd strides")
    assert list(res["period"]) == [123, 163, 203]


def test_long_window_sampled_lags():
    # one window of 2^22 samples, lags to 2^16: sampled lags against the oracle,
    # the selection against the direct scores
    n, tmax = 1 << 22, 1 << 16
    x = planted_trace(n, 3001, 9, seed=21, sigma=2.0)
    lay = oracle.Layout(1, 1, n, n, n, 2, tmax)
    g, res = gpu_run(x, lay, flags=mfma_flag())
    gd, rd = gpu_run(x, lay)
    for f in ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates"):
        assert np.array_equal(res[f], rd[f]), f
    assert res["period"][0] == 3001
    rng = np.random.default_rng(2)
    ts = np.concatenate([rng.integers(2, tmax + 1, size=40), [2, 1023, 1024, 3001, 6002, tmax]])
    o = oracle.score_list(x, lay, np.zeros(ts.size, dtype=np.int64), ts)
    check_mfma_scores(g[0, ts - 2].astype(np.float64), o, "mfma 2^22 samples", EXACT_RTOL)


@pytest.mark.parametrize("b,c,n,tmin,tmax,chunks", [
    (3, 1, 65536, 2, 2047, 32),     # 2050 steps in chunks of 66: the last holds 4; tile 1 leaves chunk 31 empty
    (1, 2, 30001, 5, 3100, 14),     # ragged N, four tiles, weighted channels
    (2, 1, 8192, 1500, 4000, 3),    # tiles from 1488, fewer steps than the window
])
def test_chunked_tiles(b, c, n, tmin, tmax, chunks):
    # Few waves: each tile's sample steps are split into chunks whose partial
    # cross terms are summed in a fixed order before D(T) is formed.
    import paper_2201_01684_amd as pkg
    x = np.stack([np.stack([planted_trace(n, 211 + 90 * k + 7 * ch, 6, seed=10 * k + ch,
                                          sigma=0.5) for ch in range(c)]) for k in range(b)])
    lay = oracle.Layout(b, c, n, c * n, n, tmin, tmax,
                        weights=np.linspace(1.0, 2.0, c).astype(np.float32))
    desc, _ = pkg.make_desc(b, c, n, c * n, n, tmin, tmax, weights=lay.weights,
                            flags=mfma_flag())
    tiles = (tmax - tmin) // 1024 + 1
    assert pkg.describe_plan(desc)["score_waves"] == b * c * tiles * chunks
    g, res, out = mfma_parity(x, lay, f"mfma chunked {b}x{c}x{n}")
    g2, res2 = gpu_run(x, lay, flags=mfma_flag())
    assert np.array_equal(g, g2) and np.array_equal(res, res2)
