"""Host-side checks of the C ABI (no GPU): the library loads, exports every
declared entry point, its structs match the header, and every invalid-argument
path returns before any launch."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gpoeo_pd.h")

pkg = pytest.importorskip("paper_2201_01684_amd")
from paper_2201_01684_amd import _binding as B  # noqa: E402


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libgpoeo_pd.so is not built (run __graft_entry__.build())")
    return B.load_library()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(gpoeo_pd_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(B.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (gpoeo_pd_\w+)$", out, re.M))
    assert exported == set(names)


def test_version_and_messages(lib):
    assert lib.gpoeo_pd_abi_version() == 1
    for code in (0, -1, -2, -3, 17):
        assert isinstance(B.strerror(code), str) and B.strerror(code)
    assert B.strerror(-2) == "workspace too small"


def test_struct_layout_matches_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text("""
#include <stdio.h>
#include <stddef.h>
#include "gpoeo_pd.h"
int main(void) {
  printf("%zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu\\n", sizeof(gpoeo_pd_desc),
         offsetof(gpoeo_pd_desc, c_lag), offsetof(gpoeo_pd_desc, channel_weights),
         offsetof(gpoeo_pd_desc, flags), sizeof(gpoeo_pd_result),
         offsetof(gpoeo_pd_result, n_rescored), sizeof(gpoeo_pd_rolling_result),
         offsetof(gpoeo_pd_rolling_result, smpdur_next), offsetof(gpoeo_pd_rolling_result, starts),
         sizeof(gpoeo_pd_plan_info), sizeof(gpoeo_pd_spectral_params),
         sizeof(gpoeo_pd_spectral_result), offsetof(gpoeo_pd_spectral_result, max_peak),
         offsetof(gpoeo_pd_spectral_result, amplitudes));
  return 0;
}
""")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    got = list(map(int, subprocess.run([str(exe)], capture_output=True, text=True,
                                       check=True).stdout.split()))
    want = [ctypes.sizeof(B.Desc), B.Desc.c_lag.offset, B.Desc.channel_weights.offset,
            B.Desc.flags.offset, ctypes.sizeof(B.Result), B.Result.n_rescored.offset,
            ctypes.sizeof(B.RollingResult), B.RollingResult.smpdur_next.offset,
            B.RollingResult.starts.offset, ctypes.sizeof(B.PlanInfo),
            ctypes.sizeof(B.SpectralParams), B.SPECTRAL_DTYPE.itemsize,
            B.SPECTRAL_DTYPE.fields["max_peak"][1], B.SPECTRAL_DTYPE.fields["amplitudes"][1]]
    assert got == want


def good_desc(**kw):
    base = dict(num_windows=4, num_channels=2, n=4096, window_stride=8192, channel_stride=4096,
                tmin=2, tmax=1024)
    base.update(kw)
    return B.make_desc(**base)


def test_workspace_size_valid_and_monotone(lib):
    d, _ = good_desc()
    small = B.workspace_bytes(d)
    d2, _ = good_desc(num_windows=8, window_stride=8192)
    assert small > 0 and B.workspace_bytes(d2) > small
    assert small % 256 == 0


@pytest.mark.parametrize("kw", [
    dict(num_windows=0), dict(num_windows=(1 << 21) + 1, window_stride=8192), dict(num_channels=0), dict(num_channels=257, channel_stride=4096),
    dict(n=7, tmin=1, tmax=3), dict(tmin=0), dict(tmin=5, tmax=6), dict(tmax=2049),
    dict(window_stride=0), dict(channel_stride=4095), dict(window_stride=-1),
    dict(c_lag=0.0), dict(c_lag=1.0), dict(c_lag=float("nan")), dict(err_max=float("nan")),
    dict(flags=32), dict(flags=4, n=4 << 20, tmax=2 << 20),
    # grids that would exceed HIP's 32-bit global size: 2^24 sequences of 256
    # threads, 2^26 lag-score waves of 64
    dict(num_windows=1 << 20, num_channels=16, n=64, tmax=32, window_stride=1024,
         channel_stride=64),
    dict(num_windows=1 << 21, num_channels=1, n=65536, tmax=32768, window_stride=65536,
         channel_stride=65536),
])
def test_invalid_descriptors_rejected(lib, kw):
    d, _ = good_desc(**kw)
    with pytest.raises(B.GpoeoError) as e:
        B.workspace_bytes(d)
    assert e.value.status == B.EINVAL


@pytest.mark.parametrize("weights", [[1.0, 0.0], [1.0, -2.0], [1.0, float("inf")],
                                     [float("nan"), 1.0]])
def test_invalid_weights_rejected(lib, weights):
    d, _keep = good_desc(weights=np.array(weights, dtype=np.float32))
    with pytest.raises(B.GpoeoError):
        B.workspace_bytes(d)


def test_size_limits(lib):
    # just inside the sequence limit: accepted
    d, _ = good_desc(num_windows=1 << 19, num_channels=16, n=64, tmax=32, window_stride=1024,
                     channel_stride=64)
    assert B.workspace_bytes(d) > 0
    assert B.MAX_WINDOWS == 1 << 21 and B.MAX_QUERIES == 1 << 23
    # too many queries: rejected before any pointer is used
    d, _ = good_desc()
    for name in ("gpoeo_pd_score_centred",):
        call = getattr(lib, name)
        assert call(ctypes.byref(d), 0x100000, 0x200000, 0x300000, B.MAX_QUERIES + 1, 0x400000,
                    None) == B.EINVAL
        assert call(ctypes.byref(d), 0x100000, 0x200000, 0x300000, -1, 0x400000,
                    None) == B.EINVAL
    sp = B.SimilarityParams(3, 20)
    assert lib.gpoeo_pd_similarity(ctypes.byref(d), ctypes.byref(sp), 0x100000, 0x200000,
                                   0x300000, B.MAX_QUERIES + 1, 0x400000, None) == B.EINVAL


def test_channel_limit_is_the_header_limit(lib):
    """The header states 1 <= C <= GPOEO_PD_MAX_CHANNELS; the library enforces
    exactly that bound, and the binding carries the same constant."""
    text = open(HEADER).read()
    m = re.search(r"#define GPOEO_PD_MAX_CHANNELS (\d+)", text)
    assert m, "the header must define GPOEO_PD_MAX_CHANNELS"
    limit = int(m.group(1))
    assert limit == B.MAX_CHANNELS == 256
    assert re.search(r"num_channels;\s*/\*\s*1 <= C <= GPOEO_PD_MAX_CHANNELS", text)
    ok, _ = good_desc(num_channels=limit, channel_stride=4096, window_stride=4096 * limit)
    assert B.workspace_bytes(ok) > 0
    bad, _ = good_desc(num_channels=limit + 1, channel_stride=4096,
                       window_stride=4096 * (limit + 1))
    with pytest.raises(B.GpoeoError) as e:
        B.workspace_bytes(bad)
    assert e.value.status == B.EINVAL


def test_reserved_fields_must_be_zero(lib):
    d, _ = good_desc()
    d.reserved0 = 1
    size = ctypes.c_size_t()
    assert lib.gpoeo_pd_workspace_bytes(ctypes.byref(d), ctypes.byref(size)) == B.EINVAL
    assert lib.gpoeo_pd_workspace_bytes(None, ctypes.byref(size)) == B.EINVAL
    d, _ = good_desc()
    assert lib.gpoeo_pd_workspace_bytes(ctypes.byref(d), None) == B.EINVAL


def test_detect_rejects_bad_pointers_before_launching(lib):
    # Fake device addresses: every call below must fail validation on the host.
    d, _ = good_desc()
    need = B.workspace_bytes(d)
    x, res, ws = 0x100000, 0x200000, 0x300000
    call = lib.gpoeo_pd_detect
    assert call(None, x, None, res, ws, need, None) == B.EINVAL
    assert call(ctypes.byref(d), None, None, res, ws, need, None) == B.EINVAL
    assert call(ctypes.byref(d), x, None, None, ws, need, None) == B.EINVAL
    assert call(ctypes.byref(d), x, None, res, None, need, None) == B.EINVAL
    assert call(ctypes.byref(d), x, None, res, ws + 8, need, None) == B.EINVAL  # misaligned ws
    assert call(ctypes.byref(d), x + 2, None, res, ws, need, None) == B.EINVAL  # misaligned x
    assert call(ctypes.byref(d), x, None, res, ws, need - 1, None) == B.ENOMEM
    bad, _ = good_desc(tmax=4000)
    assert call(ctypes.byref(bad), x, None, res, ws, need, None) == B.EINVAL


def test_scores_only_needs_no_results_pointer_but_still_a_workspace(lib):
    d, _ = good_desc(flags=B.SCORES_ONLY)
    need = B.workspace_bytes(d)
    assert lib.gpoeo_pd_detect(ctypes.byref(d), 0x100000, None, None, None, need,
                               None) == B.EINVAL
    assert lib.gpoeo_pd_detect(ctypes.byref(d), 0x100000, None, None, 0x300000, need - 1,
                               None) == B.ENOMEM


def test_plan_description(lib):
    from gen import make_workload
    wl = make_workload("w4", total=65536, n=16384, stride=2048, tmax=4096)
    d, _ = B.make_desc(wl.num_windows, 1, wl.n, wl.window_stride, wl.channel_stride, wl.tmin,
                       wl.tmax)
    info = B.describe_plan(d)
    assert info["mode"] == 1 and info["pairs_defined"] == wl.pairs()
    assert 0 < info["pairs_scored"] < info["pairs_defined"]
    assert info["workspace_bytes"] == B.workspace_bytes(d)
    # non-overlapping windows: every window scored on its own
    d, _ = good_desc()
    info = B.describe_plan(d)
    assert info["mode"] == 0 and info["pairs_scored"] == info["pairs_defined"]
    assert info["pairs_defined"] == 4 * 2 * sum(4096 - t for t in range(2, 1025))
    assert info["lags_per_lane"] in (8, 16)


@pytest.mark.parametrize("kw", [dict(c_measure=0.0), dict(step=0.0), dict(c_eval=-1.0),
                                dict(diff_threshold=float("nan")), dict(c_eval=100.0),
                                dict(step=float("inf"))])
def test_rolling_parameters_validated(lib, kw):
    d, _ = good_desc()
    with pytest.raises(B.GpoeoError) as e:
        B.rolling_workspace_bytes(d, B.rolling_params(**kw))
    assert e.value.status == B.EINVAL


def test_rolling_workspace_and_flags(lib):
    d, _ = good_desc()
    assert B.rolling_workspace_bytes(d, B.rolling_params()) > B.workspace_bytes(d)
    d, _ = good_desc(flags=B.SCORES_ONLY)
    with pytest.raises(B.GpoeoError):
        B.rolling_workspace_bytes(d, B.rolling_params())
    d, _ = good_desc()
    p = B.rolling_params()
    need = B.rolling_workspace_bytes(d, p)
    call = lib.gpoeo_pd_detect_rolling
    assert call(ctypes.byref(d), ctypes.byref(p), 0x100000, 0x200000, 0x300000, need - 1,
                None) == B.ENOMEM
    assert call(ctypes.byref(d), None, 0x100000, 0x200000, 0x300000, need, None) == B.EINVAL
    assert call(ctypes.byref(d), ctypes.byref(p), 0x100000, None, 0x300000, need,
                None) == B.EINVAL


def test_fft_plan(lib):
    d, _ = good_desc()
    direct = B.workspace_bytes(d)
    d, _ = good_desc(flags=B.FFT_SCORES)
    info = B.describe_plan(d)
    assert info["mode"] == 2 and info["score_waves"] == 0 and info["pairs_scored"] == 0
    assert info["pairs_defined"] == 4 * 2 * sum(4096 - t for t in range(2, 1025))
    # 8 complex fp64 transforms of 8192 points (4096 + 1024 <= 2^13) at least
    assert info["workspace_bytes"] >= 4 * 8192 * 16
    assert info["workspace_bytes"] != direct
    assert info["fft_len"] == 8192 and info["fft_wrap_len"] == 0 and info["fft_wrap_lags"] == 0
    # the largest transform, 2^22 points: N + Tmax <= 2^22 without the wrap term ...
    d, _ = good_desc(flags=B.FFT_SCORES, num_windows=1, n=(1 << 22) - 1000, tmax=1000,
                     channel_stride=1 << 22)
    info = B.describe_plan(d)
    assert info["mode"] == 2 and info["fft_len"] == 1 << 22 and info["fft_wrap_len"] == 0
    # ... or with it: 1 wrapped lag, a head-tail transform of 2^12 points
    d, _ = good_desc(flags=B.FFT_SCORES, num_windows=1, n=(1 << 22) - 1000, tmax=1001,
                     channel_stride=1 << 22)
    info = B.describe_plan(d)
    assert (info["fft_len"], info["fft_wrap_len"], info["fft_wrap_lags"]) == (1 << 22, 4096, 1)
    # a wrap term longer than 2^19 lags (a head-tail transform beyond 2^20): rejected
    d, _ = good_desc(flags=B.FFT_SCORES, num_windows=1, n=(1 << 22) - 1000,
                     tmax=(1 << 19) + 1000 + 1, channel_stride=1 << 22)
    with pytest.raises(B.GpoeoError):
        B.workspace_bytes(d)
    # the rule on the five workloads' shapes: N a power of two with Tmax up to
    # N / 4 takes the wrap term; 4096 + 1024 keeps the padded transform
    for n, tmax, want in [(4096, 1024, (8192, 0, 0)), (65536, 8192, (65536, 16384, 8192)),
                          (262144, 32768, (262144, 65536, 32768)),
                          (16384, 4096, (16384, 8192, 4096)),
                          (131072, 16384, (131072, 32768, 16384))]:
        d, _ = good_desc(flags=B.FFT_SCORES, num_windows=2, n=n, tmax=tmax, window_stride=n,
                         channel_stride=n, num_channels=1)
        info = B.describe_plan(d)
        assert (info["fft_len"], info["fft_wrap_len"], info["fft_wrap_lags"]) == want, (n, tmax)
    # rolling accepts the FFT flag
    d, _ = good_desc(flags=B.FFT_SCORES)
    assert B.rolling_workspace_bytes(d, B.rolling_params()) > 0


def test_mfma_plan(lib):
    d, _ = good_desc(flags=B.MFMA_SCORES)
    info = B.describe_plan(d)
    # lags 2..1024 in one tile of 1024 lags from Tmin per sequence; 8 waves are
    # too few, so each tile's 130 sample steps split into two chunks (no chunk
    # shorter than 64 steps)
    assert info["mode"] == 3 and info["score_waves"] == 4 * 2 * 1 * 2
    assert info["pairs_defined"] == 4 * 2 * sum(4096 - t for t in range(2, 1025))
    # four int8 digit planes per sequence (padded), edge sums, per-sequence statistics
    assert info["workspace_bytes"] >= 4 * 2 * 4 * 4096 + 4 * 2 * 2 * 1025 * 8
    assert info["fft_len"] == 0
    # tiles start at Tmin itself (98 steps from there: one chunk)
    d, _ = good_desc(flags=B.MFMA_SCORES, tmin=1021, tmax=2045)
    assert B.describe_plan(d)["score_waves"] == 4 * 2 * 2          # 1021 .. 3068
    d, _ = good_desc(flags=B.MFMA_SCORES, tmin=1024, tmax=2047)
    assert B.describe_plan(d)["score_waves"] == 4 * 2 * 1
    # a small batch of long windows: 64 sequences x 1 tile, 8194 steps each,
    # split into 64 chunks of 130 steps (4096 waves)
    d, _ = good_desc(flags=B.MFMA_SCORES, num_windows=64, num_channels=1, n=262144,
                     tmax=1024, window_stride=262144, channel_stride=262144)
    assert B.describe_plan(d)["score_waves"] == 64 * 1 * 64
    # a large batch keeps one chunk per tile: 1024 sequences x 32 tiles
    d, _ = good_desc(flags=B.MFMA_SCORES, num_windows=1024, num_channels=1, n=262144,
                     tmax=32767, window_stride=262144, channel_stride=262144)
    assert B.describe_plan(d)["score_waves"] == 1024 * 32
    # a tile grid beyond HIP's 32-bit global size: 2^21 windows x 8 groups of 4
    # lag tiles x 256 threads
    d, _ = good_desc(flags=B.MFMA_SCORES, num_windows=1 << 21, num_channels=1, n=65536,
                     tmax=32768, window_stride=65536, channel_stride=65536)
    with pytest.raises(B.GpoeoError) as e:
        B.workspace_bytes(d)
    assert e.value.status == B.EINVAL
    # one score source per call; rolling detection takes the flag too
    d, _ = good_desc(flags=B.MFMA_SCORES | B.FFT_SCORES)
    with pytest.raises(B.GpoeoError) as e:
        B.workspace_bytes(d)
    assert e.value.status == B.EINVAL
    d, _ = good_desc(flags=B.MFMA_SCORES)
    assert B.rolling_workspace_bytes(d, B.rolling_params()) > B.workspace_bytes(d)


@pytest.mark.parametrize("kw", [dict(c_peak=0.0), dict(c_peak=1.0), dict(max_candidates=0),
                                dict(max_candidates=17)])
def test_spectral_parameters_validated(lib, kw):
    d, _ = good_desc()
    with pytest.raises(B.GpoeoError) as e:
        B.spectral_workspace_bytes(d, B.spectral_params(**kw))
    assert e.value.status == B.EINVAL


def test_spectral_workspace_and_pointers(lib):
    d, _ = good_desc()
    p = B.spectral_params()
    need = B.spectral_workspace_bytes(d, p)
    # 8 sequences of 4096 points: amplitudes of 2049 bins each at least
    assert need >= 8 * 2049 * 8
    call = lib.gpoeo_pd_spectral_candidates
    assert call(ctypes.byref(d), ctypes.byref(p), 0x100000, 0x200000, 0x300000, need - 1,
                None) == B.ENOMEM
    assert call(ctypes.byref(d), None, 0x100000, 0x200000, 0x300000, need, None) == B.EINVAL
    assert call(ctypes.byref(d), ctypes.byref(p), 0x100000, None, 0x300000, need,
                None) == B.EINVAL


def test_noalloc_validates_on_the_host_before_touching_the_device(lib):
    """gpoeo_pd_detect_noalloc: an invalid descriptor or pointer is EINVAL and a
    workload whose workspace exceeds the static scratch is ETOOBIG, both decided
    on the host (fake device addresses are never dereferenced)."""
    call = lib.gpoeo_pd_detect_noalloc
    x, res = 0x100000, 0x200000
    d, _ = good_desc()
    assert call(None, x, None, res, None) == B.EINVAL
    assert call(ctypes.byref(d), None, None, res, None) == B.EINVAL
    assert call(ctypes.byref(d), x, None, None, None) == B.EINVAL
    bad, _ = good_desc(tmax=4000)
    assert call(ctypes.byref(bad), x, None, res, None) == B.EINVAL
    big, _ = B.make_desc(1024, 1, 262144, 262144, 262144, 2, 32768)
    assert B.workspace_bytes(big) > B.NOALLOC_MAX_WORKSPACE
    assert call(ctypes.byref(big), x, None, res, None) == B.ETOOBIG
    text = open(HEADER).read()
    assert "#define GPOEO_PD_NOALLOC_MAX_WORKSPACE ((size_t)64 << 20)" in text
    assert B.NOALLOC_MAX_WORKSPACE == 64 << 20
    assert B.strerror(B.ETOOBIG) == "workspace larger than the static no-allocation scratch"
