"""Pins of the oracle's FFT front end (Algorithm 1, lines 1-5): the amplitude
spectrum and the candidate periods drawn from its peaks.

Pinned against: the discrete Fourier transform written out as a direct sum on
small windows, pure tones on integer bins (known amplitude A L / 2 and
period), two-tone inputs on each side of the c_peak threshold, two bins
that round to one period (both listed), the lag range and the candidate limit, channel
weighting (amplitudes add), and a constant offset (removed by the centring).
"""
import math

import numpy as np
import pytest

import oracle


def tone(n, periods_amps, offset=100.0):
    i = np.arange(n, dtype=np.float64)
    x = np.full(n, offset)
    for p, a in periods_amps:
        x += a * np.sin(2 * np.pi * i / p + 0.3)
    return x.astype(np.float32)


@pytest.mark.parametrize("n", [10, 50, 64, 100])
def test_amplitude_spectrum_is_the_dft(n):
    rng = np.random.default_rng(n)
    x = rng.normal(3, 2, size=n).astype(np.float32)
    length = oracle.spectral_length(n)
    y = x.astype(np.float64) - x.astype(np.float64).mean()
    want = []
    for k in range(length // 2 + 1):
        re = sum(y[j] * math.cos(2 * math.pi * k * j / length) for j in range(n))
        im = -sum(y[j] * math.sin(2 * math.pi * k * j / length) for j in range(n))
        want.append(math.hypot(re, im))
    got = oracle.amplitude_spectrum(x)
    assert got.shape == (length // 2 + 1,)
    assert np.allclose(got, want, rtol=1e-10, atol=1e-10 * max(want))


@pytest.mark.parametrize("m", [5, 32, 100])
def test_pure_tone_on_an_integer_bin(m):
    length = 4096
    x = tone(length, [(length / m, 7.0)])
    c = oracle.spectral_candidates(x, 2, 2048)
    assert c["bins"] == [m]
    assert c["periods"] == [round(length / m + 1e-9)]
    assert c["amplitudes"][0] == pytest.approx(7.0 * length / 2, rel=1e-5)


@pytest.mark.parametrize("ratio,count", [(0.6, 1), (0.7, 2)])
def test_relative_height_threshold(ratio, count):
    length = 4096
    x = tone(length, [(length / 16, 10.0), (length / 48, 10.0 * ratio)])
    c = oracle.spectral_candidates(x, 2, 2048, c_peak=0.65)
    assert len(c["periods"]) == count
    assert c["periods"][0] == 256
    if count == 2:
        assert c["periods"][1] == round(4096 / 48)


def test_two_bins_rounding_to_one_period():
    # bins 200 and 202 of 4096 points: periods 20.48 and 20.28 both round to
    # 20; both are peaks above the threshold, listed strongest first.  (Of two
    # adjacent bins only the stronger can be a peak.)
    length = 4096
    x = tone(length, [(length / 200, 5.0), (length / 202, 4.5)])
    c = oracle.spectral_candidates(x, 2, 2048)
    assert c["periods"] == [20, 20] and c["bins"] == [200, 202]
    y = tone(length, [(length / 100, 5.0), (length / 101, 4.5)])
    assert oracle.spectral_candidates(y, 2, 2048)["bins"] == [100]


def test_lag_range_and_candidate_limit():
    length = 8192
    bins = [4, 16, 64, 256, 1024]
    x = tone(length, [(length / b, 10.0 - 0.1 * k) for k, b in enumerate(bins)])
    every = oracle.spectral_candidates(x, 2, 4096, c_peak=0.5)
    assert every["bins"] == bins
    ranged = oracle.spectral_candidates(x, 20, 1000, c_peak=0.5)
    assert ranged["periods"] == [512, 128, 32]
    first = oracle.spectral_candidates(x, 2, 4096, c_peak=0.5, k_max=2)
    assert first["bins"] == [4, 16]


def test_channel_weights_add_amplitudes():
    length = 4096
    a = tone(length, [(256, 3.0)])
    b = tone(length, [(64, 2.0)], offset=-5.0)
    w = np.array([2.0, 0.5], dtype=np.float32)
    both = oracle.amplitude_spectrum(np.stack([a, b]), w)
    assert np.allclose(both, 2.0 * oracle.amplitude_spectrum(a) + 0.5 * oracle.amplitude_spectrum(b))


def test_offset_is_removed():
    # samples on a 1/64 grid, so that adding 1024 is exact in fp32
    x = (np.round(tone(3000, [(150, 4.0), (40, 1.0)], offset=0.0).astype(np.float64) * 64) / 64)
    x = x.astype(np.float32)
    y = (x.astype(np.float64) + 1024.0).astype(np.float32)
    a, b = oracle.amplitude_spectrum(x), oracle.amplitude_spectrum(y)
    assert np.allclose(a, b, rtol=0, atol=1e-9 * a.max())
    assert oracle.spectral_candidates(x, 2, 1500)["periods"] == \
        oracle.spectral_candidates(y, 2, 1500)["periods"]
