"""Synthetic sampled-feature traces with a planted iteration period.

The paper's inputs are power, SM-utilisation, memory-utilisation and counter
traces of ML training jobs sampled at a fixed interval (Sec. 4.1, Sec. 4.2); none
of those recordings are available, so these generators stand in for them.  A
trace is one period-long *template* of K piecewise-constant levels, tiled over
the trace, plus i.i.d. Gaussian noise and, per workload, random spikes or
per-repeat length jitter.  Everything is drawn from ``numpy.random.default_rng``
with a fixed seed, in a fixed order per trace:

    P, K, cut points, levels, (jitter factors | spike mask), noise

Cut points are K-1 distinct integers drawn without replacement from
{1, ..., P-1} and sorted, so the K segment lengths are a random composition of P.

Five named workloads (``WORKLOADS``) follow the five trace configurations the
method is measured on; ``make_workload(name, ...)`` can shrink the batch, the
trace length and the lag range for tests the CPU oracle must finish quickly.

No function here computes anything of the period-detection method.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np


@dataclass
class Workload:
    """A batch of windows in one flat fp32 buffer plus its layout.

    Window ``b``, channel ``c``, sample ``i`` lives at
    ``x[b * window_stride + c * channel_stride + i]``.
    """

    name: str
    x: np.ndarray                  # flat float32 buffer
    num_windows: int
    num_channels: int
    n: int
    window_stride: int
    channel_stride: int
    tmin: int
    tmax: int
    truth: np.ndarray              # planted period per window (int64), -1 where undefined
    jitter: bool = False           # planted period only approximate (length jitter)
    weights: np.ndarray | None = None
    meta: dict = field(default_factory=dict)

    @property
    def lags(self) -> int:
        return self.tmax - self.tmin + 1

    @property
    def sha256(self) -> str:
        return hashlib.sha256(np.ascontiguousarray(self.x).tobytes()).hexdigest()

    def pairs(self) -> int:
        """Number of (x[i], x[i+T]) evaluations over all windows, channels and lags."""
        t = np.arange(self.tmin, self.tmax + 1, dtype=np.int64)
        per_window = int(np.sum(self.n - t))
        return per_window * self.num_windows * self.num_channels

    def window(self, b: int) -> np.ndarray:
        """[C][N] float32 view of window b."""
        base = b * self.window_stride
        rows = [self.x[base + c * self.channel_stride: base + c * self.channel_stride + self.n]
                for c in range(self.num_channels)]
        return np.stack(rows)


def _cuts(rng: np.random.Generator, period: int, k: int) -> np.ndarray:
    """Segment lengths of a random composition of ``period`` into ``k`` parts."""
    if k < 1 or k > period:
        raise ValueError(f"cannot split period {period} into {k} segments")
    cut = np.sort(rng.choice(np.arange(1, period), size=k - 1, replace=False))
    edges = np.concatenate(([0], cut, [period]))
    return np.diff(edges).astype(np.int64)


def _template(levels: np.ndarray, lengths: np.ndarray) -> np.ndarray:
    return np.repeat(np.asarray(levels, dtype=np.float64), lengths)


def _tile(template: np.ndarray, n: int, start: int = 0) -> np.ndarray:
    """template[(i + start) mod P] for i < n, as a cyclic copy."""
    p = template.shape[0]
    return np.resize(np.roll(template, -(start % p)), n)


def planted_trace(n: int, period: int, k: int, *, seed: int = 0, lo: float = 100.0,
                  hi: float = 350.0, sigma: float = 2.0, integer: bool = False) -> np.ndarray:
    """One float32 trace of length n: a K-level template of length ``period`` tiled, plus noise.

    ``integer=True`` rounds the levels to integers and draws no noise, so every
    sample is an exactly representable small integer (useful for exact-tie tests).
    """
    rng = np.random.default_rng(seed)
    lengths = _cuts(rng, period, k)
    levels = rng.uniform(lo, hi, size=k)
    if integer:
        levels = np.round(levels)
    clean = _tile(_template(levels, lengths), n)
    if integer or sigma == 0.0:
        return clean.astype(np.float32)
    return (clean + rng.normal(0.0, sigma, size=n)).astype(np.float32)


# ---------------------------------------------------------------------------
# The five workloads.  Each builder takes (seed, traces, n, tmax) so that tests
# can shrink them; the defaults are the full sizes.
# ---------------------------------------------------------------------------

def _w1(seed=0, traces=1, n=4096, tmax=1024, tmin=2):
    rng = np.random.default_rng(seed)
    out = np.empty((traces, n), dtype=np.float32)
    truth = np.empty(traces, dtype=np.int64)
    for b in range(traces):
        p, k = 137, 6
        lengths = _cuts(rng, p, k)
        levels = rng.uniform(100.0, 350.0, size=k)
        clean = _tile(_template(levels, lengths), n)
        out[b] = (clean + rng.normal(0.0, 2.0, size=n)).astype(np.float32)
        truth[b] = p
    return out.reshape(-1), traces, 1, n, n, n, tmin, tmax, truth, False


def _w2(seed=1, traces=64, n=65536, tmax=8192, tmin=2, pmax=5000):
    rng = np.random.default_rng(seed)
    out = np.empty((traces, n), dtype=np.float32)
    truth = np.empty(traces, dtype=np.int64)
    for b in range(traces):
        p = int(rng.integers(50, pmax + 1))
        k = int(rng.integers(4, 13))
        lengths = _cuts(rng, p, k)
        levels = rng.uniform(80.0, 400.0, size=k)
        reps = int(np.ceil(n / (0.98 * p))) + 2
        f = rng.uniform(0.98, 1.02, size=reps)
        pieces = []
        total = 0
        for r in range(reps):
            seg = np.maximum(1, np.rint(lengths * f[r]).astype(np.int64))
            pieces.append(_template(levels, seg))
            total += int(seg.sum())
            if total >= n:
                break
        clean = np.concatenate(pieces)[:n]
        if clean.shape[0] < n:
            raise AssertionError("jittered repeats do not cover the trace")
        out[b] = (clean + rng.normal(0.0, 3.0, size=n)).astype(np.float32)
        truth[b] = p
    return out.reshape(-1), traces, 1, n, n, n, tmin, tmax, truth, True


def _w3(seed=2, traces=1024, n=262144, tmax=32768, tmin=2, pmax=20000):
    rng = np.random.default_rng(seed)
    out = np.empty((traces, n), dtype=np.float32)
    truth = np.empty(traces, dtype=np.int64)
    for b in range(traces):
        p = int(np.rint(np.exp(rng.uniform(np.log(100.0), np.log(pmax)))))
        k = int(rng.integers(8, 33))
        lengths = _cuts(rng, p, k)
        levels = rng.uniform(80.0, 400.0, size=k)
        spikes = rng.random(n) < 0.05
        clean = _tile(_template(levels, lengths), n) + 50.0 * spikes
        out[b] = (clean + rng.normal(0.0, 5.0, size=n)).astype(np.float32)
        truth[b] = p
    return out.reshape(-1), traces, 1, n, n, n, tmin, tmax, truth, False


def _w4(seed=3, total=8_388_608, n=16384, stride=2048, tmax=4096, tmin=2,
        p1=900, p2=1430, switch=None):
    rng = np.random.default_rng(seed)
    if switch is None:
        switch = total // 2
    l1 = _cuts(rng, p1, 8)
    v1 = rng.uniform(100.0, 350.0, size=8)
    l2 = _cuts(rng, p2, 8)
    v2 = rng.uniform(100.0, 350.0, size=8)
    clean = np.concatenate((_tile(_template(v1, l1), switch),
                            _tile(_template(v2, l2), total - switch)))
    x = (clean + rng.normal(0.0, 3.0, size=total)).astype(np.float32)
    windows = (total - n) // stride + 1
    truth = np.full(windows, -1, dtype=np.int64)
    starts = np.arange(windows, dtype=np.int64) * stride
    truth[starts + n <= switch] = p1
    truth[starts >= switch] = p2
    return x, windows, 1, n, stride, n, tmin, tmax, truth, False


def _w5(seed=4, traces=256, n=131072, tmax=16384, tmin=2, channels=8, pmax=8000):
    rng = np.random.default_rng(seed)
    out = np.empty((traces, channels, n), dtype=np.float32)
    truth = np.empty(traces, dtype=np.int64)
    for b in range(traces):
        p = int(rng.integers(200, pmax + 1))
        k = int(rng.integers(4, 13))
        lengths = _cuts(rng, p, k)
        lv = np.empty((channels, k))
        for c in range(channels):
            if c == 0:
                lv[c] = rng.uniform(80.0, 400.0, size=k)          # power, W
            elif c < 4:
                lv[c] = rng.uniform(0.0, 1.0, size=k)             # SM / memory / DRAM utilisation
            else:
                lv[c] = np.exp(rng.uniform(np.log(1e3), np.log(1e6), size=k))  # counters
        for c in range(channels):
            clean = _tile(_template(lv[c], lengths), n)
            z = (clean - clean.mean()) / clean.std()
            out[b, c] = (z + rng.normal(0.0, 0.05, size=n)).astype(np.float32)
        truth[b] = p
    return out.reshape(-1), traces, channels, n, channels * n, n, tmin, tmax, truth, False


WORKLOADS = {
    "w1": (_w1, "1 trace x 4096 samples, P=137, 6 levels U[100,350] W, sigma 2 W, T in [2,1024]"),
    "w2": (_w2, "64 traces x 65536 samples, P~U{50..5000}, 4-12 levels U[80,400] W, "
                "per-repeat length jitter +-2%, sigma 3 W, T in [2,8192]"),
    "w3": (_w3, "1024 traces x 262144 samples, P log-uniform in [100,20000], 8-32 levels "
                "U[80,400] W, 5% +50 W one-sample spikes, sigma 5 W, T in [2,32768]"),
    "w4": (_w4, "one 8388608-sample trace, P=900 then P=1430 from sample 4194304, 4089 sliding "
                "windows of 16384 at stride 2048, sigma 3 W, T in [2,4096]"),
    "w5": (_w5, "256 traces x 8 channels x 131072 samples, shared P~U{200..8000}, z-normalised "
                "channels + N(0,0.05^2), channel scores summed, T in [2,16384]"),
}


def make_workload(name: str, **overrides) -> Workload:
    """Build a named workload; keyword overrides shrink it (traces=, n=, tmax=, total=, ...)."""
    if name not in WORKLOADS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}")
    builder, desc = WORKLOADS[name]
    x, b, c, n, ws, cs, tmin, tmax, truth, jitter = builder(**overrides)
    return Workload(name=name, x=x, num_windows=b, num_channels=c, n=n, window_stride=ws,
                    channel_stride=cs, tmin=tmin, tmax=tmax, truth=truth, jitter=jitter,
                    meta={"description": desc, "overrides": dict(overrides)})
