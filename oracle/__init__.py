"""Plain fp64 CPU oracle for batched iteration-period detection.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the bench's
CPU-baseline leg are the only users.  The product path (the HIP library and its
binding) never imports or calls this package, and this package imports nothing
from the product.

``oracle.c`` (built by ``build()`` with gcc, contraction off, OpenMP) holds the
score, reference and selection definitions; ``brute.py`` holds exact-rational
evaluations used to pin it on tiny inputs.  The definitions follow the paper's
Sec. 4.1.2 (Algorithms 1 and 2) as documented in ``oracle.h``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# GPOEO_ORACLE_LIBRARY names another build of oracle.c to load instead (the
# sanitized build of the CPU sanitizer check); by default the in-tree one.
LIB_PATH = os.environ.get("GPOEO_ORACLE_LIBRARY") or os.path.join(HERE, "liboracle_pd.so")
SAN_LIB_PATH = os.path.join(os.path.dirname(HERE), "_build", "oraclesan", "liboracle_pd.so")

PERIODIC, APERIODIC, CONSTANT = 0, 1, 2
DEFAULT_C_LAG = 0.9
DEFAULT_ERR_MAX = 1.0


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile oracle.c into liboracle_pd.so (always recompiles).  sanitize=True
    builds it with AddressSanitizer and UndefinedBehaviorSanitizer (any finding
    aborts) into SAN_LIB_PATH instead; a process loading that build preloads
    gcc's libasan and libubsan."""
    out = SAN_LIB_PATH if sanitize else os.path.join(HERE, "liboracle_pd.so")
    opt = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer"] if sanitize else ["-O2"]
    cmd = ["gcc", *opt, "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror",
           os.path.join(HERE, "oracle.c"), "-o", out + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    os.makedirs(os.path.dirname(out), exist_ok=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


class _Params(ctypes.Structure):
    _fields_ = [("num_windows", ctypes.c_int64), ("num_channels", ctypes.c_int32),
                ("n", ctypes.c_int64), ("window_stride", ctypes.c_int64),
                ("channel_stride", ctypes.c_int64), ("tmin", ctypes.c_int32),
                ("tmax", ctypes.c_int32), ("c_lag", ctypes.c_double),
                ("err_max", ctypes.c_double), ("channel_weights", ctypes.c_void_p),
                ("centred", ctypes.c_int32)]


class _Out(ctypes.Structure):
    _fields_ = [("period", ctypes.c_int32), ("verdict", ctypes.c_int32), ("err", ctypes.c_double),
                ("n_candidates", ctypes.c_int32), ("t_cand", ctypes.c_int32),
                ("t_low", ctypes.c_int32), ("t_up", ctypes.c_int32), ("n_peaks", ctypes.c_int32),
                ("r", ctypes.c_double), ("s_pk", ctypes.c_double)]


ROLLING_MAX = 32


class _SimilarityParams(ctypes.Structure):
    _fields_ = [("num_groups", ctypes.c_int32), ("em_iters", ctypes.c_int32)]


class _RollingParams(ctypes.Structure):
    _fields_ = [("c_measure", ctypes.c_double), ("step", ctypes.c_double),
                ("c_eval", ctypes.c_double), ("diff_threshold", ctypes.c_double)]


ROLLING_DTYPE = np.dtype([("period", np.int32), ("verdict", np.int32), ("stable", np.int32),
                          ("n_windows", np.int32), ("t_init", np.int32), ("best", np.int32),
                          ("smpdur_next", np.float64), ("diff", np.float64), ("err", np.float64),
                          ("starts", np.int64, ROLLING_MAX), ("periods", np.int32, ROLLING_MAX),
                          ("verdicts", np.int32, ROLLING_MAX), ("errs", np.float64, ROLLING_MAX)],
                         align=True)

OUT_DTYPE = np.dtype([("period", np.int32), ("verdict", np.int32), ("err", np.float64),
                      ("n_candidates", np.int32), ("t_cand", np.int32), ("t_low", np.int32),
                      ("t_up", np.int32), ("n_peaks", np.int32), ("r", np.float64),
                      ("s_pk", np.float64)], align=True)
assert OUT_DTYPE.itemsize == ctypes.sizeof(_Out)

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        lib = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        lib.oracle_pd_reference.restype = ctypes.c_double
        lib.oracle_pd_reference.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                            ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_pd_score.restype = ctypes.c_double
        lib.oracle_pd_score.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                        ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_pd_score_centred.restype = ctypes.c_double
        lib.oracle_pd_score_centred.argtypes = lib.oracle_pd_score.argtypes
        lib.oracle_pd_select.restype = None
        lib.oracle_pd_select.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                         ctypes.c_int32, ctypes.c_double, ctypes.c_double,
                                         ctypes.c_double, P(_Out)]
        lib.oracle_pd_detect.restype = ctypes.c_int
        lib.oracle_pd_detect.argtypes = [P(_Params), ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_void_p]
        lib.oracle_pd_score_list.restype = ctypes.c_int
        lib.oracle_pd_score_list.argtypes = [P(_Params), ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_pd_rolling.restype = ctypes.c_int
        lib.oracle_pd_rolling.argtypes = [P(_Params), P(_RollingParams), ctypes.c_void_p,
                                          ctypes.c_void_p]
        lib.oracle_pd_rolling_schedule.restype = ctypes.c_int32
        lib.oracle_pd_rolling_schedule.argtypes = [ctypes.c_int64, ctypes.c_int32,
                                                   P(_RollingParams), ctypes.c_void_p,
                                                   ctypes.c_int32, P(ctypes.c_double)]
        lib.oracle_pd_similarity.restype = ctypes.c_int
        lib.oracle_pd_similarity.argtypes = [P(_Params), P(_SimilarityParams), ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                             ctypes.c_void_p]
        lib.oracle_pd_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    return int(_load().oracle_pd_threads())


@dataclass
class Layout:
    num_windows: int
    num_channels: int
    n: int
    window_stride: int
    channel_stride: int
    tmin: int
    tmax: int
    c_lag: float = DEFAULT_C_LAG
    err_max: float = DEFAULT_ERR_MAX
    weights: np.ndarray | None = None
    centred: bool = False      # score with Algorithm 2's per-sub-curve mean removal

    @classmethod
    def of(cls, wl, **kw) -> "Layout":
        """Layout of a gen.Workload (duck-typed), optionally overriding fields."""
        d = dict(num_windows=wl.num_windows, num_channels=wl.num_channels, n=wl.n,
                 window_stride=wl.window_stride, channel_stride=wl.channel_stride,
                 tmin=wl.tmin, tmax=wl.tmax, weights=wl.weights)
        d.update(kw)
        return cls(**d)

    @property
    def lags(self) -> int:
        return self.tmax - self.tmin + 1


def _params(lay: Layout, keep: list) -> _Params:
    w = None
    if lay.weights is not None:
        w = np.ascontiguousarray(lay.weights, dtype=np.float32)
        keep.append(w)
    return _Params(lay.num_windows, lay.num_channels, lay.n, lay.window_stride,
                   lay.channel_stride, lay.tmin, lay.tmax, float(lay.c_lag), float(lay.err_max),
                   None if w is None else w.ctypes.data, 1 if lay.centred else 0)


def _as_f32(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x)
    if x.dtype != np.float32:
        raise TypeError("oracle inputs are float32 sample buffers")
    return x.reshape(-1)


def _check_extent(x: np.ndarray, lay: Layout) -> None:
    need = ((lay.num_windows - 1) * lay.window_stride
            + (lay.num_channels - 1) * lay.channel_stride + lay.n)
    if x.size < need:
        raise ValueError(f"buffer has {x.size} samples, layout needs {need}")


def detect(x: np.ndarray, lay: Layout, want_scores: bool = True):
    """Scores [B][L] (fp64, or None) and one result record per window."""
    x = _as_f32(x)
    _check_extent(x, lay)
    keep: list = []
    p = _params(lay, keep)
    scores = np.empty((lay.num_windows, lay.lags), dtype=np.float64) if want_scores else None
    out = np.zeros(lay.num_windows, dtype=OUT_DTYPE)
    rc = _load().oracle_pd_detect(ctypes.byref(p), x.ctypes.data,
                                  None if scores is None else scores.ctypes.data,
                                  out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the parameters")
    return scores, out


def score_list(x: np.ndarray, lay: Layout, windows, lags) -> np.ndarray:
    """S(T) for the given (window, lag) pairs, each one plain sequential fp64 sum."""
    x = _as_f32(x)
    _check_extent(x, lay)
    w = np.ascontiguousarray(windows, dtype=np.int64)
    t = np.ascontiguousarray(lags, dtype=np.int32)
    if w.shape != t.shape:
        raise ValueError("windows and lags differ in length")
    keep: list = []
    p = _params(lay, keep)
    out = np.empty(w.shape, dtype=np.float64)
    rc = _load().oracle_pd_score_list(ctypes.byref(p), x.ctypes.data, w.ctypes.data,
                                      t.ctypes.data, int(w.size), out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the parameters")
    return out


def score(xw: np.ndarray, t: int, weights=None) -> float:
    """S(T) of one window given as [C][N] (or [N]) float32."""
    xw = np.ascontiguousarray(np.atleast_2d(xw), dtype=np.float32)
    c, n = xw.shape
    w = None if weights is None else np.ascontiguousarray(weights, dtype=np.float32)
    return float(_load().oracle_pd_score(xw.ctypes.data, c, n, n, int(t),
                                         None if w is None else w.ctypes.data))


def score_centred(xw: np.ndarray, t: int, weights=None) -> float:
    """S_c(T), the mean-removed score, of one window given as [C][N] (or [N]) float32."""
    xw = np.ascontiguousarray(np.atleast_2d(xw), dtype=np.float32)
    c, n = xw.shape
    w = None if weights is None else np.ascontiguousarray(weights, dtype=np.float32)
    return float(_load().oracle_pd_score_centred(xw.ctypes.data, c, n, n, int(t),
                                                 None if w is None else w.ctypes.data))


def reference(xw: np.ndarray, weights=None) -> float:
    """R = 2 * sum_c w_c * Var_c of one window given as [C][N] (or [N]) float32."""
    xw = np.ascontiguousarray(np.atleast_2d(xw), dtype=np.float32)
    c, n = xw.shape
    w = None if weights is None else np.ascontiguousarray(weights, dtype=np.float32)
    return float(_load().oracle_pd_reference(xw.ctypes.data, c, n, n,
                                             None if w is None else w.ctypes.data))


def select(s: np.ndarray, n: int, tmin: int, tmax: int, r: float,
           c_lag: float = DEFAULT_C_LAG, err_max: float = DEFAULT_ERR_MAX) -> dict:
    """The selection rule on one score row s[j] = S(tmin + j)."""
    s = np.ascontiguousarray(s, dtype=np.float64)
    if s.shape != (tmax - tmin + 1,):
        raise ValueError("score row length must be tmax - tmin + 1")
    o = _Out()
    _load().oracle_pd_select(s.ctypes.data, int(n), int(tmin), int(tmax), float(r),
                             float(c_lag), float(err_max), ctypes.byref(o))
    return {name: getattr(o, name) for name, _ in _Out._fields_}


# Algorithm 3's constants as the paper sets them (Sec. 4.1.3); the stability
# threshold on the relative period spread is not given there.
C_MEASURE, STEP, C_EVAL = 2.0, 0.5, 6.5
DEFAULT_DIFF_THRESHOLD = 0.05


def rolling(x: np.ndarray, lay: Layout, c_measure: float = C_MEASURE, step: float = STEP,
            c_eval: float = C_EVAL, diff_threshold: float = DEFAULT_DIFF_THRESHOLD) -> np.ndarray:
    """Algorithm 3 on every window of the batch: one ROLLING_DTYPE record each."""
    x = _as_f32(x)
    _check_extent(x, lay)
    keep: list = []
    p = _params(lay, keep)
    rp = _RollingParams(float(c_measure), float(step), float(c_eval), float(diff_threshold))
    out = np.zeros(lay.num_windows, dtype=ROLLING_DTYPE)
    rc = _load().oracle_pd_rolling(ctypes.byref(p), ctypes.byref(rp), x.ctypes.data,
                                   out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the parameters")
    return out


def rolling_schedule(n: int, t_init: int, c_measure: float = C_MEASURE, step: float = STEP,
                     c_eval: float = C_EVAL):
    """(suffix start samples, too-short next duration) of Algorithm 3's schedule."""
    rp = _RollingParams(float(c_measure), float(step), float(c_eval), 0.0)
    starts = np.zeros(ROLLING_MAX, dtype=np.int64)
    nxt = ctypes.c_double()
    k = _load().oracle_pd_rolling_schedule(int(n), int(t_init), ctypes.byref(rp),
                                           starts.ctypes.data, ROLLING_MAX, ctypes.byref(nxt))
    if k < 0:
        raise ValueError("schedule longer than the oracle's limit")
    return starts[:k].tolist(), nxt.value


# Algorithm 2's group count and EM iterations are not given by the paper.
DEFAULT_GROUPS, DEFAULT_EM_ITERS = 3, 20


def similarity(x: np.ndarray, lay: Layout, windows, lags, num_groups: int = DEFAULT_GROUPS,
               em_iters: int = DEFAULT_EM_ITERS) -> np.ndarray:
    """Algorithm 2's Err_T for the given (window, lag) pairs (-1: fewer than two sub-curves)."""
    x = _as_f32(x)
    _check_extent(x, lay)
    w = np.ascontiguousarray(windows, dtype=np.int64)
    t = np.ascontiguousarray(lags, dtype=np.int32)
    if w.shape != t.shape:
        raise ValueError("windows and lags differ in length")
    keep: list = []
    p = _params(lay, keep)
    sp = _SimilarityParams(int(num_groups), int(em_iters))
    out = np.empty(w.shape, dtype=np.float64)
    rc = _load().oracle_pd_similarity(ctypes.byref(p), ctypes.byref(sp), x.ctypes.data,
                                      w.ctypes.data, t.ctypes.data, int(w.size), out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the parameters")
    return out


# Algorithm 1, lines 1-5 (Sec. 4.1.1-4.1.2): the FFT front end.  c_peak is
# 0.6-0.7 in the paper; the mid value is the default.
DEFAULT_C_PEAK = 0.65
SPECTRAL_MAX = 16


def spectral_length(n: int) -> int:
    """Transform length: the smallest power of two (at least 64) holding the window."""
    length = 64
    while length < n:
        length *= 2
    return length


def amplitude_spectrum(xw: np.ndarray, weights=None) -> np.ndarray:
    """A(k) = sum_c w_c |X_c(k)|, k = 0..L/2, of one window [C][N] (or [N]).

    Each channel is centred by its mean (the transform of the constant part is
    a peak at k = 0 only) and zero-padded to L = spectral_length(N); X_c is its
    fp64 discrete Fourier transform (numpy's FFT, a library primitive)."""
    xw = np.atleast_2d(np.asarray(xw, dtype=np.float32)).astype(np.float64)
    c_count, n = xw.shape
    length = spectral_length(n)
    w = np.ones(c_count) if weights is None else np.asarray(weights, dtype=np.float32).astype(np.float64)
    amp = np.zeros(length // 2 + 1)
    for c in range(c_count):
        y = xw[c] - xw[c].sum() / n
        amp += w[c] * np.abs(np.fft.rfft(y, n=length))
    return amp


def spectral_candidates(xw: np.ndarray, tmin: int, tmax: int, c_peak: float = DEFAULT_C_PEAK,
                        k_max: int = SPECTRAL_MAX, weights=None) -> dict:
    """Candidate periods of one window from its amplitude spectrum (Algorithm 1,
    lines 1-5, with T_s = 1 sample):

      peaks   bins 2 <= k <= L/2 - 1 with A(k) > A(k-1) and A(k) >= A(k+1)
              (strict on the left, as the lag-domain rule)
      cands   peaks with A(k) > c_peak * max over peaks whose period
              round(L / k) (halves up) lies in [tmin, tmax]
      order   decreasing A (ties: smaller k), at most k_max of them; two bins
              may round to the same period (the paper's TCand is a list of
              peak periods, not a set)
    """
    amp = amplitude_spectrum(xw, weights)
    half = amp.size - 1
    k = np.arange(2, half)
    peak = (amp[k] > amp[k - 1]) & (amp[k] >= amp[k + 1])
    pk = k[peak]
    out = {"periods": [], "bins": [], "amplitudes": [], "n_peaks": int(pk.size), "max_peak": 0.0}
    if pk.size == 0:
        return out
    top = amp[pk].max()
    out["max_peak"] = float(top)
    cand = pk[amp[pk] > c_peak * top]
    order = sorted(cand.tolist(), key=lambda b: (-amp[b], b))
    length = 2 * half
    for b in order:
        t = (2 * length + b) // (2 * b)          # round(L / b), halves up
        if t < tmin or t > tmax:
            continue
        out["periods"].append(int(t))
        out["bins"].append(int(b))
        out["amplitudes"].append(float(amp[b]))
        if len(out["periods"]) == k_max:
            break
    return out
