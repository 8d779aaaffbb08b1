"""ctypes binding of libgpoeo_pd.so (argument marshalling only).

Every step of the detection runs in the library's HIP kernels; this module
only builds the descriptor, hands over device pointers of torch tensors and the
current HIP stream, and allocates the caller-side buffers (scores, results,
workspace) with torch.  If the library is missing it raises: there is no other
code path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # noqa: F401  (loads the HIP runtime the library must share)

HERE = os.path.dirname(os.path.abspath(__file__))
# GPOEO_PD_LIBRARY names another build of the same library to load instead (the
# host-sanitized build of the CPU sanitizer check); by default the in-tree one.
LIB_PATH = os.environ.get("GPOEO_PD_LIBRARY") or os.path.join(HERE, "libgpoeo_pd.so")

OK, EINVAL, ENOMEM, EHIP, ETOOBIG = 0, -1, -2, -3, -4
PERIODIC, APERIODIC, CONSTANT = 0, 1, 2
SCORES_ONLY, NO_RESCUE, FFT_SCORES, MFMA_SCORES, UNFUSED = 1, 2, 4, 8, 16
FUSED_MAX_N = 16384          # GPOEO_PD_FUSED_MAX_N
UNRESOLVED, SHORT, TIER2 = 1, 2, 4
DEFAULT_C_LAG = 0.9
DEFAULT_ERR_MAX = 1.0


class Desc(ctypes.Structure):
    _fields_ = [("num_windows", ctypes.c_int64), ("num_channels", ctypes.c_int32),
                ("reserved0", ctypes.c_int32), ("n", ctypes.c_int64),
                ("window_stride", ctypes.c_int64), ("channel_stride", ctypes.c_int64),
                ("tmin", ctypes.c_int32), ("tmax", ctypes.c_int32), ("c_lag", ctypes.c_double),
                ("err_max", ctypes.c_double), ("channel_weights", ctypes.c_void_p),
                ("flags", ctypes.c_uint32), ("reserved1", ctypes.c_uint32)]


class Result(ctypes.Structure):
    _fields_ = [("period", ctypes.c_int32), ("verdict", ctypes.c_int32), ("err", ctypes.c_float),
                ("n_candidates", ctypes.c_int32), ("t_cand", ctypes.c_int32),
                ("t_low", ctypes.c_int32), ("t_up", ctypes.c_int32), ("n_rescored", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("lags_per_lane", ctypes.c_int32),
                ("score_waves", ctypes.c_int64), ("pairs_defined", ctypes.c_double),
                ("pairs_scored", ctypes.c_double), ("workspace_bytes", ctypes.c_size_t),
                ("fft_len", ctypes.c_int64), ("fft_wrap_len", ctypes.c_int64),
                ("fft_wrap_lags", ctypes.c_int64)]


ROLLING_MAX = 16
MAX_WINDOWS = 1 << 21       # GPOEO_PD_MAX_WINDOWS
MAX_QUERIES = 1 << 23       # GPOEO_PD_MAX_QUERIES
MAX_CHANNELS = 256          # GPOEO_PD_MAX_CHANNELS


class RollingParams(ctypes.Structure):
    _fields_ = [("c_measure", ctypes.c_double), ("step", ctypes.c_double),
                ("c_eval", ctypes.c_double), ("diff_threshold", ctypes.c_double)]


class RollingResult(ctypes.Structure):
    _fields_ = [("period", ctypes.c_int32), ("verdict", ctypes.c_int32),
                ("stable", ctypes.c_int32), ("n_windows", ctypes.c_int32),
                ("t_init", ctypes.c_int32), ("best", ctypes.c_int32),
                ("smpdur_next", ctypes.c_double), ("diff", ctypes.c_float),
                ("err", ctypes.c_float), ("flags", ctypes.c_uint32), ("reserved", ctypes.c_int32),
                ("periods", ctypes.c_int32 * ROLLING_MAX), ("starts", ctypes.c_int64 * ROLLING_MAX)]


ROLLING_DTYPE = np.dtype([("period", np.int32), ("verdict", np.int32), ("stable", np.int32),
                          ("n_windows", np.int32), ("t_init", np.int32), ("best", np.int32),
                          ("smpdur_next", np.float64), ("diff", np.float32), ("err", np.float32),
                          ("flags", np.uint32), ("reserved", np.int32),
                          ("periods", np.int32, ROLLING_MAX), ("starts", np.int64, ROLLING_MAX)])
assert ROLLING_DTYPE.itemsize == ctypes.sizeof(RollingResult)

# Algorithm 3's constants as the paper sets them (Sec. 4.1.3); the paper gives
# no value for the stability threshold on the relative period spread.
C_MEASURE, STEP, C_EVAL, DEFAULT_DIFF_THRESHOLD = 2.0, 0.5, 6.5, 0.05

class SimilarityParams(ctypes.Structure):
    _fields_ = [("num_groups", ctypes.c_int32), ("em_iters", ctypes.c_int32)]


SPECTRAL_MAX = 16
DEFAULT_C_PEAK = 0.65          # the paper sets c_peak to 0.6-0.7


class SpectralParams(ctypes.Structure):
    _fields_ = [("c_peak", ctypes.c_double), ("max_candidates", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


SPECTRAL_DTYPE = np.dtype([("count", np.int32), ("flags", np.uint32), ("n_peaks", np.int32),
                           ("reserved", np.int32), ("max_peak", np.float64),
                           ("periods", np.int32, SPECTRAL_MAX), ("bins", np.int32, SPECTRAL_MAX),
                           ("amplitudes", np.float64, SPECTRAL_MAX)])
assert SPECTRAL_DTYPE.itemsize == 280


# Algorithm 2's group count and EM iterations are not given by the paper.
DEFAULT_GROUPS, DEFAULT_EM_ITERS = 3, 20

RESULT_DTYPE = np.dtype([("period", np.int32), ("verdict", np.int32), ("err", np.float32),
                         ("n_candidates", np.int32), ("t_cand", np.int32), ("t_low", np.int32),
                         ("t_up", np.int32), ("n_rescored", np.int32), ("flags", np.uint32)])
RESULT_WORDS = ctypes.sizeof(Result) // 4
assert RESULT_DTYPE.itemsize == ctypes.sizeof(Result)

EXPORTS = ("gpoeo_pd_abi_version", "gpoeo_pd_strerror", "gpoeo_pd_workspace_bytes",
           "gpoeo_pd_describe_plan", "gpoeo_pd_detect", "gpoeo_pd_detect_staged",
           "gpoeo_pd_rolling_workspace_bytes", "gpoeo_pd_detect_rolling", "gpoeo_pd_similarity",
           "gpoeo_pd_score_centred", "gpoeo_pd_spectral_workspace_bytes",
           "gpoeo_pd_spectral_candidates", "gpoeo_pd_detect_noalloc",
           "gpoeo_pd_similarity_flagged")
NOALLOC_MAX_WORKSPACE = 64 << 20   # GPOEO_PD_NOALLOC_MAX_WORKSPACE

_lib = None


def load_library():
    """Load libgpoeo_pd.so (built in-tree); raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(python paper_2201_01684_amd/build.py)")
        lib = ctypes.CDLL(LIB_PATH)
        lib.gpoeo_pd_abi_version.restype = ctypes.c_int
        lib.gpoeo_pd_abi_version.argtypes = []
        lib.gpoeo_pd_strerror.restype = ctypes.c_char_p
        lib.gpoeo_pd_strerror.argtypes = [ctypes.c_int]
        lib.gpoeo_pd_workspace_bytes.restype = ctypes.c_int
        lib.gpoeo_pd_workspace_bytes.argtypes = [ctypes.POINTER(Desc),
                                                 ctypes.POINTER(ctypes.c_size_t)]
        lib.gpoeo_pd_describe_plan.restype = ctypes.c_int
        lib.gpoeo_pd_describe_plan.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(PlanInfo)]
        lib.gpoeo_pd_detect.restype = ctypes.c_int
        lib.gpoeo_pd_detect.argtypes = [ctypes.POINTER(Desc), ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                        ctypes.c_void_p]
        lib.gpoeo_pd_detect_noalloc.restype = ctypes.c_int
        lib.gpoeo_pd_detect_noalloc.argtypes = [ctypes.POINTER(Desc), ctypes.c_void_p,
                                                ctypes.c_void_p, ctypes.c_void_p,
                                                ctypes.c_void_p]
        lib.gpoeo_pd_detect_staged.restype = ctypes.c_int
        lib.gpoeo_pd_detect_staged.argtypes = [ctypes.POINTER(Desc), ctypes.c_void_p,
                                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                               ctypes.c_size_t, ctypes.c_void_p,
                                               ctypes.c_void_p]
        lib.gpoeo_pd_rolling_workspace_bytes.restype = ctypes.c_int
        lib.gpoeo_pd_rolling_workspace_bytes.argtypes = [ctypes.POINTER(Desc),
                                                         ctypes.POINTER(RollingParams),
                                                         ctypes.POINTER(ctypes.c_size_t)]
        lib.gpoeo_pd_detect_rolling.restype = ctypes.c_int
        lib.gpoeo_pd_detect_rolling.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(RollingParams),
                                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                ctypes.c_size_t, ctypes.c_void_p]
        lib.gpoeo_pd_score_centred.restype = ctypes.c_int
        lib.gpoeo_pd_score_centred.argtypes = [ctypes.POINTER(Desc), ctypes.c_void_p,
                                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                               ctypes.c_void_p, ctypes.c_void_p]
        lib.gpoeo_pd_similarity.restype = ctypes.c_int
        lib.gpoeo_pd_similarity.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(SimilarityParams),
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        lib.gpoeo_pd_similarity_flagged.restype = ctypes.c_int
        lib.gpoeo_pd_similarity_flagged.argtypes = [ctypes.POINTER(Desc),
                                                    ctypes.POINTER(SimilarityParams),
                                                    ctypes.c_void_p, ctypes.c_void_p,
                                                    ctypes.c_void_p, ctypes.c_int64,
                                                    ctypes.c_void_p, ctypes.c_void_p,
                                                    ctypes.c_void_p]
        lib.gpoeo_pd_spectral_workspace_bytes.restype = ctypes.c_int
        lib.gpoeo_pd_spectral_workspace_bytes.argtypes = [ctypes.POINTER(Desc),
                                                          ctypes.POINTER(SpectralParams),
                                                          ctypes.POINTER(ctypes.c_size_t)]
        lib.gpoeo_pd_spectral_candidates.restype = ctypes.c_int
        lib.gpoeo_pd_spectral_candidates.argtypes = [ctypes.POINTER(Desc),
                                                     ctypes.POINTER(SpectralParams),
                                                     ctypes.c_void_p, ctypes.c_void_p,
                                                     ctypes.c_void_p, ctypes.c_size_t,
                                                     ctypes.c_void_p]
        _lib = lib
    return _lib


def strerror(status: int) -> str:
    return load_library().gpoeo_pd_strerror(int(status)).decode()


class GpoeoError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {strerror(status)} ({status})")
        self.status = status


def make_desc(num_windows, num_channels, n, window_stride, channel_stride, tmin, tmax,
              c_lag=DEFAULT_C_LAG, err_max=DEFAULT_ERR_MAX, weights=None, flags=0):
    """Descriptor plus the host weight array it points at (keep both alive)."""
    w = None
    if weights is not None:
        w = np.ascontiguousarray(weights, dtype=np.float32)
        if w.shape != (num_channels,):
            raise ValueError("need one weight per channel")
    d = Desc(int(num_windows), int(num_channels), 0, int(n), int(window_stride),
             int(channel_stride), int(tmin), int(tmax), float(c_lag), float(err_max),
             None if w is None else w.ctypes.data, int(flags), 0)
    return d, w


def workspace_bytes(desc: Desc) -> int:
    size = ctypes.c_size_t(0)
    rc = load_library().gpoeo_pd_workspace_bytes(ctypes.byref(desc), ctypes.byref(size))
    if rc != OK:
        raise GpoeoError(rc, "gpoeo_pd_workspace_bytes")
    return int(size.value)


def describe_plan(desc: Desc) -> dict:
    """The launch plan of a descriptor: mode, lags per lane, waves, pair counts."""
    info = PlanInfo()
    rc = load_library().gpoeo_pd_describe_plan(ctypes.byref(desc), ctypes.byref(info))
    if rc != OK:
        raise GpoeoError(rc, "gpoeo_pd_describe_plan")
    return {name: getattr(info, name) for name, _ in PlanInfo._fields_}


def _stream_handle(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


class Detector:
    """Reusable call site: device buffers allocated once, then `run()` only enqueues.

    ``x`` is a float32 device tensor holding all windows (any shape; its
    storage is addressed with the layout in the descriptor).
    """

    def __init__(self, x: torch.Tensor, desc: Desc, weights_keepalive=None, want_scores=True):
        if not isinstance(x, torch.Tensor) or x.dtype != torch.float32 or not x.is_cuda:
            raise TypeError("x must be a float32 GPU tensor")
        if not x.is_contiguous():
            raise ValueError("x must be contiguous")
        need = ((desc.num_windows - 1) * desc.window_stride
                + (desc.num_channels - 1) * desc.channel_stride + desc.n)
        if x.numel() < need:
            raise ValueError(f"x has {x.numel()} samples, the layout addresses {need}")
        self.x = x
        self.desc = desc
        self._w = weights_keepalive
        dev = x.device
        lags = desc.tmax - desc.tmin + 1
        self.scores = (torch.empty((desc.num_windows, lags), dtype=torch.float32, device=dev)
                       if want_scores else None)
        self.results = torch.zeros((desc.num_windows, RESULT_WORDS), dtype=torch.int32,
                                   device=dev)
        self.ws_bytes = workspace_bytes(desc)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=dev)
        self._lib = load_library()

    def run(self, stream=None) -> None:
        rc = self._lib.gpoeo_pd_detect(
            ctypes.byref(self.desc), self.x.data_ptr(),
            None if self.scores is None else self.scores.data_ptr(),
            self.results.data_ptr(), self.workspace.data_ptr(), self.ws_bytes,
            _stream_handle(stream))
        if rc != OK:
            raise GpoeoError(rc, "gpoeo_pd_detect")

    def run_staged(self, events, stream=None) -> None:
        """run(), recording the five caller-created hipEvent_t handles in ``events``
        (a ctypes array of 5 void pointers) around the four stages."""
        rc = self._lib.gpoeo_pd_detect_staged(
            ctypes.byref(self.desc), self.x.data_ptr(),
            None if self.scores is None else self.scores.data_ptr(),
            self.results.data_ptr(), self.workspace.data_ptr(), self.ws_bytes,
            _stream_handle(stream), events)
        if rc != OK:
            raise GpoeoError(rc, "gpoeo_pd_detect_staged")

    def results_numpy(self) -> np.ndarray:
        return results_to_numpy(self.results)


def results_to_numpy(results: torch.Tensor) -> np.ndarray:
    host = results.detach().to("cpu").contiguous().numpy()
    return host.view(RESULT_DTYPE).reshape(-1)


class DetectParams:
    """Selection parameters and flags of one detect_period call (defaults: c_lag 0.9,
    err_max 1.0, no flags)."""

    def __init__(self, c_lag: float = DEFAULT_C_LAG, err_max: float = DEFAULT_ERR_MAX,
                 flags: int = 0, weights=None):
        self.c_lag, self.err_max, self.flags, self.weights = c_lag, err_max, flags, weights


def detect_period(traces: torch.Tensor, n: int | None, tmin: int, tmax: int, params=None, *,
                  window_stride: int | None = None, num_windows: int | None = None,
                  want_scores: bool = True, stream=None):
    """Score every lag in [tmin, tmax] of every window and select each window's period.

    The call of Algorithm 1's problem statement: a batch of sample sequences
    (T_s = 1 sample) in, per-window scores S(T) and the iteration period out.

    ``traces`` is a float32 GPU tensor shaped [B, M] (one channel), [B, C, M]
    (channel scores summed with ``params.weights``), or a 1-D long trace cut into
    ``num_windows`` windows of ``n`` samples starting every ``window_stride``
    samples.  ``n`` is the window length N; with a 2-D or 3-D tensor each window
    is the first N of its row's M samples, and None means N = M.  ``params`` is
    a DetectParams, a dict of its fields, or None for the defaults.

    Returns ``(scores, period, results)``: scores is a float32 [B, L] GPU tensor
    (L = tmax - tmin + 1, scores[b, T - tmin] = S(T)) or None, period an int32
    [B] GPU tensor (0 where no period was selected), and results a numpy
    structured array with one record per window (period, verdict, err, ...), or
    None with GPOEO_PD_SCORES_ONLY (period is then all zeros).
    """
    if params is None:
        params = DetectParams()
    elif isinstance(params, dict):
        params = DetectParams(**params)
    if traces.dim() == 1:
        if n is None or window_stride is None:
            raise ValueError("a 1-D trace needs n and window_stride")
        if num_windows is None:
            num_windows = (traces.numel() - n) // window_stride + 1
        b, c, cs = num_windows, 1, n
    elif traces.dim() == 2:
        b, m = traces.shape
        c, window_stride, cs = 1, m, m
    elif traces.dim() == 3:
        b, c, m = traces.shape
        window_stride, cs = c * m, m
    else:
        raise ValueError("traces must be 1-D, 2-D or 3-D")
    if traces.dim() > 1:
        if n is None:
            n = m
        if not 0 < n <= m:
            raise ValueError(f"window length {n} does not fit rows of {m} samples")
    desc, w = make_desc(b, c, n, window_stride, cs, tmin, tmax, params.c_lag, params.err_max,
                        params.weights, params.flags)
    det = Detector(traces.contiguous(), desc, w, want_scores=want_scores)
    det.run(stream)
    period = det.results[:, 0].clone()
    (torch.cuda.current_stream() if stream is None else stream).synchronize()
    res = None if (params.flags & SCORES_ONLY) else det.results_numpy()
    return det.scores, period, res


def rolling_params(c_measure: float = C_MEASURE, step: float = STEP, c_eval: float = C_EVAL,
                   diff_threshold: float = DEFAULT_DIFF_THRESHOLD) -> RollingParams:
    return RollingParams(float(c_measure), float(step), float(c_eval), float(diff_threshold))


def rolling_workspace_bytes(desc: Desc, params: RollingParams) -> int:
    size = ctypes.c_size_t(0)
    rc = load_library().gpoeo_pd_rolling_workspace_bytes(ctypes.byref(desc),
                                                         ctypes.byref(params),
                                                         ctypes.byref(size))
    if rc != OK:
        raise GpoeoError(rc, "gpoeo_pd_rolling_workspace_bytes")
    return int(size.value)


class RollingDetector:
    """Reusable call site of gpoeo_pd_detect_rolling (buffers allocated once)."""

    def __init__(self, x: torch.Tensor, desc: Desc, params: RollingParams,
                 weights_keepalive=None):
        if not isinstance(x, torch.Tensor) or x.dtype != torch.float32 or not x.is_cuda:
            raise TypeError("x must be a float32 GPU tensor")
        if not x.is_contiguous():
            raise ValueError("x must be contiguous")
        need = ((desc.num_windows - 1) * desc.window_stride
                + (desc.num_channels - 1) * desc.channel_stride + desc.n)
        if x.numel() < need:
            raise ValueError(f"x has {x.numel()} samples, the layout addresses {need}")
        self.x, self.desc, self.params, self._w = x, desc, params, weights_keepalive
        self.results = torch.zeros((desc.num_windows, ROLLING_DTYPE.itemsize // 4),
                                   dtype=torch.int32, device=x.device)
        self.ws_bytes = rolling_workspace_bytes(desc, params)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=x.device)
        self._lib = load_library()

    def run(self, stream=None) -> None:
        rc = self._lib.gpoeo_pd_detect_rolling(
            ctypes.byref(self.desc), ctypes.byref(self.params), self.x.data_ptr(),
            self.results.data_ptr(), self.workspace.data_ptr(), self.ws_bytes,
            _stream_handle(stream))
        if rc != OK:
            raise GpoeoError(rc, "gpoeo_pd_detect_rolling")

    def results_numpy(self) -> np.ndarray:
        host = self.results.detach().to("cpu").contiguous().numpy()
        return host.view(ROLLING_DTYPE).reshape(-1)


def detect_rolling(traces: torch.Tensor, tmin: int, tmax: int, *, weights=None,
                   c_lag: float = DEFAULT_C_LAG, err_max: float = DEFAULT_ERR_MAX,
                   flags: int = 0, stream=None, **params):
    """Algorithm 3 on every row of a [B, N] or [B, C, N] float32 GPU tensor; returns
    one ROLLING_DTYPE record per row (params: c_measure, step, c_eval, diff_threshold)."""
    if traces.dim() == 2:
        b, n = traces.shape
        c, ws, cs = 1, n, n
    elif traces.dim() == 3:
        b, c, n = traces.shape
        ws, cs = c * n, n
    else:
        raise ValueError("traces must be 2-D or 3-D")
    desc, w = make_desc(b, c, n, ws, cs, tmin, tmax, c_lag, err_max, weights, flags)
    det = RollingDetector(traces.contiguous(), desc, rolling_params(**params), w)
    det.run(stream)
    (torch.cuda.current_stream() if stream is None else stream).synchronize()
    return det.results_numpy()


def similarity(x: torch.Tensor, desc: Desc, windows: torch.Tensor, lags: torch.Tensor,
               num_groups: int = DEFAULT_GROUPS, em_iters: int = DEFAULT_EM_ITERS,
               stream=None, with_flags: bool = False):
    """Algorithm 2's Err_T for (windows[k], lags[k]) (int32 GPU tensors); returns a
    float64 GPU tensor (-1: fewer than two sub-curves, NaN: out of range), and
    with ``with_flags`` also an int32 GPU tensor of per-query flags
    (UNRESOLVED: a hard label could change under rounding)."""
    if windows.dtype != torch.int32 or lags.dtype != torch.int32:
        raise TypeError("windows and lags must be int32 tensors")
    if windows.shape != lags.shape or windows.dim() != 1:
        raise ValueError("windows and lags must be 1-D and of equal length")
    windows, lags = windows.contiguous(), lags.contiguous()
    err = torch.empty(windows.shape, dtype=torch.float64, device=x.device)
    p = SimilarityParams(int(num_groups), int(em_iters))
    lib = load_library()
    if with_flags:
        flags = torch.empty(windows.shape, dtype=torch.int32, device=x.device)
        rc = lib.gpoeo_pd_similarity_flagged(ctypes.byref(desc), ctypes.byref(p), x.data_ptr(),
                                             windows.data_ptr(), lags.data_ptr(),
                                             int(windows.numel()), err.data_ptr(),
                                             flags.data_ptr(), _stream_handle(stream))
        if rc != OK:
            raise GpoeoError(rc, "gpoeo_pd_similarity_flagged")
        return err, flags
    rc = lib.gpoeo_pd_similarity(ctypes.byref(desc), ctypes.byref(p), x.data_ptr(),
                                 windows.data_ptr(), lags.data_ptr(), int(windows.numel()),
                                 err.data_ptr(), _stream_handle(stream))
    if rc != OK:
        raise GpoeoError(rc, "gpoeo_pd_similarity")
    return err


def score_centred(x: torch.Tensor, desc: Desc, windows: torch.Tensor, lags: torch.Tensor,
                  stream=None) -> torch.Tensor:
    """Mean-removed score S_c(T) for (windows[k], lags[k]) (int32 GPU tensors); returns a
    float64 GPU tensor (-1: fewer than two sub-curves, NaN: out of range)."""
    if windows.dtype != torch.int32 or lags.dtype != torch.int32:
        raise TypeError("windows and lags must be int32 tensors")
    if windows.shape != lags.shape or windows.dim() != 1:
        raise ValueError("windows and lags must be 1-D and of equal length")
    windows, lags = windows.contiguous(), lags.contiguous()
    out = torch.empty(windows.shape, dtype=torch.float64, device=x.device)
    rc = load_library().gpoeo_pd_score_centred(ctypes.byref(desc), x.data_ptr(),
                                               windows.data_ptr(), lags.data_ptr(),
                                               int(windows.numel()), out.data_ptr(),
                                               _stream_handle(stream))
    if rc != OK:
        raise GpoeoError(rc, "gpoeo_pd_score_centred")
    return out


def spectral_params(c_peak: float = DEFAULT_C_PEAK, max_candidates: int = SPECTRAL_MAX) -> SpectralParams:
    return SpectralParams(float(c_peak), int(max_candidates), 0)


def spectral_workspace_bytes(desc: Desc, params: SpectralParams) -> int:
    size = ctypes.c_size_t()
    rc = load_library().gpoeo_pd_spectral_workspace_bytes(ctypes.byref(desc), ctypes.byref(params),
                                                          ctypes.byref(size))
    if rc != OK:
        raise GpoeoError(rc, "gpoeo_pd_spectral_workspace_bytes")
    return int(size.value)


class SpectralDetector:
    """Reusable call site of gpoeo_pd_spectral_candidates (buffers allocated once)."""

    def __init__(self, x: torch.Tensor, desc: Desc, params: SpectralParams,
                 weights_keepalive=None):
        if not isinstance(x, torch.Tensor) or x.dtype != torch.float32 or not x.is_cuda:
            raise TypeError("x must be a float32 GPU tensor")
        if not x.is_contiguous():
            raise ValueError("x must be contiguous")
        need = ((desc.num_windows - 1) * desc.window_stride
                + (desc.num_channels - 1) * desc.channel_stride + desc.n)
        if x.numel() < need:
            raise ValueError(f"x has {x.numel()} samples, the layout addresses {need}")
        self.x, self.desc, self.params, self._w = x, desc, params, weights_keepalive
        self.results = torch.zeros((desc.num_windows, SPECTRAL_DTYPE.itemsize // 4),
                                   dtype=torch.int32, device=x.device)
        self.ws_bytes = spectral_workspace_bytes(desc, params)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=x.device)
        self._lib = load_library()

    def run(self, stream=None) -> None:
        rc = self._lib.gpoeo_pd_spectral_candidates(
            ctypes.byref(self.desc), ctypes.byref(self.params), self.x.data_ptr(),
            self.results.data_ptr(), self.workspace.data_ptr(), self.ws_bytes,
            _stream_handle(stream))
        if rc != OK:
            raise GpoeoError(rc, "gpoeo_pd_spectral_candidates")

    def results_numpy(self) -> np.ndarray:
        host = self.results.detach().to("cpu").contiguous().numpy()
        return host.view(SPECTRAL_DTYPE).reshape(-1)
