"""Batched iteration-period detection on MI355X (gfx950).

The data-parallel hot path of GPOEO's period detection (Wang et al., arXiv
2201.01684, Sec. 4.1.2): every candidate period T in [Tmin, Tmax] of every
window of a batch of sampled feature traces is scored, and each window's
period is selected with Algorithm 1's peak / candidate / local-search rule.
The work runs in hand-written HIP kernels (csrc/) behind the C ABI declared in
include/gpoeo_pd.h; this package is the Python binding of that ABI.
"""
from ._binding import (  # noqa: F401
    APERIODIC,
    CONSTANT,
    DEFAULT_C_LAG,
    DEFAULT_ERR_MAX,
    EXPORTS,
    FFT_SCORES,
    MFMA_SCORES,
    LIB_PATH,
    MAX_CHANNELS,
    MAX_QUERIES,
    MAX_WINDOWS,
    NO_RESCUE,
    PERIODIC,
    RESULT_DTYPE,
    SCORES_ONLY,
    TIER2,
    UNFUSED,
    UNRESOLVED,
    ROLLING_DTYPE,
    Desc,
    DetectParams,
    Detector,
    RollingDetector,
    GpoeoError,
    describe_plan,
    detect_period,
    detect_rolling,
    rolling_params,
    similarity,
    score_centred,
    spectral_params,
    spectral_workspace_bytes,
    SpectralDetector,
    SPECTRAL_DTYPE,
    rolling_workspace_bytes,
    load_library,
    make_desc,
    results_to_numpy,
    strerror,
    workspace_bytes,
)
