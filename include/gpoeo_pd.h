/*
 * gpoeo_pd.h - batched iteration-period detection on MI355X (gfx950).
 *
 * C ABI of the HIP library libgpoeo_pd.so.  One call scores every candidate
 * period T in [tmin, tmax] of every window of a batch of sampled feature
 * traces and selects each window's iteration period, following Sec. 4.1.2 of
 * Wang et al., "Dynamic GPU Energy Optimization for Machine Learning Training
 * Workloads" (arXiv 2201.01684):
 *
 *   score   (Algorithm 2, read as the Euclidean distance between
 *           corresponding points of adjacent sub-curves, over all N-T pairs)
 *             D_c(T) = sum_{i=0}^{N-T-1} (x_c[i] - x_c[i+T])^2
 *             S(T)   = sum_c w_c * D_c(T) / (N - T)
 *           channels are combined as a weighted sum, the composite detection
 *           feature of Sec. 4.2.
 *
 *   select  (Algorithm 1: peaks, relative-height candidate filter, choice of
 *           the fundamental, local search over the neighbouring Fourier-bin
 *           periods at a one-sample step)
 *             R      = 2 * sum_c w_c * Var_c   (population variance, fp64)
 *             peaks  = { Tmin < T < Tmax : S(T) < S(T-1), S(T) <= S(T+1) }
 *             S_pk   = min S over peaks; thr = R - c_lag * (R - S_pk)
 *             T_c    = smallest peak with S(T) < thr
 *             T_low  = max(Tmin, ceil (T_c (N-1) / (N-1+T_c)))
 *             T_up   = min(Tmax, floor(T_c (N-1) / (N-1-T_c)))
 *             period = smallest T in [T_low, T_up] attaining min S
 *             err    = S(period) / R
 *
 * Precision.  D_c(T) is accumulated in fp32 over runs of at most 256 samples
 * and the runs are combined in fp64, so every score is within 2e-5 relative of
 * the exact value (scores are sums of non-negative terms; an exact zero stays
 * exactly zero).  The selection compares these bounded values; any comparison
 * the bound cannot decide is re-decided on scores (and R) recomputed on the
 * GPU as plain sequential fp64 sums over ascending i, with no fused
 * multiply-add, i.e. on the same values a straightforward fp64 evaluation of
 * the definitions gives.
 *
 * FFT scores (GPOEO_PD_FFT_SCORES).  The spectrum that Sec. 4.1.1 starts
 * from, used in the lag domain: each channel is centred by its fp64 mean,
 * zero-padded to L = 2^k >= N + Tmax points and transformed in fp64, and
 *   D_c(T) = sum_{i<N-T} y_i^2 + sum_{i>=T} y_i^2 - 2 r(T),
 * with the autocorrelation r the inverse transform of the power spectrum
 * (O(L log L) per channel instead of O(N (Tmax - Tmin))).  When a transform
 * of only L = 2^k >= N points costs less, it is used instead: the lags T > L - N
 * of its circular autocorrelation then carry the products of the first and
 * the last M = Tmax - (L - N) samples, which a second transform of at least
 * 2M points computes and which are subtracted (gpoeo_pd_describe_plan reports
 * both lengths).  A rigorous absolute error bound of each D_c(T), from the
 * channel norms, decides which scores are within 1e-6 relative of the exact
 * value; every other lag (exact zeros included) is recomputed as an fp64 sum
 * before the selection, which then proceeds as above.  Selections equal those
 * of the direct scores.  Requires a transform of at most 2^22 points: N + Tmax
 * <= 2^22, or N <= 2^22 with a head-tail transform of at most min(2^20, L / 2)
 * points.  Sliding-window block sharing does not apply.
 *
 * Matrix-core scores (GPOEO_PD_MFMA_SCORES).  The same decomposition of D_c(T)
 * with r(T) evaluated directly, as an integer cross-correlation on the int8
 * matrix instructions: each (window, channel) sequence is centred by its mean
 * rounded to fp32, scaled by a power of two 2^s into integers
 * X_i = rint((x_i - c) 2^s) with |X_i| <= 2^30, and split into four signed
 * base-256 digits; the 13 digit-pair correlations of weight 256^2 and above
 * accumulate exactly in int32 and are combined in fp64 (the three of least
 * weight, at most 2^23 per sample pair against products up to 2^60, are left
 * out and bounded).  When every x_i - c is a multiple of 2^-s (the samples of
 * the sequence span at most about 2^7 in magnitude, as sampled power does) the
 * X_i are the samples exactly and the only errors are the fp64 combination and
 * the pairs left out; otherwise the rounding of X_i adds a bounded error.  Each lag
 * whose bound exceeds 1.25e-5 of its score (exact zeros included) is
 * recomputed as an fp64 sum before the selection, which then uses the same
 * tier-0 width as the direct scores.  Selections equal those of the direct
 * scores.  A batch with too few lag tiles to fill the chip splits each tile's
 * samples into chunks whose partial sums are added in a fixed order, so the
 * results never depend on scheduling.  Not with GPOEO_PD_FFT_SCORES.  Rolling detection takes it too (its
 * suffix windows come from a window table that every kernel reads).
 *
 * Threading and ownership.  All buffers except `desc` and `desc->channel_weights`
 * are DEVICE memory owned by the caller.  The library never allocates or frees
 * memory and keeps no mutable global state: calls on different streams with
 * different workspaces may run concurrently.  `gpoeo_pd_detect` validates its
 * arguments on the host, enqueues its kernels on `stream` and returns; outputs
 * are valid once the stream has been synchronised.
 *
 * Inputs must be finite (no NaN or Inf); otherwise the outputs are unspecified.
 */
#ifndef GPOEO_PD_H
#define GPOEO_PD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GPOEO_PD_ABI_VERSION 1

/* Status codes returned by every entry point. */
#define GPOEO_PD_OK 0
#define GPOEO_PD_EINVAL (-1)   /* invalid descriptor or pointer; nothing was launched      */
#define GPOEO_PD_ENOMEM (-2)   /* workspace smaller than gpoeo_pd_workspace_bytes()        */
#define GPOEO_PD_EHIP (-3)     /* a HIP launch failed (hipGetLastError after enqueueing)    */
#define GPOEO_PD_ETOOBIG (-4)  /* gpoeo_pd_detect_noalloc: the call needs more workspace than
                                  GPOEO_PD_NOALLOC_MAX_WORKSPACE; nothing was launched     */

/* Per-window verdicts. */
#define GPOEO_PD_PERIODIC 0    /* a period was selected and err < err_max                  */
#define GPOEO_PD_APERIODIC 1   /* no candidate period, or err >= err_max                   */
#define GPOEO_PD_CONSTANT 2    /* R == 0: every weighted channel is constant               */

/* desc->flags */
#define GPOEO_PD_SCORES_ONLY 1u  /* compute scores only; `results` is not written           */
#define GPOEO_PD_NO_RESCUE 2u    /* decide on the bounded tier-0 scores only                */
#define GPOEO_PD_FFT_SCORES 4u   /* scores from an fp64 FFT autocorrelation instead of the
                                    direct sums (see below); transform limits below        */
#define GPOEO_PD_MFMA_SCORES 8u  /* scores from an integer cross-correlation on the matrix
                                    cores instead of the direct sums (see below)           */
#define GPOEO_PD_UNFUSED 16u     /* windows of at most GPOEO_PD_FUSED_MAX_N samples and
                                    GPOEO_PD_FUSED_MAX_LAGS lags with direct scores, each
                                    scored on its own, normally run everything after the
                                    lag scores (statistics, finalisation, selection and
                                    its re-scores) as one kernel; this flag runs those
                                    stages as separate kernels, with identical results   */
#define GPOEO_PD_FUSED_MAX_N 16384
#define GPOEO_PD_FUSED_MAX_LAGS 6144

/* result->flags */
#define GPOEO_PD_UNRESOLVED 1u   /* some comparison stayed undecided after the exact
                                    re-scoring limit; the result uses bounded scores       */
#define GPOEO_PD_SHORT 2u        /* (rolling detection) a suffix window too short for
                                    three lags starting at tmin; no period                 */
#define GPOEO_PD_TIER2 4u        /* some decision of this window used scores (or R)
                                    recomputed as plain sequential fp64 sums: they were
                                    too close for the bounded fp64 re-scores           */

/* Size limits, checked (EINVAL) before any launch, that keep every grid within
 * HIP's 32-bit global size.  A descriptor whose work would still need a larger
 * grid (very many sequences or lag-score waves) is rejected the same way. */
#define GPOEO_PD_MAX_WINDOWS (1 << 21)   /* windows per call (rolling: B * suffix slots) */
#define GPOEO_PD_MAX_QUERIES (1 << 23)   /* (window, lag) queries per similarity or
                                            mean-removed score call                       */
/* Channels per window.  The composite detection feature of Sec. 4.2 combines a
 * handful of sampled metrics (power, SM and memory utilisation); the weights
 * of up to this many channels travel with every launch as a kernel argument,
 * so a descriptor with more channels is EINVAL. */
#define GPOEO_PD_MAX_CHANNELS 256

typedef struct {
    int64_t num_windows;     /* 1 <= B <= GPOEO_PD_MAX_WINDOWS: traces, or sliding windows  */
    int32_t num_channels;    /* 1 <= C <= GPOEO_PD_MAX_CHANNELS: per-lag channel scores are
                                summed with weights (the composite feature of Sec. 4.2)     */
    int32_t reserved0;       /* must be 0                                                   */
    int64_t n;               /* N >= 8 samples per window                                   */
    int64_t window_stride;   /* samples between window starts (N*C when packed)            */
    int64_t channel_stride;  /* samples between channels of one window (>= N if C > 1)     */
    int32_t tmin, tmax;      /* inclusive lag range: 1 <= tmin, tmin + 2 <= tmax <= N / 2   */
    double c_lag;            /* relative-height factor of the candidate filter, in (0, 1);
                                the lag-domain counterpart of Algorithm 1's c_peak.
                                Recommended 0.9                                             */
    double err_max;          /* APERIODIC if S(period)/R >= err_max (1.0: never for a
                                selected period)                                            */
    const float* channel_weights; /* HOST array of C weights > 0, or NULL for all 1          */
    uint32_t flags;          /* GPOEO_PD_SCORES_ONLY | _NO_RESCUE | _FFT_SCORES | _MFMA_SCORES
                                | _UNFUSED                                                  */
    uint32_t reserved1;      /* must be 0                                                   */
} gpoeo_pd_desc;

typedef struct {
    int32_t period;          /* selected period in samples (times T_s for seconds); 0 if none */
    int32_t verdict;         /* GPOEO_PD_PERIODIC / _APERIODIC / _CONSTANT                   */
    float err;               /* S(period) / R, Algorithm 1's "error of period"; 0 if none    */
    int32_t n_candidates;    /* peaks passing the relative-height filter                     */
    int32_t t_cand;          /* T_c, the smallest candidate; 0 if none                       */
    int32_t t_low, t_up;     /* local-search window; 0 if none                               */
    int32_t n_rescored;      /* scores recomputed as sequential fp64 sums for this window    */
    uint32_t flags;          /* GPOEO_PD_UNRESOLVED                                          */
} gpoeo_pd_result;

/* How gpoeo_pd_detect will run a descriptor (for measurement tools). */
typedef struct {
    int32_t mode;             /* 0: every window scored on its own; 1: overlapping windows
                                 at a stride dividing N share per-block partials; 2: FFT
                                 scores (score_waves and pairs_scored are then 0); 3:
                                 matrix-core scores (score_waves: lag tiles of 1024 times
                                 the sample chunks of each tile)                          */
    int32_t lags_per_lane;    /* consecutive lags per lane of the score kernel (8 or 16)  */
    int64_t score_waves;      /* wavefronts the score stage launches                      */
    double pairs_defined;     /* sum over windows, channels and T in [tmin, tmax] of N - T:
                                 the (x[i], x[i+T]) pairs the definition of S(T) sums     */
    double pairs_scored;      /* pairs with T in [tmin, tmax] the score stage evaluates   */
    size_t workspace_bytes;   /* same as gpoeo_pd_workspace_bytes                          */
    int64_t fft_len;          /* FFT scores: points per transform (0 otherwise)           */
    int64_t fft_wrap_len;     /* FFT scores whose transform holds only N points: points
                                 of the head-tail transform of the wrap term; else 0      */
    int64_t fft_wrap_lags;    /* lags T > fft_len - N that carry the wrap term; else 0   */
} gpoeo_pd_plan_info;

/* Describes the launch plan of `desc`.  Host-only; GPOEO_PD_OK or GPOEO_PD_EINVAL. */
int gpoeo_pd_describe_plan(const gpoeo_pd_desc* desc, gpoeo_pd_plan_info* info);

/* ABI version the library was built with (GPOEO_PD_ABI_VERSION). */
int gpoeo_pd_abi_version(void);

/* Static message for a status code; never NULL. */
const char* gpoeo_pd_strerror(int status);

/* Validates `desc` and writes the device workspace size gpoeo_pd_detect needs.
 * Returns GPOEO_PD_OK or GPOEO_PD_EINVAL.  Host-only: launches nothing. */
int gpoeo_pd_workspace_bytes(const gpoeo_pd_desc* desc, size_t* bytes);

/* Scores and selects every window of the batch.
 *   x          device, fp32; window b, channel c, sample i at
 *              x[b*window_stride + c*channel_stride + i]; windows may overlap.
 *   scores     device, fp32 [B][tmax-tmin+1] row-major, scores[b][T-tmin] = S(T);
 *              may be NULL.
 *   results    device, one gpoeo_pd_result per window; may be NULL only with
 *              GPOEO_PD_SCORES_ONLY.
 *   workspace  device, at least gpoeo_pd_workspace_bytes() bytes, 256-byte
 *              aligned; its contents on entry are ignored.
 *   stream     HIP stream all kernels are enqueued on (0 = the null stream).
 * Returns GPOEO_PD_OK, GPOEO_PD_EINVAL or GPOEO_PD_ENOMEM before launching
 * anything, or GPOEO_PD_EHIP if a launch failed. */
int gpoeo_pd_detect(const gpoeo_pd_desc* desc, const float* x, float* scores,
                    gpoeo_pd_result* results, void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/* gpoeo_pd_detect for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops, harnesses that forbid hipMalloc): the same
 * kernels, with the workspace taken from a static device array of
 * GPOEO_PD_NOALLOC_MAX_WORKSPACE bytes that the library holds on every GPU it
 * runs on until the process ends.  The call itself allocates nothing; its
 * first call on a device looks up that device's array once.
 *   x, scores, results, stream   as in gpoeo_pd_detect; `stream` must belong
 *              to the current device.
 * Every call on one GPU shares that GPU's array: calls that overlap there (on
 * concurrent streams, or from several threads) race and must be serialised by
 * the caller.  The array's contents on entry are ignored.
 * Returns GPOEO_PD_EINVAL as gpoeo_pd_detect does, GPOEO_PD_ETOOBIG when
 * gpoeo_pd_workspace_bytes(desc) exceeds GPOEO_PD_NOALLOC_MAX_WORKSPACE (both
 * before launching anything), GPOEO_PD_EHIP if the array cannot be located or
 * a launch failed. */
#define GPOEO_PD_NOALLOC_MAX_WORKSPACE ((size_t)64 << 20)

int gpoeo_pd_detect_noalloc(const gpoeo_pd_desc* desc, const float* x, float* scores,
                            gpoeo_pd_result* results, hipStream_t stream);

/* gpoeo_pd_detect, additionally recording stage_events[k] on `stream` right
 * before stage k is enqueued (0 window statistics, 1 lag scores, 2 score
 * finalisation, 3 selection) and stage_events[4] after the last one, so that
 * hipEventElapsedTime between consecutive events gives each stage's device
 * time.  For measurement tools; the events are created (hipEventCreate) and
 * owned by the caller.  A stage that the flags skip records its two events
 * back to back.  Same return values as gpoeo_pd_detect; EINVAL if
 * stage_events is NULL. */
int gpoeo_pd_detect_staged(const gpoeo_pd_desc* desc, const float* x, float* scores,
                           gpoeo_pd_result* results, void* workspace, size_t workspace_bytes,
                           hipStream_t stream, hipEvent_t stage_events[5]);

/* ---------------------------------------------------------------------------
 * Rolling detection (Algorithm 3, Sec. 4.1.3).  For every window of the batch
 * (read as the samples gathered so far): T_init = the period of the whole
 * window (the rule above); then, with D = N - 1 and T_s = 1 sample,
 *   D < c_measure * T_init: too short, period T_init, smpdur_next = c_measure T_init - D;
 *   otherwise suffix windows x[floor(t) .. N-1] for t = max(0, D - (2 + c_eval step) T_init),
 *   t += step T_init while (D - t) / T_init >= c_measure, each scored and
 *   selected with lags [tmin, min(tmax, N_j / 2)]; among the suffixes with a
 *   PERIODIC verdict the smallest err gives the period (first on ties),
 *   diff = |max T - min T| / mean T, and smpdur_next = -1 (stable) when
 *   diff < diff_threshold, else ceil(D / max T) max T - D.
 * The whole pipeline runs on `stream` (two detection passes, a schedule kernel
 * and a combining kernel); the same precision rules as gpoeo_pd_detect apply.
 * ------------------------------------------------------------------------- */
#define GPOEO_PD_ROLLING_MAX 16   /* suffix windows per window, at most */

typedef struct {
    double c_measure;        /* periods a (suffix) window must span; the paper uses 2       */
    double step;             /* advance of the suffix start, in periods; the paper uses 0.5 */
    double c_eval;           /* the first suffix spans 2 + c_eval * step periods; paper 6.5 */
    double diff_threshold;   /* stable iff diff < this; not given by the paper (0.05)        */
} gpoeo_pd_rolling_params;

typedef struct {
    int32_t period;          /* T_iter in samples; 0 if none                                  */
    int32_t verdict;         /* of the whole window's first pass                              */
    int32_t stable;          /* 1 when smpdur_next == -1                                      */
    int32_t n_windows;       /* suffix windows evaluated (0: too short or not periodic)       */
    int32_t t_init;          /* period of the whole window                                    */
    int32_t best;            /* index of the selected suffix window, -1 if none               */
    double smpdur_next;      /* samples to keep sampling before the next call; -1 if stable   */
    float diff;              /* relative period spread over the periodic suffix windows       */
    float err;               /* err of the selected period                                    */
    uint32_t flags;          /* GPOEO_PD_UNRESOLVED if any selection of this window was       */
    int32_t reserved;
    int32_t periods[GPOEO_PD_ROLLING_MAX];   /* T_j per suffix window (0: none)               */
    int64_t starts[GPOEO_PD_ROLLING_MAX];    /* first sample of each suffix window            */
} gpoeo_pd_rolling_result;

/* Validates desc (flags may hold GPOEO_PD_NO_RESCUE and one of GPOEO_PD_FFT_SCORES and
 * GPOEO_PD_MFMA_SCORES) and params and writes the device workspace size of
 * gpoeo_pd_detect_rolling.  EINVAL if the schedule
 * could exceed GPOEO_PD_ROLLING_MAX suffix windows, or if B times the suffix
 * slots per window (floor((2 + c_eval step - c_measure) / step) + 2) exceeds
 * GPOEO_PD_MAX_WINDOWS. */
int gpoeo_pd_rolling_workspace_bytes(const gpoeo_pd_desc* desc,
                                     const gpoeo_pd_rolling_params* params, size_t* bytes);

/* Rolling detection of every window; results: device, one record per window. */
int gpoeo_pd_detect_rolling(const gpoeo_pd_desc* desc, const gpoeo_pd_rolling_params* params,
                            const float* x, gpoeo_pd_rolling_result* results, void* workspace,
                            size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Feature sequence similarity (Algorithm 2, Sec. 4.1.2) of finalist periods.
 * For query k, window windows[k] and candidate period T = lags[k]: whole
 * sub-curves of T samples; each sub-curve's samples grouped by a 1-D Gaussian
 * mixture (num_groups components, em_iters EM iterations in fp64, hard
 * assignment to the most responsible component); per group, its mean minus the
 * sub-curve mean, compared with the same sample indices of the next sub-curve
 * by SMAPE(a, b) = |a - b| / ((|a| + |b|) / 2) (0/0 = 0), weighted by group
 * size; err[k] = mean over adjacent pairs, weighted mean over channels.
 * err[k] = -1 when floor(N / T) < 2, NaN for a window or lag out of range.
 * windows, lags: device int32 [count], 0 <= count <= GPOEO_PD_MAX_QUERIES
 * (else EINVAL); err: device double [count].  The window layout (and the
 * channel weights) come from desc, whose lag range is not used.  No workspace.
 * ------------------------------------------------------------------------- */
typedef struct {
    int32_t num_groups;      /* NumG, 1..8 (the paper leaves it open; 3 recommended)    */
    int32_t em_iters;        /* EM iterations, >= 0 (20 recommended)                    */
} gpoeo_pd_similarity_params;

int gpoeo_pd_similarity(const gpoeo_pd_desc* desc, const gpoeo_pd_similarity_params* params,
                        const float* x, const int32_t* windows, const int32_t* lags,
                        int64_t count, double* err, hipStream_t stream);

/* gpoeo_pd_similarity, also reporting queries whose result rounding could
 * change (Algorithm 2's grouping step).  Err depends on the fitted mixture
 * only through the hard labels, and a plain fp64 fit in another evaluation
 * order moves the fitted parameters by at most a few 1e-13 relative.  For
 * every sample, the margin between its two largest log-densities is compared
 * with the change that relative errors of 1e-11 in each parameter (mu, var,
 * pi), plus the rounding of the densities, can cause in either; if it is not
 * larger, the label could differ from an exact evaluation's and flags[k] is
 * GPOEO_PD_UNRESOLVED (else 0).  err[k] is still written.
 * flags: device uint32 [count], required when count > 0 (else EINVAL). */
int gpoeo_pd_similarity_flagged(const gpoeo_pd_desc* desc,
                                const gpoeo_pd_similarity_params* params, const float* x,
                                const int32_t* windows, const int32_t* lags, int64_t count,
                                double* err, uint32_t* flags, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Mean-removed score of finalist periods (Algorithm 2's relative values, Sec.
 * 4.1.2, with one group per sample).  For query k, window windows[k] and
 * candidate period T = lags[k]: floor(N / T) whole sub-curves of T samples;
 * every adjacent pair compared point by point after removing each
 * sub-curve's own mean,
 *   S_c(T) = sum_c w_c * sum_{i,j} ((x[iT+j] - mu_i) - (x[(i+1)T+j] - mu_{i+1}))^2
 *            / ((floor(N/T) - 1) T),
 * i.e. the whole-sub-curve pair sum minus T sum_i (mu_i - mu_{i+1})^2: adding
 * a linear drift to a channel changes no S_c.  Short lags lose most of their
 * differences to the means, so this re-scores candidates rather than scanning
 * every T.  score[k] = -1 when floor(N / T) < 2, NaN for a window or lag out of
 * range.  windows, lags: device int32 [count], 0 <= count <=
 * GPOEO_PD_MAX_QUERIES (else EINVAL); score: device double [count]; layout
 * and weights from desc (its lag range is not used).  fp64 throughout.  No
 * workspace.
 * ------------------------------------------------------------------------- */
int gpoeo_pd_score_centred(const gpoeo_pd_desc* desc, const float* x, const int32_t* windows,
                           const int32_t* lags, int64_t count, double* score,
                           hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Spectral candidates: Algorithm 1's FFT front end (lines 1-5; Sec. 4.1.1-4.1.2,
 * with T_s = 1 sample).  Per window:
 *   every channel centred by its fp64 mean and zero-padded to L = 2^k >= N
 *   (at least 64) points; A(k) = sum_c w_c |X_c(k)|, k = 0..L/2, from an fp64
 *   FFT ("Ampl");
 *   peaks = bins 2 <= k <= L/2 - 1 with A(k) > A(k-1) and A(k) >= A(k+1);
 *   candidates = peaks with A(k) > c_peak * (largest peak) whose period
 *   round(L / k) (halves up) lies in [tmin, tmax], strongest first (ties: the
 *   smaller k), at most max_candidates; two bins may give the same period.
 * A window whose list could change within the rounding error bound of the
 * amplitudes (a peak test, the threshold or the order of the listed
 * candidates within that margin), or with more than 1024 qualifying peaks, is
 * flagged GPOEO_PD_UNRESOLVED; its list is still written.  The candidates are
 * what Algorithm 1 evaluates with Algorithm 2 (gpoeo_pd_similarity,
 * gpoeo_pd_score_centred).  desc gives the window layout, channel weights and
 * lag range (its flags are not used); L <= 2^22.  results: device, one record
 * per window; workspace: caller-owned, gpoeo_pd_spectral_workspace_bytes.
 * ------------------------------------------------------------------------- */
#define GPOEO_PD_SPECTRAL_MAX 16

typedef struct {
    double c_peak;           /* relative peak height in (0, 1); the paper uses 0.6-0.7   */
    int32_t max_candidates;  /* 1..GPOEO_PD_SPECTRAL_MAX                                 */
    int32_t reserved;        /* must be 0                                                */
} gpoeo_pd_spectral_params;

typedef struct {
    int32_t count;           /* candidates written                                       */
    uint32_t flags;          /* GPOEO_PD_UNRESOLVED                                      */
    int32_t n_peaks;         /* peaks of A                                               */
    int32_t reserved;
    double max_peak;         /* the largest peak of A; 0 if none                         */
    int32_t periods[GPOEO_PD_SPECTRAL_MAX];   /* round(L / bin)                          */
    int32_t bins[GPOEO_PD_SPECTRAL_MAX];      /* k                                       */
    double amplitudes[GPOEO_PD_SPECTRAL_MAX]; /* A(k)                                    */
} gpoeo_pd_spectral_result;

int gpoeo_pd_spectral_workspace_bytes(const gpoeo_pd_desc* desc,
                                      const gpoeo_pd_spectral_params* params, size_t* bytes);

int gpoeo_pd_spectral_candidates(const gpoeo_pd_desc* desc, const gpoeo_pd_spectral_params* params,
                                 const float* x, gpoeo_pd_spectral_result* results,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* GPOEO_PD_H */
