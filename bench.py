#!/usr/bin/env python3
"""Throughput of batched iteration-period detection on one MI355X.

One step = one gpoeo_pd_detect call over the whole batch: window statistics,
lag scores for every T in [Tmin, Tmax] of every window, finalisation and the
per-window selection.  Inputs are generated (seeded) on the host, copied to HBM
once, and resident there before the timed region starts.

Prints one JSON line with the throughput (lag*samples/s), traces/s, the
roofline of the lag-score kernel (timed with HIP events recorded around it on
the stream it runs on) and the CPU oracle timed on a bounded sample of the same
workload.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_VECTOR_PEAK_TFLOPS = 157.3   # MI355X published FP32 vector peak
FP64_VECTOR_PEAK_TFLOPS = 78.6    # MI355X published FP64 vector peak
HBM_PEAK_GBS = 8000.0              # MI355X published HBM3E bandwidth
INT8_MFMA_PEAK_TOPS = 5000.0       # MI355X published dense int8 matrix peak
# Matrix-core scores: 13 digit-pair products (four int8 digits per sample on
# each side; the three pairs of least weight are left out) per (x[i], x[i+T])
# pair, one multiply and one add each.
MFMA_OPS_PER_PAIR = 26
# Algorithmic fp64 FLOP of the EM per (sample, component, iteration): the
# log-density (sub, mul, mul, sub), the exponential (counted as one), the
# normalisation (add, mul) and the three moments (add; mul, add; mul, mul, add).
EM_FLOP = 13
# Mean-removed score per pair of corresponding points: the two mean sums (add,
# add), the centred difference (sub, sub, sub) and its square accumulated (mul, add).
CENTRED_FLOP = 7
FLOP_PER_PAIR = 3                 # one subtraction, one multiply, one add per (x[i], x[i+T])
# Pairs per second the direct kernel can issue at most: one v_sub_f32 and one
# v_fmac_f32 per pair, two VALU instructions per clock per CU with dual issue,
# 256 CUs at 2.4 GHz.
VALU_PAIR_CEILING = 256 * 2.4e9 * 64
METRIC = "lag·samples/sec and traces/sec for batched period detection; % FP32 peak"
CSRC = os.path.join(ROOT, "paper_2201_01684_amd", "csrc")
# committed rocprofv3 HBM counter summaries per score mode (w3), and the source
# whose hash they were taken with
COUNTERS = {"detect": (os.path.join(ROOT, "profiles", "lag_score_w3_counters.txt"),
                       os.path.join(CSRC, "lag_score.hip")),
            "fft": (os.path.join(ROOT, "profiles", "fft_stage_w3_counters.txt"),
                    os.path.join(CSRC, "fft_score.hip")),
            "mfma": (os.path.join(ROOT, "profiles", "mfma_xcorr_w3_counters.txt"),
                     os.path.join(CSRC, "mfma_score.hip"))}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="w3", help="w1..w5 (default w3, the 1024-trace batch)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time budget of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mode", choices=("detect", "fft", "mfma", "rolling", "similarity",
                                       "centred", "spectral"),
                    default="detect",
                    help="detect: gpoeo_pd_detect (the default measurement); fft: the same "
                         "call with GPOEO_PD_FFT_SCORES (fp64 FFT autocorrelation scores); "
                         "mfma: the same call with GPOEO_PD_MFMA_SCORES (integer "
                         "cross-correlation on the int8 matrix cores); "
                         "rolling: "
                         "Algorithm 3's rolling detection, gpoeo_pd_detect_rolling; "
                         "similarity: Algorithm 2's grouped similarity of 5 finalist periods "
                         "per window (the selected one, its neighbours, its double and half); "
                         "centred: the mean-removed score of the same 5 finalists; "
                         "spectral: Algorithm 1's FFT front end (candidate periods)")
    ap.add_argument("--graph", action="store_true",
                    help="detect/fft/mfma mode: also time replays of one call captured in a HIP "
                         "graph")
    ap.add_argument("--no-fft-compare", action="store_true",
                    help="detect mode: skip the untimed FFT- and matrix-core-scores runs of the "
                         "same batch")
    ap.add_argument("--no-configs", action="store_true",
                    help="detect mode: skip the per-configuration timings (c1-c5) after the "
                         "timed region")
    ap.add_argument("--fft-scores", action="store_true",
                    help="rolling mode: score with GPOEO_PD_FFT_SCORES")
    ap.add_argument("--mfma-scores", action="store_true",
                    help="rolling mode: score with GPOEO_PD_MFMA_SCORES")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a device-to-device copy of this many MiB (the reference "
                         "kernel that scales rocprofv3 FETCH_SIZE / WRITE_SIZE) and exit")
    return ap.parse_args()


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch loaded (one runtime per process)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventCreate.restype = ctypes.c_int
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventElapsedTime.restype = ctypes.c_int
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.restype = ctypes.c_int

    def create(self, count):
        arr = (ctypes.c_void_p * count)()
        for k in range(count):
            h = ctypes.c_void_p()
            rc = self.hip.hipEventCreate(ctypes.byref(h))
            if rc != 0:
                raise RuntimeError(f"hipEventCreate failed ({rc})")
            arr[k] = h.value
        return arr

    def elapsed_ms(self, a, b) -> float:
        out = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(out), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(out.value)

    def destroy(self, arr):
        for h in arr:
            self.hip.hipEventDestroy(h)

    def attribute(self, attr: int, device: int = 0) -> int:
        fn = self.hip.hipDeviceGetAttribute
        fn.argtypes = [ctypes.POINTER(ctypes.c_int), ctypes.c_int, ctypes.c_int]
        fn.restype = ctypes.c_int
        out = ctypes.c_int()
        if fn(ctypes.byref(out), attr, device) != 0:
            raise RuntimeError("hipDeviceGetAttribute failed")
        return int(out.value)


HIP_ATTR_CLOCK_RATE_KHZ = 5      # hipDeviceAttributeClockRate (ROCm 7 hip_runtime_api.h)


def device_info(ev: "HipEvents") -> dict:
    """The GPU as the runtime reports it, and the FP32 peak and the lag-score
    pair ceiling (one v_sub + one v_fmac per pair, two VALU instructions per
    clock per CU with dual issue) recomputed from its CU count and peak clock."""
    import torch
    p = torch.cuda.get_device_properties(0)
    mhz = ev.attribute(HIP_ATTR_CLOCK_RATE_KHZ) / 1e3
    cus = p.multi_processor_count
    return {"name": p.name, "arch": p.gcnArchName, "compute_units": cus,
            "peak_clock_mhz": mhz, "fp32_peak_tflops_at_clock": cus * mhz * 1e6 * 256 / 1e12,
            "pair_ceiling_per_s": cus * mhz * 1e6 * 64}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def counters_traffic(workload: str, mode: str = "detect"):
    """HBM bytes per launch of the mode's score stage from the committed
    rocprofv3 counter summary (FETCH_SIZE and WRITE_SIZE scaled by a copy kernel
    of known size), or None if the summary is missing, covers another workload,
    or the kernel source changed since the counters were taken."""
    if workload != "w3" or mode not in COUNTERS:
        return None
    counters_file, source = COUNTERS[mode]
    try:
        fields = {}
        with open(counters_file) as f:
            for line in f:
                if line.startswith("#") or ":" not in line:
                    continue
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        src = hashlib.sha256(open(source, "rb").read()).hexdigest()
        if fields.get("source_sha256") != src:
            return None
        return float(fields["hbm_bytes_per_launch"])
    except (OSError, ValueError, KeyError):
        return None


def fft_stage_bytes(wl, plan) -> float:
    """HBM bytes the FFT score stage moves per call, for the transform lengths of
    the plan (`describe_plan`): the samples read once by the column transforms
    (the centring sums come with the window statistics), the first and last
    Tmax samples of each sequence read and their head and tail sums written
    and read back, each pair's complex fp64 transform written by the column
    kernel, read and written by the row kernel and read by the inverse column
    kernel (none of that up to 2048 points, where a pair stays in LDS), and the
    per-channel D(T) written.  With the wrap correction: the first and last M
    samples read again, the head and tail transforms written, read, the cross
    spectrum written and read back (six sweeps of the head-tail length), and
    the M wrap terms per sequence written and read."""
    s = wl.num_windows * wl.num_channels
    pairs = (s + 1) // 2
    length = plan["fft_len"]
    lags = wl.tmax - wl.tmin + 1
    sweeps = 0 if length <= 2048 else 4
    edges = 2 * 4 * s * wl.tmax + 2 * 8 * s * (wl.tmax + 1) + 2 * 8 * s * lags
    total = 4 * s * wl.n + edges + sweeps * 16 * pairs * length + 8 * s * lags
    m = plan["fft_wrap_lags"]
    if plan["fft_wrap_len"]:
        total += 2 * 4 * s * m + 6 * 16 * pairs * plan["fft_wrap_len"] + 2 * 8 * s * m
    return float(total)


def pow2_at_least(v: int, lo: int = 64) -> int:
    length = lo
    while length < v:
        length *= 2
    return length


def transform_bytes(pairs_lengths, seq_samples: int, seqs: int, lag_counts) -> float:
    """HBM bytes of the FFT scores of a batch: every pair of sequences (length L
    of its transform) writes, reads, writes and reads its complex fp64 transform
    (none of that up to 2048 points, where a pair stays in LDS); the samples
    are read once, the head and tail sums written and read back, and D(T)
    written per lag."""
    sweeps = sum(16 * 4 * length for length in pairs_lengths if length > 2048)
    edges = sum(2 * 4 * t + 2 * 8 * (t + 1) + 2 * 8 * t for t in lag_counts)
    return float(4 * seq_samples + edges + sweeps + 8 * sum(lag_counts))


def call_roofline(kernel, bound, work, ms, extra=None):
    """Roofline object of a mode timed as a whole call: `work` is the algorithmic
    FLOP (bound "alu": fp32 or fp64 given by the kernel), int8 matrix operations
    (bound "mfma") or bytes (bound "hbm") of one call, `ms` the mean call time from HIP events on the call's stream."""
    if bound == "hbm":
        achieved, peak, unit = work / (ms / 1e3) / 1e9, HBM_PEAK_GBS, "GB/s"
    elif bound == "mfma":   # int8 matrix operations
        achieved, peak, unit = work / (ms / 1e3) / 1e12, INT8_MFMA_PEAK_TOPS, "TOP/s"
    else:
        peak = FP64_VECTOR_PEAK_TFLOPS if bound == "alu_f64" else FP32_VECTOR_PEAK_TFLOPS
        achieved, unit = work / (ms / 1e3) / 1e12, "TFLOP/s"
    line = {"kernel": kernel, "bound": bound if bound in ("hbm", "mfma") else "alu",
            "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
            "traffic": None, "timed": "whole call (HIP events on its stream)"}
    if extra:
        line.update(extra)
    return line


# The five trace configurations, timed after the headline's timed region:
# repeats of the per-call timing (median and minimum), and the windows the
# oracle checks.  c3 is the headline workload itself.
CONFIGS = (("c1", "w1", 1000, (0,)), ("c2", "w2", 100, (0, 63)), ("c3", "w3", 5, (0,)),
           ("c4", "w4", 20, (0, 2040, 2044, 2048, 4088)), ("c5", "w5", 5, (0,)))


def bench_config(pkg, ev, wl, repeats, check_windows, x=None, warmup=2):
    """One configuration: `repeats` back-to-back gpoeo_pd_detect calls timed by
    wall clock around the loop (throughput), then up to 100 calls with per-stage
    HIP events (median and minimum per call, the lag-score stage for the
    roofline), planted-period hits and the oracle on a few windows."""
    import numpy as np
    import torch
    import oracle
    dev = torch.device("cuda:0")
    if x is None:
        x = torch.from_numpy(wl.x).to(dev)
    desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                               wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights)
    det = pkg.Detector(x, desc, keep, want_scores=True)
    plan = pkg.describe_plan(desc)
    pairs, scored = float(wl.pairs()), plan["pairs_scored"]
    for _ in range(warmup):
        det.run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(repeats):
        det.run()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / repeats
    n_ev = min(repeats, 100)
    sets = [ev.create(5) for _ in range(n_ev)]
    torch.cuda.synchronize()
    for k in range(n_ev):
        det.run_staged(sets[k])
    torch.cuda.synchronize()
    call = np.array([ev.elapsed_ms(s_[0], s_[4]) for s_ in sets])
    score = np.array([ev.elapsed_ms(s_[1], s_[2]) for s_ in sets])
    select = np.array([ev.elapsed_ms(s_[3], s_[4]) for s_ in sets])
    for s_ in sets:
        ev.destroy(s_)
    res = det.results_numpy()
    med = float(np.median(call))
    out = {"workload": wl.name, "description": wl.meta["description"], "sha256": wl.sha256,
           "windows": wl.num_windows, "channels": wl.num_channels, "n": wl.n,
           "tmin": wl.tmin, "tmax": wl.tmax, "pairs": pairs, "pairs_scored": scored,
           "repeats": repeats, "ms_per_call_back_to_back": wall,
           "call_ms": {"median": med, "min": float(call.min()), "calls": n_ev},
           # throughput over the back-to-back calls (the per-stage events add
           # their own overhead, which a 4096-sample call feels)
           "lag_samples_per_sec": pairs / (wall / 1e3),
           "traces_per_sec": wl.num_windows / (wall / 1e3),
           "lag_score_ms": float(np.median(score)),
           "select_ms": float(np.median(select)),
           "frac_fp32_lag_score": FLOP_PER_PAIR * scored / (float(np.median(score)) / 1e3)
                                  / 1e12 / FP32_VECTOR_PEAK_TFLOPS,
           "frac_fp32_call": FLOP_PER_PAIR * scored / (med / 1e3) / 1e12
                             / FP32_VECTOR_PEAK_TFLOPS,
           "windows_rescored": int(np.count_nonzero(res["n_rescored"])),
           "windows_flagged_unresolved": int(np.count_nonzero(res["flags"] & pkg.UNRESOLVED))}
    if wl.truth is not None:
        d = wl.truth > 0
        ok = (np.abs(res["period"][d] - wl.truth[d]) <= np.ceil(0.02 * wl.truth[d])
              if wl.jitter else res["period"][d] == wl.truth[d])
        out["planted_period_hits"] = f"{int(ok.sum())}/{int(d.sum())}"
    s_host = det.scores.double().cpu().numpy()
    match, worst = 0, 0.0
    for b in check_windows:
        base = b * wl.window_stride
        sub = wl.x[base: base + (wl.num_channels - 1) * wl.channel_stride + wl.n]
        o_s, o_out = oracle.detect(sub, oracle.Layout.of(wl, num_windows=1))
        nz = o_s[0] != 0
        worst = max(worst, float(np.max(np.abs(s_host[b][nz] - o_s[0][nz]) / o_s[0][nz])))
        match += int(all(o_out[f][0] == res[f][b] for f in
                         ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates")))
    out["oracle_check"] = {"windows": list(check_windows), "selections_equal": match,
                           "max_score_rel_err": worst}
    del det
    # the same batch with FFT scores and with matrix-core scores: wall time per
    # call over back-to-back calls, and whether every selection field equals
    # the direct path's
    for key, flag in (("fft_scores", pkg.FFT_SCORES), ("mfma_scores", pkg.MFMA_SCORES)):
        adesc, akeep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                                     wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights,
                                     flags=flag)
        adet = pkg.Detector(x, adesc, akeep, want_scores=False)
        adet.run()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(repeats):
            adet.run()
        torch.cuda.synchronize()
        a_ms = (time.perf_counter() - t0) * 1e3 / repeats
        ares = adet.results_numpy()
        same = all(np.array_equal(ares[f], res[f]) for f in
                   ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates"))
        out[key] = {"ms_per_call_back_to_back": a_ms, "lag_samples_per_sec": pairs / (a_ms / 1e3),
                    "traces_per_sec": wl.num_windows / (a_ms / 1e3),
                    "selections_equal_direct": bool(same)}
        del adet
        torch.cuda.empty_cache()
    return out


def timed_calls(call, steps):
    """Runs call() `steps` times between two events on the current stream;
    returns (wall ms per call, event ms per call, last result)."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    out = None
    for _ in range(steps):
        out = call()
    e1.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    return wall, e0.elapsed_time(e1) / steps, out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for "
              f"--gpus {args.gpus}); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2201_01684_amd as pkg
    from gen import make_workload

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")

    if args.calibrate_copy_mib:
        nbytes = args.calibrate_copy_mib << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": nbytes, "launches": 3}), flush=True)
        return

    if args.mode == "rolling":
        return bench_rolling(args)
    if args.mode in ("similarity", "centred"):
        return bench_similarity(args)
    if args.mode == "spectral":
        return bench_spectral(args)

    t_gen = time.perf_counter()
    wl = make_workload(args.workload)
    sha = wl.sha256
    t_gen = time.perf_counter() - t_gen
    pairs = wl.pairs()
    x = torch.from_numpy(wl.x).to(dev)
    fft = args.mode == "fft"
    mfma = args.mode == "mfma"
    desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                               wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights,
                               flags=pkg.FFT_SCORES if fft else (pkg.MFMA_SCORES if mfma else 0))
    det = pkg.Detector(x, desc, keep, want_scores=True)
    plan = pkg.describe_plan(desc)
    scored = plan["pairs_scored"]
    print(f"# {wl.name}: {wl.num_windows} windows x {wl.num_channels} ch x {wl.n} samples, "
          f"T {wl.tmin}..{wl.tmax}, {pairs:.4e} pairs, generated in {t_gen:.1f}s, "
          f"workspace {det.ws_bytes / 2**20:.1f} MiB", file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        det.run()
    torch.cuda.synchronize()

    ev = HipEvents()
    sets = [ev.create(5) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        det.run_staged(sets[k])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    stage_ms = np.array([[ev.elapsed_ms(s[j], s[j + 1]) for j in range(4)] for s in sets])
    call_ms = np.array([ev.elapsed_ms(s[0], s[4]) for s in sets])   # each whole call
    for s in sets:
        ev.destroy(s)
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = pairs / (ms_per_step / 1e3)
    score_ms = float(stage_ms[:, 1].mean())
    # the roofline counts what the score kernels evaluate: with overlapping
    # windows sharing block partials that is fewer pairs than the definition sums
    achieved = FLOP_PER_PAIR * scored / (score_ms / 1e3) / 1e12
    res = det.results_numpy()
    scores = det.scores
    if fft:
        fft_bytes = fft_stage_bytes(wl, plan)
        roofline = {"kernel": "FFT score stage (prep, column, row and inverse-column "
                              "transform kernels)", "bound": "hbm",
                    "achieved": fft_bytes / (score_ms / 1e3) / 1e9,
                    "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": fft_bytes / (score_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
                    "traffic": counters_traffic(wl.name, "fft"), "bytes_per_launch": fft_bytes}
    elif mfma:
        ops = MFMA_OPS_PER_PAIR * scored
        roofline = {"kernel": "mfma_xcorr_kernel (score stage: digit preparation, edge sums, "
                              "matrix-core lag tiles)", "bound": "mfma",
                    "achieved": ops / (score_ms / 1e3) / 1e12, "peak": INT8_MFMA_PEAK_TOPS,
                    "unit": "TOP/s", "frac": ops / (score_ms / 1e3) / 1e12 / INT8_MFMA_PEAK_TOPS,
                    "traffic": counters_traffic(wl.name, "mfma"), "ops_per_launch": ops,
                    "fp32_equivalent_tflops": FLOP_PER_PAIR * scored / (score_ms / 1e3) / 1e12,
                    # the method's own unit: (x[i], x[i+T]) pairs per second, against
                    # the direct kernel's VALU pair ceiling (two instructions per pair)
                    "pairs_per_s": scored / (score_ms / 1e3),
                    "vs_valu_pair_ceiling": scored / (score_ms / 1e3) / VALU_PAIR_CEILING}
    else:
        roofline = {"kernel": "lag_score_kernel", "bound": "alu", "achieved": achieved,
                    "peak": FP32_VECTOR_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": achieved / FP32_VECTOR_PEAK_TFLOPS,
                    "traffic": counters_traffic(wl.name)}
    # HBM bandwidth the stage drew: the counter bytes per launch over the
    # stage's measured time (null with the traffic)
    roofline["hbm_gbs"] = (roofline["traffic"] / (score_ms / 1e3) / 1e9
                           if roofline["traffic"] else None)

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "lag·samples/s",
        "traces_per_sec": wl.num_windows / (ms_per_step / 1e3),
        "pct_fp32_peak": None if (fft or mfma) else 100.0 * FLOP_PER_PAIR * scored
                         / (ms_per_step / 1e3) / 1e12 / FP32_VECTOR_PEAK_TFLOPS,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64" if fft else ("i8" if mfma else "f32"),
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.meta["description"],
                   "windows": wl.num_windows, "channels": wl.num_channels, "n": wl.n,
                   "tmin": wl.tmin, "tmax": wl.tmax, "pairs": pairs, "sha256": sha,
                   "scoring": {0: "per window", 1: "shared block partials",
                               2: "fp64 FFT autocorrelation",
                               3: "int8-digit cross-correlation on the matrix cores"}[
                                   plan["mode"]],
                   "pairs_scored": scored, "lags_per_lane": plan["lags_per_lane"]},
        "call_ms": {"median": float(np.median(call_ms)), "min": float(call_ms.min())},
        "stage_ms": {"window_stats": float(stage_ms[:, 0].mean()),
                     "lag_score": score_ms,
                     "finalize": float(stage_ms[:, 2].mean()),
                     "select": float(stage_ms[:, 3].mean())},
        "roofline": roofline,
        "device": device_info(ev),
        "windows_flagged_unresolved": int(np.count_nonzero(res["flags"] & pkg.UNRESOLVED)),
        "windows_rescored": int(np.count_nonzero(res["n_rescored"])),
    }
    if args.graph:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            det.run()
        g.replay()
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        g_ms = (time.perf_counter() - t) * 1e3 / args.steps
        line["graph_replay"] = {"ms_per_step": g_ms, "value": pairs / (g_ms / 1e3),
                                "traces_per_sec": wl.num_windows / (g_ms / 1e3)}
        del g
    if not fft and not mfma and not args.no_fft_compare:
        # the same batch with FFT scores and with matrix-core scores, after and
        # outside the timed region: time per call and whether every selection matches
        del det
        torch.cuda.empty_cache()
        for key, flag in (("fft_scores", pkg.FFT_SCORES), ("mfma_scores", pkg.MFMA_SCORES)):
            adesc, akeep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n,
                                         wl.window_stride, wl.channel_stride, wl.tmin, wl.tmax,
                                         weights=wl.weights, flags=flag)
            adet = pkg.Detector(x, adesc, akeep, want_scores=False)
            adet.run()
            torch.cuda.synchronize()
            t = time.perf_counter()
            for _ in range(args.steps):
                adet.run()
            torch.cuda.synchronize()
            a_ms = (time.perf_counter() - t) * 1e3 / args.steps
            ares = adet.results_numpy()
            same = all(np.array_equal(ares[k], res[k]) for k in
                       ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates"))
            line[key] = {"ms_per_step": a_ms, "value": pairs / (a_ms / 1e3),
                         "traces_per_sec": wl.num_windows / (a_ms / 1e3),
                         "selections_equal_direct": bool(same)}
            if key == "mfma_scores":   # whole call, every pair of the definition
                line[key]["vs_valu_pair_ceiling"] = pairs / (a_ms / 1e3) / VALU_PAIR_CEILING
            del adet
            torch.cuda.empty_cache()
    if wl.truth is not None:
        d = wl.truth > 0
        if wl.jitter:
            ok = np.abs(res["period"][d] - wl.truth[d]) <= np.ceil(0.02 * wl.truth[d])
        else:
            ok = res["period"][d] == wl.truth[d]
        line["planted_period_hits"] = f"{int(ok.sum())}/{int(d.sum())}"
    if args.mode == "detect" and not args.no_configs:
        # every trace configuration, after and outside the timed region
        if "det" in locals():
            del det
        torch.cuda.empty_cache()
        configs = {}
        for key, name, repeats, check in CONFIGS:
            if name == wl.name:
                cwl, cx = wl, x
            else:
                cwl, cx = make_workload(name), None
            configs[key] = bench_config(pkg, ev, cwl, repeats, check, x=cx)
            del cwl, cx
            torch.cuda.empty_cache()
            print(f"# {key} ({name}): {configs[key]['call_ms']['median']:.4f} ms per call",
                  file=sys.stderr, flush=True)
        line["configs"] = configs

    if not args.no_cpu_baseline:
        import oracle
        lay = oracle.Layout.of(wl)
        per_window = pairs // wl.num_windows
        done, t_cpu, match, worst = 0, 0.0, 0, 0.0
        s_host = None
        while done < wl.num_windows and (done == 0 or t_cpu < args.cpu_seconds):
            b = done
            base = b * wl.window_stride
            sub = wl.x[base: base + (wl.num_channels - 1) * wl.channel_stride + wl.n]
            lay1 = oracle.Layout.of(wl, num_windows=1)
            t = time.perf_counter()
            o_scores, o_out = oracle.detect(sub, lay1)
            t_cpu += time.perf_counter() - t
            if s_host is None:
                s_host = scores.double().cpu().numpy()
            g = s_host[b]
            o = o_scores[0]
            nz = o != 0
            worst = max(worst, float(np.max(np.abs(g[nz] - o[nz]) / o[nz])) if nz.any() else 0.0)
            match += int(o_out["period"][0] == res["period"][b])
            done += 1
        line["cpu_baseline"] = {"value": done * per_window / t_cpu, "unit": "lag·samples/s",
                                "cores": oracle.threads(), "kind": "oracle",
                                "cpu_model": cpu_model(), "nproc": os.cpu_count(),
                                "sample": f"first {done} of {wl.num_windows} windows, all "
                                          f"{wl.lags} lags each, {t_cpu:.1f} s"}
        line["parity_sample"] = {"windows": done, "period_match": match,
                                 "max_score_rel_err": worst}
    # Device memory is released and the stream drained before the line is
    # printed; bench.py starts no child process (the oracle's OpenMP workers
    # are threads of this one), so nothing outlives the JSON line.
    del x, scores
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    print(json.dumps(line), flush=True)


def bench_similarity(args):
    """Algorithm 2 on finalist periods: one step is one gpoeo_pd_similarity call
    (or, with --mode centred, one gpoeo_pd_score_centred call) on 5 (window,
    period) queries per window, built from a detection run before timing."""
    import numpy as np
    import torch

    import paper_2201_01684_amd as pkg
    from gen import make_workload

    wl = make_workload(args.workload)
    x = torch.from_numpy(wl.x).to("cuda:0")
    desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                               wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights)
    det = pkg.Detector(x, desc, keep, want_scores=False)
    det.run()
    res = det.results_numpy()
    ws, ts = [], []
    for b in range(wl.num_windows):
        p = max(int(res["period"][b]), 2)
        for t in (p, p - 1, p + 1, 2 * p, max(1, p // 2)):
            ws.append(b)
            ts.append(t)
    wt = torch.tensor(np.asarray(ws, dtype=np.int32), device="cuda:0")
    tt = torch.tensor(np.asarray(ts, dtype=np.int32), device="cuda:0")
    centred = args.mode == "centred"
    call = pkg.score_centred if centred else pkg.similarity
    for _ in range(args.warmup):
        call(x, desc, wt, tt)
    ms, ev_ms, err = timed_calls(lambda: call(x, desc, wt, tt), args.steps)
    g = err.cpu().numpy()
    samples = sum(wl.num_channels * (wl.n // t) * t for t in ts if wl.n // t >= 2)
    # point pairs (sub-curve i against i + 1): each EM fit and each centred
    # comparison covers one pair's T points
    pair_points = sum(wl.num_channels * (wl.n // t - 1) * t for t in ts if wl.n // t >= 2)
    if centred:
        roofline = call_roofline("centred_kernel", "alu_f64", CENTRED_FLOP * pair_points, ev_ms,
                                 {"flop_per_launch": CENTRED_FLOP * pair_points})
    else:
        em = EM_FLOP * 3 * 20 * pair_points
        roofline = call_roofline("similarity_kernel<3>", "alu_f64", em, ev_ms,
                                 {"flop_per_launch": em})
    metric = ("mean-removed score evaluations/sec (Algorithm 2 relative values, 5 finalist "
              "periods per window)" if centred else
              "grouped-similarity evaluations/sec (Algorithm 2, 5 finalist periods per window)")
    line = {
        "metric": metric,
        "value": len(ts) / (ms / 1e3), "unit": "period evaluations/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.meta["description"],
                   "windows": wl.num_windows, "queries": len(ts),
                   "sub_curve_samples": samples, "sha256": wl.sha256,
                   **({} if centred else {"num_groups": 3, "em_iters": 20})},
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        import oracle
        lay = oracle.Layout.of(wl, centred=centred)
        done, t_cpu, worst = 0, 0.0, 0.0
        while done < len(ts) and (done == 0 or t_cpu < args.cpu_seconds):
            k = min(len(ts), done + 5)
            t = time.perf_counter()
            if centred:
                o = oracle.score_list(wl.x, lay, ws[done:k], ts[done:k])
            else:
                o = oracle.similarity(wl.x, lay, ws[done:k], ts[done:k])
            t_cpu += time.perf_counter() - t
            nz = o > 0
            if nz.any():
                worst = max(worst, float(np.max(np.abs(g[done:k][nz] - o[nz]) / o[nz])))
            done = k
        line["cpu_baseline"] = {"value": done / t_cpu, "unit": "period evaluations/s",
                                "cores": oracle.threads(), "kind": "oracle", "cpu_model": cpu_model(),
                                "sample": f"first {done} of {len(ts)} queries, {t_cpu:.1f} s"}
        line["parity_sample"] = {"queries": done, "max_rel_err": worst}
    print(json.dumps(line), flush=True)


def bench_spectral(args):
    """Algorithm 1's FFT front end over the workload's windows: one step is one
    gpoeo_pd_spectral_candidates call (amplitude spectra, peaks, candidates)."""
    import numpy as np
    import torch

    import paper_2201_01684_amd as pkg
    from gen import make_workload

    wl = make_workload(args.workload)
    x = torch.from_numpy(wl.x).to("cuda:0")
    desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                               wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights)
    params = pkg.spectral_params()
    det = pkg.SpectralDetector(x, desc, params, keep)
    for _ in range(args.warmup):
        det.run()
    ms, ev_ms, _ = timed_calls(det.run, args.steps)
    res = det.results_numpy()
    # window statistics (two passes over the samples), the transforms (the
    # samples once more; above 2048 points each pair's complex fp64 transform
    # written and read back), the amplitudes written and read by the selection
    seqs = wl.num_windows * wl.num_channels
    length = pow2_at_least(wl.n)
    half = length // 2 + 1
    sweeps = 2 * 16 * ((seqs + 1) // 2) * length if length > 2048 else 0
    spec_bytes = float(3 * 4 * seqs * wl.n + sweeps + 2 * 8 * seqs * half)
    roofline = call_roofline("spectral call: window statistics, column and row transforms, "
                             "amplitude selection", "hbm", spec_bytes, ev_ms,
                             {"bytes_per_launch": spec_bytes})
    line = {
        "metric": "spectral candidate lists/sec (Algorithm 1's FFT front end over every window)",
        "value": wl.num_windows / (ms / 1e3), "unit": "windows/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.meta["description"],
                   "windows": wl.num_windows, "channels": wl.num_channels, "n": wl.n,
                   "tmin": wl.tmin, "tmax": wl.tmax, "sha256": wl.sha256,
                   "c_peak": params.c_peak, "max_candidates": params.max_candidates},
        "mean_candidates": float(res["count"].mean()),
        "windows_flagged_unresolved": int(np.count_nonzero(res["flags"])),
        "roofline": roofline,
    }
    if wl.truth is not None:
        d = wl.truth > 0
        hit = [any(abs(int(t) - int(wl.truth[b])) <= max(1, int(wl.truth[b]) // 50)
                   for t in res["periods"][b][:res["count"][b]]) for b in np.nonzero(d)[0]]
        line["planted_period_among_candidates"] = f"{int(sum(hit))}/{int(d.sum())}"
    if not args.no_cpu_baseline:
        import oracle
        span = (wl.num_channels - 1) * wl.channel_stride + wl.n
        done, t_cpu, match = 0, 0.0, 0
        while done < wl.num_windows and (done == 0 or t_cpu < args.cpu_seconds):
            base = done * wl.window_stride
            xw = np.stack([wl.x.reshape(-1)[base + c * wl.channel_stride:
                                            base + c * wl.channel_stride + wl.n]
                           for c in range(wl.num_channels)])
            t = time.perf_counter()
            o = oracle.spectral_candidates(xw, wl.tmin, wl.tmax, params.c_peak,
                                           params.max_candidates, wl.weights)
            t_cpu += time.perf_counter() - t
            r = res[done]
            match += int(list(r["bins"][:r["count"]]) == o["bins"])
            done += 1
        line["cpu_baseline"] = {"value": done / t_cpu, "unit": "windows/s", "cores": 1,
                                "kind": "oracle", "cpu_model": cpu_model(),
                                "sample": f"first {done} of {wl.num_windows} windows, "
                                          f"{t_cpu:.1f} s (numpy FFT, one thread)"}
        line["parity_sample"] = {"windows": done, "candidate_lists_equal": match}
    print(json.dumps(line), flush=True)


def bench_rolling(args):
    """Rolling detection (Algorithm 3) over the workload's windows: one step is one
    gpoeo_pd_detect_rolling call (whole-window pass, suffix schedule, suffix pass,
    combination)."""
    import numpy as np
    import torch

    import paper_2201_01684_amd as pkg
    from gen import make_workload

    wl = make_workload(args.workload)
    x = torch.from_numpy(wl.x).to("cuda:0")
    desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                               wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights,
                               flags=pkg.FFT_SCORES if args.fft_scores
                               else (pkg.MFMA_SCORES if args.mfma_scores else 0))
    params = pkg.rolling_params()
    det = pkg.RollingDetector(x, desc, params, keep)
    for _ in range(args.warmup):
        det.run()
    ms, ev_ms, _ = timed_calls(det.run, args.steps)
    res = det.results_numpy()
    # the work of both passes: every whole window, then every suffix window
    # (N_j = N - start_j samples, lags up to min(Tmax, N_j / 2))
    c = wl.num_channels
    lag_sum = lambda n, tm: (tm - wl.tmin + 1) * n - (tm * (tm + 1) - (wl.tmin - 1) * wl.tmin) // 2
    pairs_a = wl.num_windows * c * lag_sum(wl.n, wl.tmax)
    suffix = [(wl.n - int(st), min(wl.tmax, (wl.n - int(st)) // 2))
              for b in range(wl.num_windows) for st in res["starts"][b][:res["n_windows"][b]]]
    pairs_c = sum(c * lag_sum(n, tm) for n, tm in suffix if tm >= wl.tmin)
    if args.fft_scores:
        work = fft_stage_bytes(wl, pkg.describe_plan(desc))   # the whole-window pass
        # suffix pass: slots j of window b are sequences (b * jmax + j) * C + c,
        # paired two by two; a pair's transform holds its longer suffix
        jmax = int(np.floor((2 + params.c_eval * params.step - params.c_measure) / params.step)) + 2
        need = np.zeros(wl.num_windows * jmax * c, dtype=np.int64)
        tms = []
        for b in range(wl.num_windows):
            for j, st in enumerate(res["starts"][b][:res["n_windows"][b]]):
                n_j = wl.n - int(st)
                tm = min(wl.tmax, n_j // 2)
                for ch in range(c):
                    need[(b * jmax + j) * c + ch] = n_j + tm
                    tms.append(tm)
        if need.size % 2:
            need = np.append(need, 0)
        lens = [pow2_at_least(int(v)) for v in need.reshape(-1, 2).max(axis=1) if v > 0]
        work += transform_bytes(lens, sum(n * c for n, _ in suffix), len(tms), tms)
        roofline = call_roofline("both FFT score passes (whole windows, then suffix windows "
                                 "by length class)", "hbm", work, ev_ms,
                                 {"bytes_per_launch": work})
    elif args.mfma_scores:
        work = MFMA_OPS_PER_PAIR * (pairs_a + pairs_c)
        roofline = call_roofline("mfma_xcorr_kernel, both passes (whole windows, suffix "
                                 "windows)", "mfma", work, ev_ms,
                                 {"ops_per_launch": work, "pairs": pairs_a + pairs_c})
    else:
        work = FLOP_PER_PAIR * (pairs_a + pairs_c)
        roofline = call_roofline("lag_score_kernel, both passes (whole windows, suffix "
                                 "windows)", "alu_f32", work, ev_ms,
                                 {"flop_per_launch": work, "pairs": pairs_a + pairs_c})
    line = {
        "metric": "rolling detections/sec (Algorithm 3 over every window of the batch)",
        "value": wl.num_windows / (ms / 1e3), "unit": "windows/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64" if args.fft_scores else ("i8" if args.mfma_scores else "f32"),
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.meta["description"],
                   "windows": wl.num_windows, "channels": wl.num_channels, "n": wl.n,
                   "tmin": wl.tmin, "tmax": wl.tmax, "sha256": wl.sha256,
                   "c_measure": params.c_measure, "step": params.step, "c_eval": params.c_eval,
                   "diff_threshold": params.diff_threshold,
                   "scoring": "fp64 FFT autocorrelation" if args.fft_scores
                   else ("int8-digit cross-correlation on the matrix cores" if args.mfma_scores
                         else "direct")},
        "stable_windows": int(np.count_nonzero(res["stable"])),
        "mean_suffix_windows": float(res["n_windows"].mean()),
        "windows_flagged_unresolved": int(np.count_nonzero(res["flags"])),
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        import oracle
        lay1 = oracle.Layout.of(wl, num_windows=1)
        span = (wl.num_channels - 1) * wl.channel_stride + wl.n
        done, t_cpu, match = 0, 0.0, 0
        while done < wl.num_windows and (done == 0 or t_cpu < args.cpu_seconds):
            sub = wl.x[done * wl.window_stride: done * wl.window_stride + span]
            t = time.perf_counter()
            o = oracle.rolling(sub, lay1)[0]
            t_cpu += time.perf_counter() - t
            g = res[done]
            match += int(o["period"] == g["period"] and o["stable"] == g["stable"]
                         and o["smpdur_next"] == g["smpdur_next"])
            done += 1
        line["cpu_baseline"] = {"value": done / t_cpu, "unit": "windows/s",
                                "cores": oracle.threads(), "kind": "oracle",
                                "cpu_model": cpu_model(),
                                "sample": f"first {done} of {wl.num_windows} windows, {t_cpu:.1f} s"}
        line["parity_sample"] = {"windows": done, "period_stable_next_match": match}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
