"""Full-size parity on every window of the five workloads (not collected by pytest;
about 8 minutes of oracle time on 16 host threads).

    python tests/full_parity.py [w1 w2 w3 w4 w5]
    python tests/full_parity.py --rolling [w1 w2 w3 w4 w5]

For each workload: one gpoeo_pd_detect call over the whole batch with the
direct scores, one with GPOEO_PD_FFT_SCORES and one with GPOEO_PD_MFMA_SCORES,
then the fp64 oracle on every
window (in chunks, printing progress).  Reports, per path, the windows whose
selection differs from the oracle (period, verdict, T_c, local-search window,
candidate count), the largest relative score error over every (window, lag),
whether every oracle zero is reproduced, and the windows flagged UNRESOLVED.
Prints one JSON line per workload and a final summary line.

With --rolling: one gpoeo_pd_detect_rolling call over the whole batch with
each scoring (direct, FFT, matrix cores), then the oracle's rolling detection
on every window; reports the
windows whose verdict, T_init, suffix schedule (count, starts, periods),
selected window and period, stability or next sampling duration differ, the
largest relative difference of diff and of err, and the flagged windows.
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

FIELDS = ("period", "verdict", "t_cand", "t_low", "t_up", "n_candidates")


def main(names):
    import torch

    import oracle
    import paper_2201_01684_amd as pkg
    from gen import make_workload

    dev = torch.device("cuda:0")
    summary = {}
    for name in names:
        t0 = time.perf_counter()
        wl = make_workload(name)
        print(f"[{name}] {wl.num_windows} windows x {wl.num_channels} ch x {wl.n}, "
              f"sha256 {wl.sha256[:16]}", flush=True)
        x = torch.from_numpy(wl.x).to(dev)
        gpu = {}
        for mode, flags in (("direct", 0), ("fft", pkg.FFT_SCORES), ("mfma", pkg.MFMA_SCORES)):
            desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                                       wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights,
                                       flags=flags)
            det = pkg.Detector(x, desc, keep)
            det.run()
            torch.cuda.synchronize()
            gpu[mode] = (det.scores.cpu().numpy(), det.results_numpy())
            del det
            torch.cuda.empty_cache()
        del x
        torch.cuda.empty_cache()

        stats = {m: {"selection_mismatch": 0, "max_rel": 0.0, "zeros_ok": True, "unresolved": 0}
                 for m in gpu}
        lay1 = oracle.Layout.of(wl, num_windows=1)
        span = (wl.num_channels - 1) * wl.channel_stride + wl.n
        chunk = max(1, min(64, wl.num_windows))
        last = time.perf_counter()
        for b0 in range(0, wl.num_windows, chunk):
            b1 = min(wl.num_windows, b0 + chunk)
            lay = oracle.Layout.of(wl, num_windows=b1 - b0)
            sub = wl.x[b0 * wl.window_stride: (b1 - 1) * wl.window_stride + span]
            o_scores, o_out = oracle.detect(sub, lay)
            for m, (g_scores, g_res) in gpu.items():
                st = stats[m]
                g = g_scores[b0:b1].astype(np.float64)
                r = g_res[b0:b1]
                bad = np.zeros(b1 - b0, dtype=bool)
                for f in FIELDS:
                    bad |= r[f] != o_out[f]
                st["selection_mismatch"] += int(bad.sum())
                st["unresolved"] += int(np.count_nonzero(r["flags"] & pkg.UNRESOLVED))
                zero = o_scores == 0
                st["zeros_ok"] &= bool(np.all(g[zero] == 0))
                if (~zero).any():
                    rel = np.abs(g[~zero] - o_scores[~zero]) / np.abs(o_scores[~zero])
                    st["max_rel"] = max(st["max_rel"], float(rel.max()))
            if time.perf_counter() - last > 20 or b1 == wl.num_windows:
                print(f"[{name}] oracle windows {b1}/{wl.num_windows}, "
                      f"{time.perf_counter() - t0:.0f} s", flush=True)
                last = time.perf_counter()
        line = {"workload": name, "windows": wl.num_windows, "sha256": wl.sha256,
                "seconds": round(time.perf_counter() - t0, 1), **stats}
        print(json.dumps(line), flush=True)
        summary[name] = line
    ok = all(s[m]["selection_mismatch"] == 0 and s[m]["zeros_ok"] and s[m]["unresolved"] == 0
             and s[m]["max_rel"] <= 1e-4 for s in summary.values() for m in ("direct", "fft", "mfma"))
    print(json.dumps({"all_windows_match": ok,
                      "oracle_threads": oracle.threads()}), flush=True)
    return 0 if ok else 1


ROLL_FIELDS = ("verdict", "t_init", "n_windows", "period", "stable", "best", "smpdur_next")


def main_rolling(names):
    import torch

    import oracle
    import paper_2201_01684_amd as pkg
    from gen import make_workload

    dev = torch.device("cuda:0")
    summary = {}
    for name in names:
        t0 = time.perf_counter()
        wl = make_workload(name)
        print(f"[{name}] rolling: {wl.num_windows} windows x {wl.num_channels} ch x {wl.n}, "
              f"sha256 {wl.sha256[:16]}", flush=True)
        x = torch.from_numpy(wl.x).to(dev)
        gpu = {}
        for mode, flags in (("direct", 0), ("fft", pkg.FFT_SCORES), ("mfma", pkg.MFMA_SCORES)):
            desc, keep = pkg.make_desc(wl.num_windows, wl.num_channels, wl.n, wl.window_stride,
                                       wl.channel_stride, wl.tmin, wl.tmax, weights=wl.weights,
                                       flags=flags)
            det = pkg.RollingDetector(x, desc, pkg.rolling_params(), keep)
            det.run()
            torch.cuda.synchronize()
            gpu[mode] = det.results_numpy()
            del det
            torch.cuda.empty_cache()
        del x
        torch.cuda.empty_cache()
        stats = {m: {"mismatch": 0, "diff_rel": 0.0, "err_rel": 0.0, "flagged": 0} for m in gpu}
        span = (wl.num_channels - 1) * wl.channel_stride + wl.n
        chunk = max(1, min(32, wl.num_windows))
        last = time.perf_counter()
        for b0 in range(0, wl.num_windows, chunk):
            b1 = min(wl.num_windows, b0 + chunk)
            lay = oracle.Layout.of(wl, num_windows=b1 - b0)
            sub = wl.x[b0 * wl.window_stride: (b1 - 1) * wl.window_stride + span]
            o = oracle.rolling(sub, lay)
            for m, res in gpu.items():
                st = stats[m]
                g = res[b0:b1]
                bad = np.zeros(b1 - b0, dtype=bool)
                for f in ROLL_FIELDS:
                    bad |= g[f] != o[f]
                for k in range(b1 - b0):
                    c = int(o["n_windows"][k])
                    bad[k] |= not np.array_equal(g["starts"][k][:c], o["starts"][k][:c])
                    bad[k] |= not np.array_equal(g["periods"][k][:c], o["periods"][k][:c])
                st["mismatch"] += int(bad.sum())
                st["flagged"] += int(np.count_nonzero(g["flags"]))
                nz = o["diff"] != 0
                if nz.any():
                    st["diff_rel"] = max(st["diff_rel"], float(np.max(
                        np.abs(g["diff"][nz] - o["diff"][nz]) / np.abs(o["diff"][nz]))))
                nz = (o["period"] > 0) & (o["err"] != 0)
                if nz.any():
                    st["err_rel"] = max(st["err_rel"], float(np.max(
                        np.abs(g["err"][nz] - o["err"][nz]) / np.abs(o["err"][nz]))))
            if time.perf_counter() - last > 20 or b1 == wl.num_windows:
                print(f"[{name}] oracle windows {b1}/{wl.num_windows}, "
                      f"{time.perf_counter() - t0:.0f} s", flush=True)
                last = time.perf_counter()
        line = {"workload": name, "rolling": True, "windows": wl.num_windows,
                "sha256": wl.sha256, "seconds": round(time.perf_counter() - t0, 1), **stats}
        print(json.dumps(line), flush=True)
        summary[name] = line
    ok = all(s[m]["mismatch"] == 0 and s[m]["flagged"] == 0 and s[m]["err_rel"] <= 1e-4
             and s[m]["diff_rel"] <= 1e-6 for s in summary.values() for m in ("direct", "fft", "mfma"))
    print(json.dumps({"all_rolling_windows_match": ok, "oracle_threads": oracle.threads()}),
          flush=True)
    return 0 if ok else 1


if __name__ == "__main__":
    argv = sys.argv[1:]
    if argv and argv[0] == "--rolling":
        sys.exit(main_rolling(argv[1:] or ["w1", "w2", "w4", "w5", "w3"]))
    sys.exit(main(argv or ["w1", "w2", "w4", "w5", "w3"]))
