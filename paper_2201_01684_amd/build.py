"""Builds libgpoeo_pd.so for gfx950 from the HIP sources in csrc/ (in-tree).

Every source is compiled by hipcc with packed FP32 instructions disabled
(``-Xclang -target-feature -Xclang -packed-fp32-ops``) and linked into one
shared library next to this file.  The library's HIP runtime dependency
(libamdhip64.so.7) resolves first against PyTorch's bundled runtime, so the
library and torch share one HIP runtime (streams and device pointers are
interchangeable).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJ_DIR = os.path.join(ROOT, "_build", "obj")
LIB_NAME = "libgpoeo_pd.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)

SOURCES = ["api.cpp", "lag_score.hip", "window_stats.hip", "select.hip", "rolling.hip",
           "similarity.hip", "fft_score.hip", "centred.hip", "mfma_score.hip", "noalloc.hip"]
# The selection re-evaluates scores and thresholds as plain fp64 expressions
# (one rounding per operation, as written); no multiply-add contraction there,
# nor in the FFT, whose error bound assumes separately rounded products, nor in
# the statistics and finalisation, which the fused small-window kernel repeats
# bit for bit.
EXTRA_FLAGS = {"select.hip": ["-ffp-contract=off"], "rolling.hip": ["-ffp-contract=off"],
               "window_stats.hip": ["-ffp-contract=off"],
               "similarity.hip": ["-ffp-contract=off"], "fft_score.hip": ["-ffp-contract=off"],
               "centred.hip": ["-ffp-contract=off"], "mfma_score.hip": ["-ffp-contract=off"]}
ARCH = os.environ.get("GPOEO_PD_ARCH", "gfx950")
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-command-line-argument", "-Wno-unknown-pragmas",
             "-I", INCLUDE, "-I", CSRC]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _torch_lib_dir() -> str | None:
    try:
        import importlib.util
        spec = importlib.util.find_spec("torch")
        if spec and spec.origin:
            d = os.path.join(os.path.dirname(spec.origin), "lib")
            if os.path.exists(os.path.join(d, "libamdhip64.so")):
                return d
    except Exception:
        pass
    return None


# Host-code sanitizer build (a CPU check of the argument validation, plan and
# workspace arithmetic): AddressSanitizer and UndefinedBehaviorSanitizer on the
# host side of every source only (each flag after -Xarch_host; the gfx950 code
# is built as usual), into _build/, never next to the package.  Its runtime is
# not linked in: the process that loads it preloads ROCm clang's ASan runtime.
SAN_DIR = os.path.join(ROOT, "_build", "hostsan")
SAN_LIB_PATH = os.path.join(SAN_DIR, LIB_NAME)
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def sanitizer_runtime() -> str:
    """ROCm clang's shared ASan runtime (it carries the UBSan handlers too)."""
    import glob
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("clang ASan runtime not found under /opt/rocm/llvm")
    return hits[-1]


def _compile(src: str, verbose: bool, sanitize: bool = False) -> str:
    obj_dir = os.path.join(SAN_DIR, "obj") if sanitize else OBJ_DIR
    obj = os.path.join(obj_dir, os.path.splitext(src)[0] + ".o")
    flags = [f for f in HIP_FLAGS if f != "-O3"] + ["-O1", "-g", *SAN_FLAGS] if sanitize \
        else HIP_FLAGS
    cmd = [_hipcc(), *flags, *EXTRA_FLAGS.get(src, []), "-x", "hip", "-c",
           os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile every source and link the shared library (always rebuilds).
    sanitize=True builds the host-sanitized library at SAN_LIB_PATH instead."""
    lib_path = SAN_LIB_PATH if sanitize else LIB_PATH
    os.makedirs(os.path.join(SAN_DIR, "obj") if sanitize else OBJ_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, sanitize), SOURCES))
    link = [_hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", lib_path + ".tmp"]
    tl = _torch_lib_dir()
    if tl:
        link += [f"-L{tl}", f"-Wl,-rpath,{tl}"]
    if verbose:
        print(" ".join(link), flush=True)
    r = subprocess.run(link, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(lib_path + ".tmp", lib_path)
    return lib_path


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize-host" in sys.argv))
