"""CPU sanitizer leg: the oracle and the library's host code under
AddressSanitizer and UndefinedBehaviorSanitizer.

Two builds, each made by the committed build switch of its side:
  - oracle.c with gcc -fsanitize=address,undefined (oracle.build(sanitize=True));
  - every library source with the sanitizers on its host side only
    (paper_2201_01684_amd/build.py --sanitize-host): the argument validation,
    launch plan and workspace arithmetic of the C ABI (make_plan's int64 size
    products, the rolling and spectral plans, the no-allocation entry point's
    checks).
Each runs its own test files in a child process that preloads the matching
sanitizer runtime; any finding aborts that process (-fno-sanitize-recover), so
the leg passes only if the whole child test run passes.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pytestmark = pytest.mark.slow


def _stale(target, sources):
    if not os.path.exists(target):
        return True
    t = os.path.getmtime(target)
    return any(os.path.getmtime(s) > t for s in sources)


def _child(env_extra, tests):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:alloc_dealloc_mismatch=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "-m", "not gpu and not slow", *tests], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    return out


def test_oracle_under_asan_ubsan():
    import oracle
    src = [os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(ROOT, "oracle", "oracle.h")]
    if _stale(oracle.SAN_LIB_PATH, src):
        oracle.build(sanitize=True)
    pre = " ".join(subprocess.run(["gcc", f"-print-file-name={lib}"], capture_output=True,
                                  text=True, check=True).stdout.strip()
                   for lib in ("libasan.so", "libubsan.so"))
    tests = sorted(glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")))
    out = _child({"LD_PRELOAD": pre, "GPOEO_ORACLE_LIBRARY": oracle.SAN_LIB_PATH}, tests)
    assert " passed" in out


def test_library_host_code_under_asan_ubsan():
    from paper_2201_01684_amd import build as hb
    src = [os.path.join(hb.CSRC, s) for s in hb.SOURCES]
    src += glob.glob(os.path.join(hb.CSRC, "*.h")) + [os.path.join(ROOT, "include", "gpoeo_pd.h")]
    if _stale(hb.SAN_LIB_PATH, src):
        hb.build(sanitize=True)
    out = _child({"LD_PRELOAD": hb.sanitizer_runtime(), "GPOEO_PD_LIBRARY": hb.SAN_LIB_PATH},
                 [os.path.join(ROOT, "tests", "test_abi_host.py")])
    assert " passed" in out
