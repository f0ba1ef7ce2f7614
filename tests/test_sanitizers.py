"""The CPU-side code under AddressSanitizer and UndefinedBehaviorSanitizer.

Two builds, cached under _build/san/ by the hash of their sources:
* oracle.c (gcc, -fsanitize=address,undefined), exercised by the oracle pins
  (tests/test_oracle_pins.py and the other oracle pin modules) in a process that
  preloads gcc's ASan runtime;
* the product library with its host code sanitized (hipcc, -Xarch_host
  -fsanitize=..., device code as usual), exercised by the C-ABI and host-only
  tests (argument validation, plans, layout offsets, the per-bit fits and the
  Eq. 4 dynamic programme) in a process that preloads clang's ASan runtime.

A sanitizer report, or any test failure, fails this test.  No GPU is used: the
tests run here make no HIP compute call.
"""
import hashlib
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CACHE = os.path.join(ROOT, "_build", "san")

ORACLE_TESTS = ["tests/test_oracle_pins.py", "tests/test_colwise_oracle.py",
                "tests/test_blockwise_oracle.py", "tests/test_terms_oracle.py"]
LIBRARY_TESTS = ["tests/test_abi_cpu.py", "tests/test_alloc_host.py"]


def _digest(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _run(tests, env_extra, timeout):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider", *tests]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=timeout)
    out = r.stdout + r.stderr
    return r.returncode, out


def _no_report(out):
    return "AddressSanitizer" not in out and "runtime error:" not in out and \
        "UndefinedBehaviorSanitizer" not in out


def test_oracle_under_sanitizers():
    import oracle

    os.makedirs(CACHE, exist_ok=True)
    lib = os.path.join(CACHE, f"liboracle_san_{_digest([os.path.join(ROOT, 'oracle', 'oracle.c')])}.so")
    if not os.path.exists(lib):
        oracle.build_sanitized(lib)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    env = {"LD_PRELOAD": asan, "ORACLE_LIB": lib}
    probe = subprocess.run(
        [sys.executable, "-c", "import ctypes, oracle; oracle._load(); "
         "print(hasattr(ctypes.CDLL(None), '__asan_init'))"],
        cwd=ROOT, env={**os.environ, **env, "ASAN_OPTIONS": "detect_leaks=0"},
        capture_output=True, text=True, timeout=300)
    assert probe.stdout.split() == ["True"], probe.stdout + probe.stderr[-2000:]
    rc, out = _run(ORACLE_TESTS, env, timeout=900)
    assert rc == 0 and _no_report(out), out[-4000:]
    assert " passed" in out


def test_library_host_code_under_sanitizers():
    pytest.importorskip("torch")
    sys.path.insert(0, ROOT)
    from paper_2406_05981_amd import build as hip_build

    srcs = hip_build.SOURCES + [os.path.join(ROOT, "include", "shiftadd.h")]
    os.makedirs(CACHE, exist_ok=True)
    lib = os.path.join(CACHE, f"libshiftadd_san_{_digest(srcs)}.so")
    if not os.path.exists(lib):
        hip_build.build_sanitized(lib)
    env = {"LD_PRELOAD": hip_build.asan_runtime(), "SHIFTADD_LIB": lib}
    # the child really loads the sanitized build with the ASan runtime in place
    probe = subprocess.run(
        [sys.executable, "-c", "import ctypes, paper_2406_05981_amd.shiftadd as sa; "
         "print(sa.LIB_PATH); print(hasattr(ctypes.CDLL(None), '__asan_init'))"],
        cwd=ROOT, env={**os.environ, **env, "ASAN_OPTIONS": "detect_leaks=0"},
        capture_output=True, text=True, timeout=300)
    assert probe.stdout.split() == [lib, "True"], probe.stdout + probe.stderr[-2000:]
    rc, out = _run(LIBRARY_TESTS, env, timeout=900)
    assert rc == 0 and _no_report(out), out[-4000:]
    assert " passed" in out and " skipped" not in out.split("\n")[-2], out[-2000:]
