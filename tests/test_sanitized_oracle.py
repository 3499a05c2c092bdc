"""The oracle's CPU tests once more, with the oracle built under
AddressSanitizer and UndefinedBehaviorSanitizer (any finding aborts).

The C oracle is the ground truth of every parity test, so an out-of-bounds
read, a use of uninitialised or freed memory, a signed overflow or an
oversized shift inside it could make it agree with a wrong kernel.  The child
pytest loads ``liboracle_san.so`` (``OQ_SANITIZE=1``) with gcc's libasan
preloaded, which an instrumented library loaded into an uninstrumented
interpreter needs; leak checking is off (the interpreter's own allocations)."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def _libasan():
    try:
        p = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return p if os.path.isabs(p) and os.path.exists(p) else None


def test_oracle_suite_under_asan_and_ubsan():
    asan = _libasan()
    if asan is None:
        pytest.skip("gcc's libasan is not installed")
    files = sorted(os.path.join("tests", f) for f in os.listdir(HERE)
                   if f.startswith("test_oracle_") and f.endswith(".py"))
    env = dict(os.environ)
    env["OQ_SANITIZE"] = "1"
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["LD_PRELOAD"] = " ".join(x for x in (asan, os.environ.get("LD_PRELOAD", "")) if x)
    env.setdefault("OMP_NUM_THREADS", "4")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu"] + files,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail
