"""The oracle's CPU pins again, with hco.c built under AddressSanitizer and
UndefinedBehaviorSanitizer (host code only): any out-of-bounds access, use
after free or undefined arithmetic in the oracle fails the run.  The pins run
in a child process that preloads the ASan runtime and loads the sanitizer
build through HCO_LIB."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    if shutil.which("gcc") is None:
        return None
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = out.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(900)
def test_oracle_pins_under_address_and_ub_sanitizers():
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    sys.path.insert(0, os.path.join(ROOT, "oracle"))
    import build as oracle_build  # the oracle's own build script
    lib = oracle_build.build(sanitize=True)
    env = dict(os.environ)
    env.update(HCO_LIB=lib, LD_PRELOAD=asan,
               # the interpreter's own allocations are not the oracle's
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
           os.path.join(ROOT, "tests", "test_oracle.py"),
           os.path.join(ROOT, "tests", "test_oracle_blocked.py"),
           os.path.join(ROOT, "tests", "test_oracle_bloom.py")]
    res = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=880)
    tail = (res.stdout[-3000:] + res.stderr[-3000:])
    assert res.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in res.stderr and "runtime error" not in res.stderr, tail
    assert " passed" in res.stdout
