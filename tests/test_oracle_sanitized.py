"""The oracle's pins, run again against a build of the oracle with
AddressSanitizer and UndefinedBehaviorSanitizer (every report fatal): an
out-of-bounds access, a use after free or undefined behaviour anywhere the
pins reach fails this test.  The sanitized library is loaded into a child
Python with the sanitizer runtimes preloaded (leak detection off: the
interpreter's own allocations at exit are not the oracle's)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["tests/test_oracle.py", "tests/test_oracle_heads.py", "tests/test_oracle_block.py",
        "tests/test_oracle_rounding.py", "tests/test_oracle_explicit.py"]


def _runtime(name):
    r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_under_sanitizers():
    from oracle.build import build
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc's sanitizer runtimes are not installed")
    lib = build(variant="sanitized")
    env = dict(os.environ)
    env.update({
        "PA_ORACLE_VARIANT": "sanitized",
        "LD_PRELOAD": f"{asan}:{ubsan}",
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "OMP_NUM_THREADS": "4",
    })
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PINS]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr, tail
    assert "runtime error" not in r.stderr, tail
    assert os.path.exists(lib)
