"""The oracle's pin suites again, with the oracle built under AddressSanitizer
and UndefinedBehaviorSanitizer (CPU only). Any out-of-bounds access, signed
overflow, invalid shift or other undefined behaviour inside the oracle aborts
the run, so a guard that only works by wrapping arithmetic fails here even
where the pins' values happen to come out right.

The pool generator is numpy code with no native part, so there is nothing of
its own to sanitize; the pins drive it through the same run."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_FILES = ["tests/test_oracle_pins.py", "tests/test_oracle_group_pins.py", "tests/test_oracle_stream_pins.py",
             "tests/test_oracle_prefix_pins.py", "tests/test_oracle_diag_pins.py"]


def _runtime(name):
    path = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.slow
def test_pins_pass_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_san.so"))
    env = dict(os.environ)
    # the ASan runtime has to come first in the process; the interpreter's own
    # allocations are not the oracle's, so leak reports are off
    env["LD_PRELOAD"] = asan + ((" " + env["LD_PRELOAD"]) if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["PACE_ORACLE_LIB"] = lib
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-s", "-p", "no:cacheprovider", *PIN_FILES],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert "runtime error" not in out and "AddressSanitizer" not in out, out
    assert " passed" in r.stdout, out
