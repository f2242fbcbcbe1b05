"""The CPU oracle under the compiler's sanitizers (CPU only).

- AddressSanitizer + UndefinedBehaviorSanitizer: tests/sanitize_oracle.c drives every oracle entry
  point over small inputs and their edge cases (empty programs, zero rows, k = 0 and k = n, NaN,
  +-inf, +-0, denormal values, irregular trees of every depth up to 12, degenerate refit sets) in an
  executable built with -fsanitize=address,undefined; any out-of-bounds access, leak or undefined
  behaviour ends it with a non-zero status.
- UndefinedBehaviorSanitizer over the pins: the oracle's pin suites (tree routing, sums, policy,
  ranking, tracks, selection, refit) run in a child process against a -fsanitize=undefined build of
  the oracle that aborts at the first report.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "harl_oracle.c")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc is needed for the sanitizer builds")


def test_oracle_entry_points_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "sanitize_oracle")
    subprocess.run(["gcc", "-std=c99", *SAN, "-fopenmp", os.path.join(ROOT, "tests", "sanitize_oracle.c"), SRC,
                    "-o", exe, "-lm"], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                                UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1"))
    assert r.returncode == 0, "sanitizer report:\n%s\n%s" % (r.stdout[-4000:], r.stderr[-4000:])
    assert "ok" in r.stdout


def test_pins_under_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_ubsan.so")
    flags = [f for f in oracle.CFLAGS if f != "-O2"]
    subprocess.run(["gcc", *flags, "-O1", "-g", "-fsanitize=undefined", "-fno-sanitize-recover=undefined", SRC,
                    "-o", lib, "-lm"], check=True)
    tests = [os.path.join(ROOT, "tests", t) for t in ("test_oracle_pins.py", "test_oracle_gbdt.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *tests], cwd=ROOT,
                       capture_output=True, text=True, timeout=900,
                       env=dict(os.environ, HARL_ORACLE_LIBRARY=lib, UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1"))
    assert r.returncode == 0, "pins under UBSan failed:\n%s\n%s" % (r.stdout[-4000:], r.stderr[-4000:])
