"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer:
every ABI test (validation of shapes, strides, batches, pointers and
arguments; size helpers; the debug switch) against a host-instrumented build.
CPU only: nothing is launched."""

import subprocess
import sys
from pathlib import Path

ROOT = Path(__file__).resolve().parents[1]


def test_abi_tests_pass_under_host_asan_and_ubsan():
    r = subprocess.run([sys.executable, "-m", "paper_2609_20971_amd.sanitize_host"], cwd=ROOT,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout
