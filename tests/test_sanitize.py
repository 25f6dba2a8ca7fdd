"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU):
runs tests/sanitize.py, which rebuilds the oracle, the input generators and
the library's host code with both sanitizers and reruns the CPU tests against
those builds; any report aborts that run."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.slow
def test_host_code_is_clean_under_sanitizers():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "sanitize.py")],
                       capture_output=True, text=True, timeout=1500)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "[sanitize] clean" in r.stdout, tail
