"""The oracle's pins pass under AddressSanitizer and UndefinedBehaviorSanitizer.

The full CPU suite runs the same way with ``python oracle/run_sanitized.py``
(a few minutes); this test keeps the quick part of it in every run.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("nm") is None,
                    reason="needs gcc and nm")
def test_oracle_pins_run_clean_under_asan_and_ubsan():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "oracle", "run_sanitized.py"),
                        "tests/test_oracle_pins.py", "-x"],
                       cwd=ROOT, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "sanitized oracle:" in out and " passed" in out, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
