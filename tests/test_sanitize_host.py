"""The host side of libtoc (encoder, upload image builder, physical encoding)
under AddressSanitizer and UndefinedBehaviorSanitizer: a sanitizer build of the
library (device code unsanitized) runs the encoder, layout and physical-encoding
test files in a subprocess; any report aborts that run.  CPU only."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(900)
def test_host_code_under_asan_and_ubsan():
    if os.environ.get("TOC_LIB_PATH"):
        pytest.skip("already running against the sanitizer build")
    r = subprocess.run([sys.executable, "-m", "paper_1702_06943_amd.sanitize"], cwd=ROOT,
                       capture_output=True, text=True)
    assert r.returncode == 0, (r.stdout[-3000:] + r.stderr[-3000:])
    assert " passed" in r.stdout
