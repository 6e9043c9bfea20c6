"""Division by launch constants (FastDiv): the host build of the library's own
header against plain integer division.  The kernels' index decoding (tile,
image, row, split) depends on it; GPU parity covers its device use."""
import os
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_fastdiv_matches_integer_division():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "fastdiv_check")
        src = os.path.join(HERE, "fastdiv_check.hip")
        r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-O2", "-std=c++17", src, "-o", exe],
                           capture_output=True, text=True, timeout=300)
        assert r.returncode == 0, r.stderr
        r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
        assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout + r.stderr
