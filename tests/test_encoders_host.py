"""The library's bit-level encoders built for the host and run over all
their inputs (tests/native/encoders_host_check.cpp): the e3m2 code of
every int4 value and its place in a 192-bit unit, the tiled layout's
head/tail slots, and the signed base-64 digits of every fp16 value that
the large-m rotation feeds to the integer matrix cores.  Same source as
the GPU kernels; nothing runs on a GPU."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "native", "encoders_host_check.cpp")
HIPCC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
def test_encoders_over_all_inputs():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "check")
        subprocess.run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O2", "-std=c++17",
                        "-I", os.path.join(ROOT, "include"), SRC, "-o", exe], check=True,
                       capture_output=True)
        res = subprocess.run([exe], capture_output=True, text=True, timeout=300)
        assert res.returncode == 0 and res.stdout.strip() == "ok", res.stdout + res.stderr
