"""The integer GEMM launcher's choice of kernel and grid
(paper_2404_00456_amd/csrc/gemm_plan.hpp), built for the host with the
address and undefined-behaviour sanitizers and checked on the Llama-2
projection shapes and at the boundaries of its rule
(tests/native/gemm_plan_check.cpp).  Nothing runs on a GPU."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "native", "gemm_plan_check.cpp")
CSRC = os.path.join(ROOT, "paper_2404_00456_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_gemm_plan_choices():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "check")
        subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-fsanitize=address,undefined",
                        "-fno-sanitize-recover=all", "-I", CSRC, SRC, "-o", exe], check=True,
                       capture_output=True)
        res = subprocess.run([exe], capture_output=True, text=True, timeout=60)
        assert res.returncode == 0 and res.stdout.strip() == "ok", res.stdout + res.stderr
