"""Memory and undefined-behaviour checks of the native host code on the
CPU (no GPU):

- the oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
  (gcc, every UB report fatal) and run under its own pin tests, on the
  sizes that finish quickly there;
- the C ABI's host code (argument validation, size rules, the failure
  injection, the scratch entry point's size limit) built with both
  sanitizers (clang through hipcc, sanitizer flags for the host pass only)
  against counting stand-ins of the kernel launchers, and driven by
  tests/native/abi_host_check.cpp with no device.
"""
import glob
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def gcc_runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = p.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(gcc_runtime("libasan.so") is None, reason="needs gcc's ASan runtime")
def test_oracle_under_asan_ubsan():
    with tempfile.TemporaryDirectory() as d:
        lib = os.path.join(d, "liborc_san.so")
        subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                        "-fopenmp", "-fPIC", "-shared", "-fsanitize=address,undefined",
                        "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                        os.path.join(ROOT, "oracle", "quarot_oracle.c"), "-o", lib, "-lm"],
                       check=True)
        env = dict(os.environ, QUAROT_ORACLE_LIB=lib, LD_PRELOAD=gcc_runtime("libasan.so"),
                   ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", OMP_NUM_THREADS="2")
        tests = [os.path.join(ROOT, "tests", f) for f in (
            "test_oracle_pins.py", "test_oracle_clip_search.py", "test_oracle_grouped.py",
            "test_oracle_int8.py", "test_oracle_prologues.py", "test_oracle_kv_attention.py")]
        sel = ("not 8192 and not 4096 and not 64-128 and not rotation_helps and not shrinks "
               "and not columns_of_h and not kronecker_identity and not 172")
        res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                              "-k", sel, *tests], env=env, capture_output=True, text=True,
                             cwd=ROOT, timeout=900)
        assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
        assert "passed" in res.stdout


def clang_asan_runtime():
    hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return hits[0] if hits else None


@pytest.mark.skipif(not os.path.exists(HIPCC) or clang_asan_runtime() is None,
                    reason="needs hipcc and clang's ASan runtime")
def test_abi_host_code_under_asan_ubsan():
    csrc = os.path.join(ROOT, "paper_2404_00456_amd", "csrc")
    native = os.path.join(ROOT, "tests", "native")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
           "-fno-omit-frame-pointer"]
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "abi_check")
        # the ABI's host code and size rules, against counting stand-ins of
        # the kernel launchers (no device code at all)
        subprocess.run([HIPCC, "-O1", "-g", "-std=c++17", *san, "-I", os.path.join(ROOT, "include"),
                        os.path.join(csrc, "capi.cpp"), os.path.join(csrc, "host_rules.cpp"),
                        os.path.join(native, "launch_stubs.cpp"),
                        os.path.join(native, "abi_host_check.cpp"), "-o", exe],
                       check=True, capture_output=True, timeout=600)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
                   HIP_VISIBLE_DEVICES="-1")
        res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
        assert res.returncode == 0 and res.stdout.strip().endswith("ok"), \
            res.stdout[-3000:] + res.stderr[-3000:]
