"""The quantizer kernels form RN(y / s) with Markstein's correction from a
correctly rounded reciprocal (three operations instead of a division).
This checks the method itself on the CPU: for every positive finite fp16
divisor (the stored scales) the int4 and uint4 codes equal those from IEEE
division; quotients differ only where they underflow.  The same sequence
divides the KV group range by 15 exactly for every binary32 input."""
import ctypes
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def helper(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("mk") / "libmarkstein.so")
    # -mfma: a hardware fused multiply-add; -ffp-contract=off: nothing else fused
    subprocess.run(["gcc", "-O2", "-mfma", "-ffp-contract=off", "-fPIC", "-shared",
                    os.path.join(HERE, "native", "markstein_check.c"), "-o", out, "-lm"],
                   check=True)
    lib = ctypes.CDLL(out)
    lib.markstein_check.restype = ctypes.c_long
    lib.markstein_check.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_long),
                                    ctypes.POINTER(ctypes.c_double)]
    return lib


def test_markstein_codes_match_ieee_division(helper):
    qbad = ctypes.c_long()
    worst = ctypes.c_double()
    bad = helper.markstein_check(2000, ctypes.byref(qbad), ctypes.byref(worst))
    assert bad == 0
    # any quotient mismatch is an underflow case, far below a code boundary
    assert worst.value < 1e-30, worst.value


@pytest.fixture(scope="module")
def divconst(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("dc") / "libdivconst.so")
    subprocess.run(["gcc", "-O2", "-mfma", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    os.path.join(HERE, "native", "divconst_check.c"), "-o", out, "-lm"],
                   check=True)
    lib = ctypes.CDLL(out)
    lib.divconst_check.restype = ctypes.c_long
    lib.divconst_check.argtypes = [ctypes.c_float, ctypes.c_uint32, ctypes.c_uint32]
    return lib


@pytest.mark.parametrize("d", [15.0])
def test_division_by_constant_is_exact(divconst, d):
    """The KV group scale RN(RN(mx' - mn') / 15) is formed as
    fma(fma(-q0, 15, x), RN(1/15), q0) with q0 = RN(x RN(1/15)): equal to
    the IEEE quotient for every positive finite binary32 x (all 2^31 - 2^23
    of them; negative x mirror them)."""
    assert divconst.divconst_check(d, 1, 0x7F7FFFFF) == 0
