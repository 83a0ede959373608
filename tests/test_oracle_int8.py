"""Pins for the oracle's 6- and 8-bit variants (§5.3 RTN ablation and App.
A.6: the same symmetric scheme with 2^(bits-1) - 1 levels a side, one code
per byte): closed forms at power-of-two scales, ties to even, exact-rational
brute force of the nearest code, error bounds, composition with the
rotation, and the int8 GEMM against numpy's int64 matmul."""
from fractions import Fraction

import numpy as np
import pytest

import workloads


@pytest.mark.parametrize("bits", [6, 8])
def test_closed_form_power_of_two_scale(orc, bits):
    """y = k * 2^e with max |k| = qmax: scale 2^e exactly, codes k."""
    qmax = (1 << (bits - 1)) - 1
    rng = np.random.default_rng(bits)
    k = rng.integers(-qmax, qmax + 1, size=(6, 64))
    k[:, 0] = qmax
    e = rng.integers(-10, 6, size=(6, 1)).astype(np.float64)
    y = (k * 2.0 ** e).astype(np.float32)
    q, s = orc.quant_sym8_f32(y, 1.0, bits)
    assert np.array_equal(s.astype(np.float64), 2.0 ** e[:, 0])
    assert np.array_equal(q.astype(np.int64), k)


@pytest.mark.parametrize("bits", [6, 8])
def test_ties_to_even(orc, bits):
    qmax = (1 << (bits - 1)) - 1
    y = np.array([[qmax, 2.5, -2.5, 3.5, 0.5, -0.5, 1.5, qmax - 0.5]], np.float32)
    q, s = orc.quant_sym8_f32(y, 1.0, bits)
    assert float(s[0]) == 1.0
    assert q[0].tolist() == [qmax, 2, -2, 4, 0, 0, 2, qmax - 1 if (qmax - 1) % 2 == 0 else qmax]


@pytest.mark.parametrize("bits", [6, 8])
def test_brute_force_nearest_code(orc, bits):
    """Each code is the nearest integer in [-qmax-1, qmax] to y / s16
    (exact rationals), up to the one rounding of the binary32 quotient."""
    qmax = (1 << (bits - 1)) - 1
    rng = np.random.default_rng(10 + bits)
    y = (rng.standard_normal((20, 48)) * rng.uniform(0.01, 100, size=(20, 1))).astype(np.float32)
    for clip in (1.0, 0.9):
        q, s = orc.quant_sym8_f32(y, clip, bits)
        for r in range(y.shape[0]):
            sf = Fraction(float(s[r]))
            amax = max(abs(Fraction(float(v))) for v in y[r])
            assert abs(sf - amax * Fraction(float(np.float32(clip))) / qmax) <= \
                sf * Fraction(1, 1024) + amax * Fraction(1, 2 ** 22)
            for j in range(y.shape[1]):
                ratio = Fraction(float(y[r, j])) / sf
                best = min(range(-qmax - 1, qmax + 1), key=lambda c: (abs(ratio - c), c % 2))
                if q[r, j] != best:
                    half = Fraction(2 * best + (1 if q[r, j] > best else -1), 2)
                    assert abs(ratio - half) <= abs(ratio) * Fraction(1, 2 ** 23)
            if clip == 1.0:
                assert q[r].min() >= -qmax


@pytest.mark.parametrize("bits", [6, 8])
def test_zero_rows_and_error_bound(orc, bits):
    y = np.zeros((2, 16), np.float32)
    y[1, 3] = 1e-30
    q, s = orc.quant_sym8_f32(y, 1.0, bits)
    assert np.all(s == 0) and np.all(q == 0)
    x = workloads.random_rows(19, 16, 256, "student_t3")
    q, s = orc.quant_int8(x, rotate=False, clip=1.0, bits=bits)
    err = np.abs(x.astype(np.float64) - q.astype(np.float64) * s.astype(np.float64)[:, None])
    assert np.all(err <= s.astype(np.float64)[:, None] / 2 * (1 + 2.0 ** -10))


@pytest.mark.parametrize("n,bits", [(4096, 8), (11008, 6), (28672, 8), (56, 8)])
def test_quant_int8_rotate_composes(orc, n, bits):
    x = workloads.random_rows(n + bits, 3, n)
    for clip in (1.0, 0.9):
        q, s = orc.quant_int8(x, rotate=True, clip=clip, bits=bits)
        q2, s2 = orc.quant_sym8_f32(orc.rotate_f16(x), clip, bits)
        assert np.array_equal(q, q2) and np.array_equal(s.view(np.uint16), s2.view(np.uint16))


def test_more_bits_smaller_error(orc):
    """The 8-bit codes reconstruct the rotated rows far better than 4-bit."""
    x = workloads.random_rows(3, 8, 4096, "student_t3")
    y = orc.rotate_f16(x).astype(np.float64)
    q8, s8 = orc.quant_int8(x, bits=8)
    q4, s4 = orc.quant_int4(x)
    e8 = np.linalg.norm(y - q8 * s8.astype(np.float64)[:, None])
    e4 = np.linalg.norm(y - orc.unpack_int4(q4) * s4.astype(np.float64)[:, None])
    assert e8 < e4 / 8


def test_gemm_i8_vs_numpy(orc):
    rng = np.random.default_rng(7)
    xq = rng.integers(-128, 128, size=(33, 320), dtype=np.int8)
    wq = rng.integers(-128, 128, size=(45, 320), dtype=np.int8)
    acc = orc.gemm_i8(xq, wq)
    assert np.array_equal(acc, xq.astype(np.int64) @ wq.astype(np.int64).T)
    ext = orc.gemm_i8(np.full((1, 4096), -128, np.int8), np.full((2, 4096), -128, np.int8))
    assert ext[0, 0] == 128 * 128 * 4096
