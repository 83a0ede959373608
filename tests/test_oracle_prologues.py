"""Pins for the oracle's prologues of the two online-Hadamard sites (§4
Stage 1b: silu(gate) * up before the down-projection; §4 Stage 1c: the
Hadamard transform across heads before out_proj).

Each test checks the oracle against mathematics it does not share code
with: fp64 exp, closed forms, scipy's Sylvester matrix with numpy integer
products, or the composition with oracle steps pinned elsewhere.
"""
import math

import numpy as np
import pytest
import scipy.linalg

import workloads

U32 = 2.0 ** -24


def all_f16():
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16).view(np.float16)
    return h[np.isfinite(h)]


def test_silu_within_4_ulp_of_fp64(orc):
    """Every finite fp16 input: the binary32 SiLU recipe lies within 4 ulps of
    g / (1 + exp(-g)) evaluated in fp64 (a wrong polynomial coefficient or a
    dropped LN2_LO term would miss by far more)."""
    g = all_f16().astype(np.float64)
    ref = g / (1.0 + np.exp(-np.clip(g, -700, 700)))
    got = np.array([orc.silu_f32(v) for v in g], np.float64)
    big = np.abs(ref) > 1e-30
    rel = np.abs(got[big] - ref[big]) / np.abs(ref[big])
    assert rel.max() <= 4 * U32, rel.max()
    # the far negative tail underflows to (signed) values far below fp16
    assert np.all(np.abs(got[~big]) < 1e-30)


def test_silu_closed_forms(orc):
    assert orc.silu_f32(0.0) == 0.0
    # exp(-g) < 2^-25 for g >= 18: 1 + E rounds to 1 and silu(g) = g exactly
    for g in (18.0, 24.0, 100.5, 65504.0):
        assert orc.silu_f32(g) == np.float32(g)
    # the recipe is odd-free but satisfies silu(g) - silu(-g) = g up to rounding
    for g in (0.5, 1.0, 3.0, 7.25):
        assert abs(float(orc.silu_f32(g)) - float(orc.silu_f32(-g)) - g) <= 4 * U32 * g


def test_swiglu_is_rn16_of_the_product(orc):
    """h = RN16(RN(silu(g) u)); against fp64 silu * u rounded to fp16 it may
    differ only where the binary32 product sits within a few ulps of an fp16
    rounding midpoint."""
    rng = np.random.default_rng(5)
    g = (rng.standard_normal(200000) * 3).astype(np.float16)
    u = (rng.standard_normal(200000) * 2).astype(np.float16)
    h = orc.swiglu(g, u).astype(np.float64)
    g64, u64 = g.astype(np.float64), u.astype(np.float64)
    exact = g64 / (1 + np.exp(-g64)) * u64
    ref = exact.astype(np.float16).astype(np.float64)
    diff = h != ref
    assert diff.mean() < 1e-3
    # where they differ, exact lies within 8 binary32 ulps of the midpoint
    mid = (h[diff] + ref[diff]) / 2
    assert np.all(np.abs(exact[diff] - mid) <= 8 * U32 * np.abs(exact[diff]))


@pytest.mark.parametrize("n,rotate", [(11008, True), (28672, True), (4096, True), (256, False)])
def test_swiglu_quant_is_quant_of_swiglu(orc, n, rotate):
    rows = 5
    g = workloads.random_rows(n, rows, n, "normal", 3.0)
    u = workloads.random_rows(n + 1, rows, n, "normal", 2.0)
    q, s = orc.swiglu_quant_int4(g, u, rotate=rotate, clip=1.0)
    q2, s2 = orc.quant_int4(orc.swiglu(g, u), rotate=rotate, clip=1.0)
    assert np.array_equal(q, q2) and np.array_equal(s.view(np.uint16), s2.view(np.uint16))


def kron_heads(nh, dh):
    return np.kron(scipy.linalg.hadamard(nh).astype(np.int64), np.eye(dh, dtype=np.int64))


@pytest.mark.parametrize("nh,dh", [(2, 8), (8, 16), (32, 128), (64, 128), (64, 8)])
def test_heads_unit_vectors(orc, nh, dh):
    """z = e_i gives c * (row i of H_nh (x) I_dh): pins the head-major layout,
    the stride d_h and every sign."""
    n = nh * dh
    idx = np.arange(n) if n <= 1024 else np.random.default_rng(n).choice(n, 300, replace=False)
    z = np.zeros((len(idx), n), np.float16)
    z[np.arange(len(idx)), idx] = 1
    y = orc.heads_f32(z, nh)
    c = np.float64(orc.rotation_scale(nh))
    ref = (kron_heads(nh, dh)[idx].astype(np.float64) * c).astype(np.float32)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("nh,dh", [(32, 128), (64, 128), (16, 64)])
def test_heads_exact_on_small_integers(orc, nh, dh):
    """Small-integer rows keep every butterfly exact, so y = RN32(c * z M)
    with the integer matrix M = H_nh (x) I_dh."""
    rng = np.random.default_rng(nh * dh)
    z = rng.integers(-200, 201, size=(6, nh * dh)).astype(np.int64)
    exact = z @ kron_heads(nh, dh)
    c = np.float64(orc.rotation_scale(nh))
    ref = (exact.astype(np.float64) * c).astype(np.float32)
    assert np.array_equal(orc.heads_f32(z.astype(np.float16), nh), ref)


def test_heads_then_dh_rotation_is_the_full_rotation(orc):
    """(H_nh (x) I)(I (x) H_dh) = H_nh (x) H_dh = H_n: on small integers, the
    head-wise transform of the exact per-head transform equals the full
    Walsh-Hadamard product of the rotation pinned elsewhere."""
    nh, dh = 16, 64
    rng = np.random.default_rng(3)
    z = rng.integers(-40, 41, size=(4, nh * dh)).astype(np.int64)
    per_head = z @ np.kron(np.eye(nh, dtype=np.int64), scipy.linalg.hadamard(dh).astype(np.int64))
    full_unscaled = orc.heads_f32(per_head.astype(np.float16), nh).astype(np.float64) / \
        np.float64(orc.rotation_scale(nh))
    n = nh * dh
    rot = orc.rotate_f16(z.astype(np.float16)).astype(np.float64) / np.float64(orc.rotation_scale(n))
    assert np.allclose(full_unscaled, rot, rtol=1e-6, atol=1e-6)


def test_heads_involution_and_norm(orc):
    nh, dh = 64, 128
    z = workloads.random_rows(9, 4, nh * dh, "student_t3")
    y = orc.heads_f32(z, nh)
    assert np.allclose(np.linalg.norm(y, axis=1),
                       np.linalg.norm(z.astype(np.float64), axis=1), rtol=1e-5)
    y2 = orc.heads_f32(y.astype(np.float16), nh).astype(np.float64)
    assert np.allclose(y2, z.astype(np.float64), atol=2e-3 * np.abs(z).max())


def test_heads_quant_is_quant_of_heads(orc):
    nh, dh = 64, 128
    z = workloads.random_rows(10, 7, nh * dh, "normal", 2.0)
    z[0] = 0
    for clip in (1.0, 0.9):
        q, s = orc.heads_quant_int4(z, nh, clip=clip)
        q2, s2 = orc.quant_sym_f32(orc.heads_f32(z, nh), clip=clip)
        assert np.array_equal(q, q2) and np.array_equal(s.view(np.uint16), s2.view(np.uint16))


def test_heads_zero_outputs_positive(orc):
    nh, dh = 8, 16
    z = np.zeros((3, nh * dh), np.float16)
    z[0] = -0.0
    z[1] = 0.5            # equal heads: every output but head 0 cancels
    y = orc.heads_f32(z, nh)
    assert not np.signbit(y[y == 0]).any()
    assert (y[1] != 0).sum() == dh
