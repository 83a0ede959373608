"""Pins for the oracle's group-wise W4A4 (§5.3 group-wise ablation: a scale
per group of consecutive input channels for activations and weights): one
group per row reduces to the per-token path pinned elsewhere, each group is
that quantizer applied to the group's slice, and the product agrees with an
fp64 sum of per-group integer matmuls (numpy) within the binary32 rounding
of the group sum."""
import numpy as np
import pytest

import workloads


def test_one_group_is_per_token(orc):
    x = workloads.random_rows(4, 9, 1024, "student_t3")
    q, s = orc.quant_int4_grouped(x, group=1024)
    q2, s2 = orc.quant_int4(x)
    assert np.array_equal(q, q2) and np.array_equal(s[0].view(np.uint16), s2.view(np.uint16))


@pytest.mark.parametrize("G", [64, 128, 256])
def test_groups_are_slices(orc, G):
    x = workloads.random_rows(G, 5, 4096, "normal", 2.0)
    q, s = orc.quant_int4_grouped(x, group=G, rotate=True, clip=0.9)
    y = orc.rotate_f16(x)
    for g in range(4096 // G):
        qg, sg = orc.quant_sym_f32(np.ascontiguousarray(y[:, g * G:(g + 1) * G]), 0.9)
        assert np.array_equal(q[:, g * G // 2:(g + 1) * G // 2], qg)
        assert np.array_equal(s[g].view(np.uint16), sg.view(np.uint16))


def test_grouped_product(orc):
    M, N, K, G = 12, 17, 512, 128
    rng = np.random.default_rng(3)
    xq = rng.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    wq = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    sx = rng.uniform(0.01, 1, size=(K // G, M)).astype(np.float16)
    sw = rng.uniform(0.001, 0.05, size=(K // G, N)).astype(np.float16)
    y = orc.gemm_grouped(xq, sx, wq, sw, group=G).astype(np.float64)
    cx = orc.unpack_int4(xq).astype(np.int64)
    cw = orc.unpack_int4(wq).astype(np.int64)
    ref = np.zeros((M, N))
    for g in range(K // G):
        acc = cx[:, g * G:(g + 1) * G] @ cw[:, g * G:(g + 1) * G].T
        ref += acc * sx[g].astype(np.float64)[:, None] * sw[g].astype(np.float64)[None, :]
    bound = np.abs(ref) * 2.0 ** -10 + 8 * 2.0 ** -24 * np.abs(ref).max()
    assert np.all(np.abs(y - ref) <= bound)
    # one group equals the per-token dequant of the whole product
    y1 = orc.gemm_grouped(xq, sx[:1].repeat(1, 0), wq, sw[:1], group=K)
    assert np.array_equal(y1, orc.dequant(orc.gemm_i32(xq, wq), sx[0], sw[0]))
