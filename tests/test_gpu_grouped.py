"""GPU parity of the group-wise W4A4 variant (§5.3 group-size ablation)
through the C ABI against the CPU oracle: group codes and group-major scales
bit for bit, and the grouped product's fp16 output bit for bit (each group's
integer dot product is exact, its dequant is two binary32 roundings and the
groups are summed in increasing order on both sides)."""
import numpy as np
import pytest

import workloads
from test_gpu_parity import H, T, assert_fp16_close, assert_same, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_00456_amd as q
    q.lib()
    return torch.device("cuda:0")


@pytest.mark.parametrize("n,group,rotate,rows", [
    (4096, 128, True, 67), (4096, 64, True, 40), (4096, 256, True, 33), (11008, 128, True, 19),
    (8192, 256, False, 50), (128, 8, True, 300), (512, 512, True, 9), (28672, 128, True, 5),
    (5120, 32, True, 17), (256, 16, False, 130),
    # multi-wave rows of m = 12, 20, 28 (binary32 rows staged through LDS)
    (6144, 128, True, 7), (24576, 256, True, 3), (20480, 128, True, 4), (14336, 64, True, 6)])
def test_group_quant(dev, orc, n, group, rotate, rows):
    import paper_2404_00456_amd as q
    say(f"group quant n={n} group={group} rotate={rotate} rows={rows}")
    x = workloads.random_rows(n + group + rows, rows, n, "student_t3")
    x[0] = 0           # an all-zero row: every group's scale is 0, codes 0
    x[1, :group] = 0   # one zero group in an otherwise normal row
    codes, scale = q.quarot_quant_int4_grouped(T(x, dev), group=group, rotate=rotate,
                                               clip_ratio=0.9)
    rq, rs = orc.quant_int4_grouped(x, group=group, rotate=rotate, clip=0.9)
    assert_same(H(codes), rq, "group codes")
    assert_same(H(scale).view(np.uint16), rs.view(np.uint16), "group scales")


def rand_group_case(seed, M, N, K, group):
    rng = np.random.default_rng(seed)
    xq = rng.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    wq = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    sx = rng.uniform(0.01, 2.0, (K // group, M)).astype(np.float16)
    sw = rng.uniform(0.0005, 0.05, (K // group, N)).astype(np.float16)
    return xq, sx, wq, sw


@pytest.mark.parametrize("M,N,K,group", [
    (1, 1, 128, 128), (16, 256, 128, 64), (255, 257, 256, 128), (300, 520, 1024, 256),
    (513, 100, 4096, 128), (64, 1000, 11008, 64), (64, 1000, 11008, 128),
    (40, 300, 11008, 256), (2, 3, 65536, 64), (7, 129, 65536, 256),
    # M, N multiples of 8 (the persistent ring kernel): ragged tiles, fewer
    # k-steps than ring stages (one tile per block), a single k-step
    (8, 8, 256, 256), (264, 136, 2048, 128), (1024, 1024, 256, 128), (520, 392, 128, 64),
    (24, 8192, 65536, 128), (16, 264, 65536, 256), (8, 136, 65536, 64)])
def test_gemm_grouped(dev, orc, M, N, K, group):
    import paper_2404_00456_amd as q
    say(f"grouped gemm M={M} N={N} K={K} group={group}")
    xq, sx, wq, sw = rand_group_case(M * 5 + N + K + group, M, N, K, group)
    y = q.quarot_w4a4_gemm_grouped(T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev), group=group)
    ry = orc.gemm_grouped(xq, sx, wq, sw, group=group)
    assert_fp16_close(H(y), ry, f"grouped y M={M} N={N} K={K} G={group}")


@pytest.mark.parametrize("M,N,K,group", [(2200, 8400, 1024, 128), (2048, 8448, 512, 64),
                                         (2304, 8448, 768, 256)])
def test_gemm_grouped_many_tiles(dev, orc, M, N, K, group):
    """More 256 x 128 tiles than one wave of blocks, ragged edges; the oracle
    on sampled rows (a row of y depends on its own codes and scales only)."""
    import paper_2404_00456_amd as q
    say(f"grouped gemm many tiles M={M} N={N} K={K} group={group}")
    xq, sx, wq, sw = rand_group_case(M + N + K, M, N, K, group)
    y = q.quarot_w4a4_gemm_grouped(T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev), group=group)
    rows = np.sort(np.random.default_rng(3).choice(M, 24, replace=False))
    rows[0], rows[-1] = 0, M - 1
    ry = orc.gemm_grouped(xq[rows], np.ascontiguousarray(sx[:, rows]), wq, sw, group=group)
    assert_fp16_close(H(y)[rows], ry, f"grouped y rows M={M} N={N} K={K} G={group}")


def test_gemm_grouped_extremes(dev, orc):
    """All -8 codes (|acc_g| = 64 G, the largest) and scales spanning fp16
    subnormals, so that group terms and sums underflow."""
    import paper_2404_00456_amd as q
    M, N, K, group = 300, 260, 4096, 256
    rng = np.random.default_rng(5)
    xq = np.full((M, K // 2), 0x88, np.uint8)
    wq = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    wq[0] = 0x88
    sx = (2.0 ** rng.uniform(-24, -14, (K // group, M))).astype(np.float16)
    sw = (2.0 ** rng.uniform(-14, -8, (K // group, N))).astype(np.float16)
    y = q.quarot_w4a4_gemm_grouped(T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev), group=group)
    ry = orc.gemm_grouped(xq, sx, wq, sw, group=group)
    assert (np.abs(ry.astype(np.float32)) < 2.0 ** -14).mean() > 0.05
    assert_fp16_close(H(y), ry, "grouped extremes")


# ---- the same product on e3m2 operands (quarot_pack_e3m2 of the codes) ----

def grouped_e3m2(q, dev, xq, sx, wq, sw, group):
    return q.quarot_w4a4_gemm_grouped_e3m2(q.quarot_pack_e3m2(T(xq, dev)), T(sx, dev),
                                           q.quarot_pack_e3m2(T(wq, dev)), T(sw, dev),
                                           group=group)


@pytest.mark.parametrize("M,N,K,group", [
    # one tile, a single k-step or one group of two (fewer k-steps than ring
    # stages: one tile per block)
    (8, 8, 128, 128), (8, 8, 256, 256), (8, 16, 384, 128),
    # ragged tiles in both directions, several groups
    (264, 136, 2048, 128), (264, 136, 2048, 256), (520, 392, 1280, 128),
    # 32 tiles with 2 / 3 / 4 k-steps
    (1024, 1024, 256, 128), (1024, 1024, 384, 128), (1024, 1024, 512, 256),
    # the largest K
    (24, 8192, 65536, 128), (16, 264, 65536, 256)])
def test_gemm_grouped_e3m2(dev, orc, M, N, K, group):
    import paper_2404_00456_amd as q
    say(f"grouped e3m2 gemm M={M} N={N} K={K} group={group}")
    xq, sx, wq, sw = rand_group_case(M * 7 + N + K + group, M, N, K, group)
    y = grouped_e3m2(q, dev, xq, sx, wq, sw, group)
    ry = orc.gemm_grouped(xq, sx, wq, sw, group=group)
    assert_fp16_close(H(y), ry, f"grouped e3m2 y M={M} N={N} K={K} G={group}")


@pytest.mark.parametrize("M,N,K,group", [(2200, 8400, 1024, 128), (2304, 8448, 768, 256),
                                         (4096, 4096, 2048, 128)])
def test_gemm_grouped_e3m2_many_tiles(dev, orc, M, N, K, group):
    """More 256 x 128 tiles than compute units (the persistent ring runs
    across tiles), ragged edges; the oracle on sampled rows, and every output
    against the int4-operand kernel."""
    import paper_2404_00456_amd as q
    say(f"grouped e3m2 gemm many tiles M={M} N={N} K={K} group={group}")
    xq, sx, wq, sw = rand_group_case(M + 3 * N + K, M, N, K, group)
    y = grouped_e3m2(q, dev, xq, sx, wq, sw, group)
    y4 = q.quarot_w4a4_gemm_grouped(T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev), group=group)
    rows = np.sort(np.random.default_rng(4).choice(M, 24, replace=False))
    rows[0], rows[-1] = 0, M - 1
    ry = orc.gemm_grouped(xq[rows], np.ascontiguousarray(sx[:, rows]), wq, sw, group=group)
    yh = H(y)
    assert_fp16_close(yh[rows], ry, f"grouped e3m2 y rows M={M} N={N} K={K} G={group}")
    assert_same(yh.view(np.uint16), H(y4).view(np.uint16), "e3m2 == int4 operands")


def test_gemm_grouped_e3m2_extremes(dev, orc):
    """All -8 codes (|acc_g| = 64 G, the largest) and scales spanning fp16
    subnormals."""
    import paper_2404_00456_amd as q
    M, N, K, group = 304, 264, 4096, 256
    rng = np.random.default_rng(6)
    xq = np.full((M, K // 2), 0x88, np.uint8)
    wq = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    wq[0] = 0x88
    sx = (2.0 ** rng.uniform(-24, -14, (K // group, M))).astype(np.float16)
    sw = (2.0 ** rng.uniform(-14, -8, (K // group, N))).astype(np.float16)
    y = grouped_e3m2(q, dev, xq, sx, wq, sw, group)
    ry = orc.gemm_grouped(xq, sx, wq, sw, group=group)
    assert (np.abs(ry.astype(np.float32)) < 2.0 ** -14).mean() > 0.05
    assert_fp16_close(H(y), ry, "grouped e3m2 extremes")


def test_gemm_grouped_e3m2_refusals(dev):
    import paper_2404_00456_amd as q
    xq, sx, wq, sw = rand_group_case(1, 16, 16, 256, 64)
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        grouped_e3m2(q, dev, xq, sx, wq, sw, 64)
    xq, sx, wq, sw = rand_group_case(1, 12, 16, 256, 128)
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        grouped_e3m2(q, dev, xq, sx, wq, sw, 128)


@pytest.mark.parametrize("name,group,sample", [("tiny", 64, None), ("llama2_7b_up", 128, 64),
                                               ("llama2_7b_down", 128, 48),
                                               ("llama2_7b_up", 256, 32),
                                               ("llama2_70b_up", 128, 12)])
def test_linear_grouped(dev, orc, name, group, sample):
    import paper_2404_00456_amd as q
    import torch
    wl = workloads.LINEAR[name]
    say(f"grouped linear {name} group={group}: inputs M={wl.M} K={wl.K} N={wl.N}")
    x, w, _ = workloads.linear_inputs(wl)
    wq_d, sw_d = q.quarot_quant_int4_grouped(T(w, dev), group=group, rotate=True)
    say(f"grouped linear {name}: oracle weight prep")
    rwq, rsw = orc.quant_int4_grouped(w, group=group, rotate=True)
    assert_same(H(wq_d), rwq, f"{name} weight codes")
    assert_same(H(sw_d).view(np.uint16), rsw.view(np.uint16), f"{name} weight scales")
    del w
    x_d = T(x, dev)
    y_d = q.quarot_linear_w4a4_grouped(x_d, wq_d, sw_d, group=group, rotate=True,
                                       clip_ratio=0.9)
    xq_d, sx_d = q.quarot_quant_int4_grouped(x_d, group=group, rotate=True, clip_ratio=0.9)
    y2_d = q.quarot_w4a4_gemm_grouped(xq_d, sx_d, wq_d, sw_d, group=group)
    torch.cuda.synchronize()
    rows = np.arange(wl.M) if sample is None else \
        np.sort(np.random.default_rng(2).choice(wl.M, sample, replace=False))
    rows[0], rows[-1] = 0, wl.M - 1
    say(f"grouped linear {name}: oracle on {len(rows)} rows")
    rxq, rsx = orc.quant_int4_grouped(x[rows], group=group, rotate=True, clip=0.9)
    assert_same(H(xq_d)[rows], rxq, f"{name} activation codes")
    assert_same(H(sx_d)[:, rows].view(np.uint16), rsx.view(np.uint16), f"{name} act scales")
    ry = orc.gemm_grouped(rxq, rsx, rwq, rsw, group=group)
    assert_fp16_close(H(y_d)[rows], ry, f"{name} grouped y")
    assert_same(H(y2_d)[rows].view(np.uint16), H(y_d)[rows].view(np.uint16),
                f"{name} linear == quant + gemm")
    if group >= 128 and wl.M % 8 == 0 and wl.N % 8 == 0:
        y6_d = q.quarot_w4a4_gemm_grouped_e3m2(q.quarot_pack_e3m2(xq_d), sx_d,
                                               q.quarot_pack_e3m2(wq_d), sw_d, group=group)
        assert_fp16_close(H(y6_d)[rows], ry, f"{name} grouped y, e3m2 operands")
        assert_same(H(y6_d).view(np.uint16), H(y_d).view(np.uint16),
                    f"{name} e3m2 == int4 operands")
