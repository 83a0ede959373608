"""GPU parity of the e3m2 operand path of the W4A4 GEMM (§4 Stage 2b,
App. A.10): int4 codes stored as e3m2 numbers and multiplied by gfx950's
fp6 matrix instruction.  The packed bytes are decoded on the host from the
layout's definition and must give back every code; the GEMM's int32
accumulators and fp16 outputs must equal the oracle's bit for bit, and the
int4 path's on the full-size shapes."""
import numpy as np
import pytest

from test_gpu_parity import H, T, assert_fp16_close, assert_same, rand_codes, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_00456_amd as q
    q.lib()
    return torch.device("cuda:0")


def e3m2_value(c: int) -> float:
    """Value of a 6-bit e3m2 code: sign, 3 exponent bits (bias 3), 2 mantissa
    bits, subnormals at exponent field 0, no infinities or NaNs."""
    s = -1.0 if c & 0x20 else 1.0
    e, m = (c >> 2) & 7, c & 3
    if e == 0:
        return s * 2.0 ** -2 * (m / 4)
    return s * 2.0 ** (e - 3) * (1 + m / 4)


E3M2 = np.array([e3m2_value(c) for c in range(64)])


def decode_e3m2_layout(q6: np.ndarray, rows: int, k: int, sel=None) -> np.ndarray:
    """Tiled e3m2 layout [k/128, rows*96] -> code values [rows, k] (or of
    the rows listed in sel).  In block b, row r's unit u is the 192-bit
    little-endian word made of the 16-byte head at slot u ^ ((r >> 1) & 3)
    of the row's 64 bytes (heads of all rows first) and the 8-byte tail at
    slot u ^ ((r >> 2) & 3) of its 32 bytes (after the heads); code e sits
    at bits 6e..6e+5."""
    kb = k // 128
    buf = np.asarray(q6, np.uint8).reshape(kb, rows * 96)
    heads = buf[:, :rows * 64].reshape(kb, rows, 4, 16)
    tails = buf[:, rows * 64:].reshape(kb, rows, 4, 8)
    r = np.arange(rows) if sel is None else np.asarray(sel)
    out = np.empty((len(r), kb, 4, 32))
    for u in range(4):
        h = heads[:, r, u ^ ((r >> 1) & 3), :]
        t = tails[:, r, u ^ ((r >> 2) & 3), :]
        word = np.concatenate([h, t], axis=2)
        bits = np.unpackbits(word, axis=2, bitorder="little").reshape(kb, len(r), 32, 6)
        codes = bits.astype(np.int64) @ (1 << np.arange(6))
        out[:, :, u, :] = E3M2[codes].transpose(1, 0, 2)
    return out.reshape(len(r), k)


def test_e3m2_table_holds_int4():
    """Every int4 code is an e3m2 number (exactly one 6-bit code each, up to
    the sign of zero)."""
    for qv in range(-8, 8):
        hits = [c for c in range(64) if E3M2[c] == qv and not (qv == 0 and c & 0x20)]
        assert len(hits) == 1, qv


@pytest.mark.parametrize("rows,k", [(1, 128), (37, 384), (300, 8192), (5, 65536)])
def test_pack_e3m2_layout(dev, orc, rows, k):
    import paper_2404_00456_amd as q
    say(f"pack e3m2 rows={rows} k={k}")
    rng = np.random.default_rng(rows * 3 + k)
    q4 = rand_codes(rng, rows, k)
    q4[0, : min(8, k // 2)] = np.arange(0, 256, 32, dtype=np.uint8)[: min(8, k // 2)] | 0x08
    q6 = H(q.quarot_pack_e3m2(T(q4, dev)))
    assert q6.shape == (k // 128, rows * 96)
    assert_same(decode_e3m2_layout(q6, rows, k), orc.unpack_int4(q4).astype(np.float64),
                f"e3m2 layout rows={rows} k={k}")


def _gemm_case(dev, orc, M, N, K, xq, wq, sx, sw):
    import paper_2404_00456_amd as q
    x6 = q.quarot_pack_e3m2(T(xq, dev))
    w6 = q.quarot_pack_e3m2(T(wq, dev))
    y, acc = q.quarot_w4a4_gemm_e3m2(x6, T(sx, dev), w6, T(sw, dev), want_acc=True)
    y_only = q.quarot_w4a4_gemm_e3m2(x6, T(sx, dev), w6, T(sw, dev))
    racc = orc.gemm_i32(xq, wq)
    assert_same(H(acc), racc, f"e3m2 acc M={M} N={N} K={K}")
    ry = orc.dequant(racc, sx, sw)
    assert_fp16_close(H(y), ry, f"e3m2 y M={M} N={N} K={K}")
    assert_fp16_close(H(y_only), ry, f"e3m2 y (no acc) M={M} N={N} K={K}")


@pytest.mark.parametrize("M,N,K", [(1, 1, 128), (16, 256, 128), (255, 257, 384),
                                   (300, 520, 1024), (513, 100, 4096), (64, 1000, 11008),
                                   (256, 256, 28672), (2, 3, 65536),
                                   (2048, 8448, 128), (2048, 8448, 256), (2048, 8448, 384),
                                   (2304, 8448, 512), (2200, 8400, 1024),
                                   # whole 256 x 256 tiles and an even number of
                                   # k-steps (four 128 x 128 waves per block):
                                   # one tile, one per block, several per block
                                   (512, 512, 1024), (2048, 8192, 1280), (4096, 8192, 512),
                                   (8192, 4096, 768), (4352, 4352, 1536),
                                   # 128-row tiles with split k-steps: the
                                   # fewest pairs (K = 512), one row past a
                                   # tile, N not a multiple of 4, one column
                                   # of tiles
                                   (129, 300, 512), (1000, 36, 768), (640, 1030, 2048)])
def test_gemm_e3m2_exact(dev, orc, M, N, K):
    """Ragged edges, k-step counts below, at and above the LDS ring depth,
    blocks that walk several tiles, the largest K."""
    say(f"e3m2 gemm M={M} N={N} K={K}")
    rng = np.random.default_rng(M * 7 + N * 3 + K + 1)
    xq = rand_codes(rng, M, K)
    wq = rand_codes(rng, N, K)
    sx = rng.uniform(0.01, 2.0, M).astype(np.float16)
    sw = rng.uniform(0.0005, 0.05, N).astype(np.float16)
    _gemm_case(dev, orc, M, N, K, xq, wq, sx, sw)


def test_gemm_e3m2_extreme_codes(dev, orc):
    """All -8 codes at K = 65536: acc = 2^22, the largest magnitude, still an
    exact binary32 integer."""
    M, N, K = 40, 300, 65536
    xq = np.full((M, K // 2), 0x88, np.uint8)
    wq = np.full((N, K // 2), 0x88, np.uint8)
    sx = np.full(M, 0.001, np.float16)
    sw = np.full(N, 0.002, np.float16)
    _gemm_case(dev, orc, M, N, K, xq, wq, sx, sw)


def test_gemm_e3m2_tiny_scales(dev, orc):
    """Outputs across the fp16 subnormal range and underflow."""
    M, N, K = 512, 768, 2048
    rng = np.random.default_rng(12)
    xq = rand_codes(rng, M, K)
    wq = rand_codes(rng, N, K)
    sx = (2.0 ** rng.uniform(-24, -10, M)).astype(np.float16)
    sw = (2.0 ** rng.uniform(-14, -6, N)).astype(np.float16)
    _gemm_case(dev, orc, M, N, K, xq, wq, sx, sw)


@pytest.mark.parametrize("M,N,K", [(16384, 28672, 8192), (16384, 8192, 28672)])
def test_gemm_e3m2_full_size(dev, orc, M, N, K):
    """Llama-2-70B FFN shapes at prefill (16384 tokens), in the launch
    configuration the benchmark times: every output equal to the int4
    path's, and sampled rows equal to the oracle's."""
    import torch
    import paper_2404_00456_amd as q
    say(f"e3m2 gemm full size M={M} N={N} K={K}")
    g = torch.Generator(device=dev).manual_seed(M + N + K)
    xq = torch.randint(0, 256, (M, K // 2), generator=g, device=dev, dtype=torch.uint8)
    wq = torch.randint(0, 256, (N, K // 2), generator=g, device=dev, dtype=torch.uint8)
    sx = (torch.rand(M, generator=g, device=dev) * 0.05 + 0.01).half()
    sw = (torch.rand(N, generator=g, device=dev) * 0.002 + 0.0005).half()
    x6, w6 = q.quarot_pack_e3m2(xq), q.quarot_pack_e3m2(wq)
    for name, a4, a6 in (("X", xq, x6), ("W", wq, w6)):
        h4, h6 = H(a4), H(a6)
        assert_same(decode_e3m2_layout(h6, h4.shape[0], K), orc.unpack_int4(h4).astype(np.float64),
                    f"full size e3m2 layout {name}")
    y4 = q.quarot_w4a4_gemm(xq, sx, wq, sw)
    y6 = q.quarot_w4a4_gemm_e3m2(x6, sx, w6, sw)
    torch.cuda.synchronize()
    nd = int((y4.view(torch.int16) != y6.view(torch.int16)).sum().item())
    say(f"full size e3m2 vs int4: {nd} differing of {M * N}")
    assert nd == 0
    rows = np.array([0, 1, 255, 256, 8191, M - 1])
    xs, ss = H(xq[rows]), H(sx[rows])
    racc = orc.gemm_i32(xs, H(wq))
    ry = orc.dequant(racc, ss, H(sw))
    assert_same(H(y6[rows]).view(np.uint16), ry.view(np.uint16), "full size sampled rows")


@pytest.mark.parametrize("M,N,K", [(2048, 11008, 4096), (2048, 4096, 11008),
                                   # 128-row tiles with split k-steps, one or
                                   # two tiles per block, a ragged last column
                                   # of tiles
                                   (384, 33000, 512)])
def test_gemm_e3m2_7b_shapes(dev, orc, M, N, K):
    """Llama-2-7B FFN shapes at 2048 tokens, in the launch configuration the
    benchmark times, and a grid whose blocks walk two 128-row tiles with
    split k-steps: every acc and y equal to the int4 path's, and one seeded
    row of every 128-row tile, plus the first and last, equal to the
    oracle's, with and without the int32 output."""
    import torch
    import paper_2404_00456_amd as q
    say(f"e3m2 gemm 7B shape M={M} N={N} K={K}")
    g = torch.Generator(device=dev).manual_seed(M * 3 + N + K)
    xq = torch.randint(0, 256, (M, K // 2), generator=g, device=dev, dtype=torch.uint8)
    wq = torch.randint(0, 256, (N, K // 2), generator=g, device=dev, dtype=torch.uint8)
    sx = (torch.rand(M, generator=g, device=dev) * 0.05 + 0.01).half()
    sw = (torch.rand(N, generator=g, device=dev) * 0.002 + 0.0005).half()
    x6, w6 = q.quarot_pack_e3m2(xq), q.quarot_pack_e3m2(wq)
    y4, acc4 = q.quarot_w4a4_gemm(xq, sx, wq, sw, want_acc=True)
    y6, acc6 = q.quarot_w4a4_gemm_e3m2(x6, sx, w6, sw, want_acc=True)
    y6o = q.quarot_w4a4_gemm_e3m2(x6, sx, w6, sw)
    torch.cuda.synchronize()
    nd_acc = int((acc4 != acc6).sum().item())
    nd_y = int((y4.view(torch.int16) != y6.view(torch.int16)).sum().item())
    nd_yo = int((y4.view(torch.int16) != y6o.view(torch.int16)).sum().item())
    say(f"7B shape e3m2 vs int4: acc {nd_acc}, y {nd_y}, y (no acc) {nd_yo} differing of {M * N}")
    assert nd_acc == 0 and nd_y == 0 and nd_yo == 0
    rng = np.random.default_rng(M + N + K)
    rows = np.unique(np.concatenate([[0, M - 1], np.arange(0, M, 128) + rng.integers(0, 128, M // 128)]))
    xs, ss = H(xq[rows]), H(sx[rows])
    racc = orc.gemm_i32(xs, H(wq))
    assert_same(H(acc6[rows]), racc, "7B shape sampled acc")
    ry = orc.dequant(racc, ss, H(sw))
    assert_same(H(y6o[rows]).view(np.uint16), ry.view(np.uint16), "7B shape sampled rows")


@pytest.mark.parametrize("case", range(24))
def test_gemm_e3m2_random_grids(dev, orc, case):
    """Seeded random shapes with more than 128 rows and K a multiple of 256
    (the tile walks of both e3m2 kernels, one to three tiles per block,
    ragged edges): every acc and y equal to the int4 path's, with and
    without the int32 output, and two seeded rows equal to the oracle's."""
    import torch
    import paper_2404_00456_amd as q
    rng = np.random.default_rng(1000 + case)
    M = int(rng.integers(129, 4097))
    N = int(rng.integers(1, 8193))
    K = 256 * int(rng.integers(2, 33))
    say(f"e3m2 gemm random grid {case}: M={M} N={N} K={K}")
    g = torch.Generator(device=dev).manual_seed(case)
    xq = torch.randint(0, 256, (M, K // 2), generator=g, device=dev, dtype=torch.uint8)
    wq = torch.randint(0, 256, (N, K // 2), generator=g, device=dev, dtype=torch.uint8)
    sx = (torch.rand(M, generator=g, device=dev) * 0.05 + 0.001).half()
    sw = (torch.rand(N, generator=g, device=dev) * 0.01 + 0.0001).half()
    x6, w6 = q.quarot_pack_e3m2(xq), q.quarot_pack_e3m2(wq)
    y4, a4 = q.quarot_w4a4_gemm(xq, sx, wq, sw, want_acc=True)
    y6, a6 = q.quarot_w4a4_gemm_e3m2(x6, sx, w6, sw, want_acc=True)
    y6o = q.quarot_w4a4_gemm_e3m2(x6, sx, w6, sw)
    torch.cuda.synchronize()
    assert int((a4 != a6).sum().item()) == 0
    assert int((y4.view(torch.int16) != y6.view(torch.int16)).sum().item()) == 0
    assert int((y4.view(torch.int16) != y6o.view(torch.int16)).sum().item()) == 0
    rows = np.array(sorted({int(rng.integers(0, M)), M - 1}))
    racc = orc.gemm_i32(H(xq[rows]), H(wq))
    assert_same(H(a6[rows]), racc, "random grid sampled acc")
    ry = orc.dequant(racc, H(sx[rows]), H(sw))
    assert_same(H(y6o[rows]).view(np.uint16), ry.view(np.uint16), "random grid sampled rows")


# ------------------------------------------- quantizer writing e3m2 ---

E3M2_ROTATED_N = [128, 256, 1024, 4096, 8192, 16384, 32768, 12288, 24576, 10240, 20480, 14336,
                  28672, 3456, 6912, 13824, 5504, 11008]


@pytest.mark.parametrize("n", E3M2_ROTATED_N)
def test_quant_int4_e3m2_rotated(dev, orc, n):
    """Rotated rows quantized straight into the tiled e3m2 layout: every
    code (decoded on the host) and every scale equal to the oracle's, with
    clipping (the code -8 appears), an all-zero row and a spike."""
    import paper_2404_00456_amd as q
    import workloads
    rows = 37 if n <= 8192 else 9
    say(f"quant e3m2 rotate n={n} rows={rows}")
    x = workloads.random_rows(n + 5, rows, n, "student_t3", 2.0)
    x[0] = 0
    x[1, 0] = 100.0
    for clip in (1.0, 0.9):
        q6, s6 = q.quarot_quant_int4_e3m2(T(x, dev), rotate=True, clip_ratio=clip)
        rq, rs = orc.quant_int4(x, rotate=True, clip=clip)
        assert_same(decode_e3m2_layout(H(q6), rows, n), orc.unpack_int4(rq).astype(np.float64),
                    f"e3m2 codes n={n} clip={clip}")
        assert_same(H(s6).view(np.uint16), rs.view(np.uint16), f"e3m2 scales n={n} clip={clip}")


@pytest.mark.parametrize("n", [128, 384, 4096, 28672])
def test_quant_int4_e3m2_plain(dev, orc, n):
    import paper_2404_00456_amd as q
    import workloads
    rows = 13
    x = workloads.random_rows(3 * n + 1, rows, n, "student_t3")
    q6, s6 = q.quarot_quant_int4_e3m2(T(x, dev), rotate=False, clip_ratio=0.9)
    rq, rs = orc.quant_int4(x, rotate=False, clip=0.9)
    assert_same(decode_e3m2_layout(H(q6), rows, n), orc.unpack_int4(rq).astype(np.float64),
                f"e3m2 plain codes n={n}")
    assert_same(H(s6).view(np.uint16), rs.view(np.uint16), f"e3m2 plain scales n={n}")


@pytest.mark.parametrize("rows", [1, 3, 255, 257])
def test_quant_int4_e3m2_ragged_rows(dev, orc, rows):
    """Row counts across the 4-rows-per-block kernels (n = 128, 1024) and the
    row-per-block ones (n = 8192, 28672): the layout's row terms use the
    total row count."""
    import paper_2404_00456_amd as q
    import workloads
    for n in (128, 1024, 8192, 28672, 11008):
        x = workloads.random_rows(rows * 7 + n, rows, n)
        q6, s6 = q.quarot_quant_int4_e3m2(T(x, dev), rotate=True)
        rq, rs = orc.quant_int4(x, rotate=True)
        assert_same(decode_e3m2_layout(H(q6), rows, n), orc.unpack_int4(rq).astype(np.float64),
                    f"e3m2 codes n={n} rows={rows}")
        assert_same(H(s6).view(np.uint16), rs.view(np.uint16), f"e3m2 scales n={n} rows={rows}")


@pytest.mark.parametrize("n", [14336, 28672])
def test_swiglu_quant_e3m2(dev, orc, n):
    import paper_2404_00456_amd as q
    import workloads
    rows = 9
    g = workloads.random_rows(2 * n, rows, n, "normal", 3.0)
    u = workloads.random_rows(2 * n + 1, rows, n, "student_t3", 1.0)
    g[0] = -100.0
    for clip in (1.0, 0.9):
        q6, s6 = q.quarot_swiglu_quant_e3m2(T(g, dev), T(u, dev), clip_ratio=clip)
        rq, rs = orc.swiglu_quant_int4(g, u, rotate=True, clip=clip)
        assert_same(decode_e3m2_layout(H(q6), rows, n), orc.unpack_int4(rq).astype(np.float64),
                    f"swiglu e3m2 codes n={n} clip={clip}")
        assert_same(H(s6).view(np.uint16), rs.view(np.uint16), f"swiglu e3m2 scales n={n}")


@pytest.mark.parametrize("M,N,K", [(37, 300, 1024), (300, 520, 8192), (257, 264, 28672)])
def test_linear_e3m2(dev, orc, M, N, K):
    """The e3m2 linear layer equals quarot_linear bit for bit, and the
    oracle's layer within its defined arithmetic."""
    import paper_2404_00456_amd as q
    import workloads
    say(f"linear e3m2 M={M} N={N} K={K}")
    x = workloads.random_rows(M + K, M, K, "student_t3", 2.0)
    w = workloads.random_rows(N + 2 * K, N, K, "normal", 0.05)
    xd, wd = T(x, dev), T(w, dev)
    wq, sw = q.prepare_weight(wd, rotate=True)
    w6, sw6 = q.prepare_weight_e3m2(wd, rotate=True)
    assert_same(H(sw6).view(np.uint16), H(sw).view(np.uint16), "e3m2 weight scales")
    y4 = q.quarot_linear(xd, wq, sw, rotate=True, clip_ratio=0.9)
    y6 = q.quarot_linear_e3m2(xd, w6, sw6, rotate=True, clip_ratio=0.9)
    assert_same(H(y6).view(np.uint16), H(y4).view(np.uint16), "e3m2 linear == int4 linear")
    rq, rs = orc.quant_int4(x, rotate=True, clip=0.9)
    racc = orc.gemm_i32(rq, H(wq))
    ry = orc.dequant(racc, rs, H(sw))
    assert_fp16_close(H(y6), ry, f"e3m2 linear M={M} N={N} K={K}")
