"""GPU parity of the 6- and 8-bit variants (§5.3 RTN ablation, App. A.6)
through the C ABI against the CPU oracle: codes, scales and int32
accumulators bit for bit, fp16 outputs within max |err| <= 1e-2 max |oracle|
and bit for bit."""
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


@pytest.mark.parametrize("n", [8, 128, 4096, 8192, 24, 5120, 13824, 11008, 28672])
@pytest.mark.parametrize("bits", [6, 8])
def test_quant_int8_rotated(dev, orc, n, bits):
    import paper_2404_00456_amd as q
    rows = 21 if n <= 8192 else 7
    x = workloads.random_rows(n + bits, rows, n, "student_t3", 2.0)
    x[0] = 0
    for clip in (1.0, 0.9):
        codes, scale = q.quarot_quant_int8(T(x, dev), rotate=True, clip_ratio=clip, bits=bits)
        rq, rs = orc.quant_int8(x, rotate=True, clip=clip, bits=bits)
        assert_same(H(codes), rq, f"int{bits} codes n={n} clip={clip}")
        assert_same(H(scale).view(np.uint16), rs.view(np.uint16), f"int{bits} scales n={n}")


@pytest.mark.parametrize("n", [8, 200, 4096])
def test_quant_int8_plain(dev, orc, n):
    import paper_2404_00456_amd as q
    x = workloads.random_rows(n, 13, n, "normal", 5.0)
    codes, scale = q.quarot_quant_int8(T(x, dev), rotate=False, clip_ratio=0.9, bits=8)
    rq, rs = orc.quant_int8(x, rotate=False, clip=0.9, bits=8)
    assert_same(H(codes), rq, f"int8 plain codes n={n}")
    assert_same(H(scale).view(np.uint16), rs.view(np.uint16), f"int8 plain scales n={n}")


@pytest.mark.parametrize("M,N,K", [(1, 1, 64), (16, 256, 128), (255, 257, 192), (300, 520, 1024),
                                   (2048, 8448, 256), (2200, 8400, 1024), (64, 1000, 11008),
                                   (2, 3, 65536)])
def test_w8a8_gemm_exact(dev, orc, M, N, K):
    import paper_2404_00456_amd as q
    say(f"w8a8 gemm M={M} N={N} K={K}")
    rng = np.random.default_rng(M * 5 + N * 3 + K)
    xq = rng.integers(-128, 128, size=(M, K), dtype=np.int8)
    wq = rng.integers(-128, 128, size=(N, K), dtype=np.int8)
    sx = rng.uniform(0.001, 0.05, M).astype(np.float16)
    sw = rng.uniform(0.0005, 0.01, N).astype(np.float16)
    args = (T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev))
    y, acc = q.quarot_w8a8_gemm(*args, want_acc=True)
    y_only = q.quarot_w8a8_gemm(*args)
    racc = orc.gemm_i8(xq, wq)
    assert_same(H(acc), racc, f"w8a8 acc M={M} N={N} K={K}")
    ry = orc.dequant(racc, sx, sw)
    assert_fp16_close(H(y), ry, f"w8a8 y M={M} N={N} K={K}")
    assert_fp16_close(H(y_only), ry, f"w8a8 y (no acc) M={M} N={N} K={K}")


def test_w8a8_gemm_extreme(dev, orc):
    import paper_2404_00456_amd as q
    M, N, K = 40, 300, 65536
    xq = np.full((M, K), -128, np.int8)
    wq = np.full((N, K), -128, np.int8)
    wq[1] = 127
    sx = np.ones(M, np.float16)
    sw = np.full(N, 2.0 ** -24, np.float16)
    y, acc = q.quarot_w8a8_gemm(T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev), want_acc=True)
    racc = orc.gemm_i8(xq, wq)
    assert racc[0, 0] == 2 ** 30
    assert_same(H(acc), racc, "w8a8 extreme acc")
    assert_fp16_close(H(y), orc.dequant(racc, sx, sw), "w8a8 extreme y")


@pytest.mark.parametrize("name,rows,bits", [("llama2_7b_up", 64, 8), ("llama2_7b_down", 64, 6),
                                            ("llama2_70b_up", 16, 8)])
def test_linear_w8a8_layer(dev, orc, name, rows, bits):
    import paper_2404_00456_amd as q
    wl = workloads.LINEAR[name]
    x, w, _ = workloads.linear_inputs(wl, M=256)
    say(f"linear w8a8 {name} bits={bits}")
    wq_d, sw_d = q.quarot_quant_int8(T(w, dev), rotate=True, bits=bits)
    rwq, rsw = orc.quant_int8(w, rotate=True, clip=1.0, bits=bits)
    assert_same(H(wq_d), rwq, f"{name} int{bits} weight codes")
    y = H(q.quarot_linear_w8a8(T(x, dev), wq_d, sw_d, rotate=True, bits=bits))
    sel = np.arange(0, 256, 256 // rows)
    rxq, rsx = orc.quant_int8(x[sel], rotate=True, clip=1.0, bits=bits)
    ry = orc.dequant(orc.gemm_i8(rxq, rwq), rsx, rsw)
    assert_fp16_close(y[sel], ry, f"{name} int{bits} y")


@pytest.mark.parametrize("name", ["llama2_70b_up", "llama2_70b_down"])
def test_linear_w8a8_full_size(dev, orc, name):
    """The benchmarked W8A8 shapes (M = 16384), outputs sampled by row: a
    row of y depends on its own codes and scale only."""
    import paper_2404_00456_amd as q
    wl = workloads.LINEAR[name]
    say(f"linear w8a8 full size {name}: inputs M={wl.M} K={wl.K} N={wl.N}")
    x, w, _ = workloads.linear_inputs(wl)
    wq_d, sw_d = q.quarot_quant_int8(T(w, dev), rotate=True, bits=8)
    rwq, rsw = orc.quant_int8(w, rotate=True, clip=1.0, bits=8)
    assert_same(H(wq_d), rwq, f"{name} int8 weight codes")
    assert_same(H(sw_d).view(np.uint16), rsw.view(np.uint16), f"{name} int8 weight scales")
    del w
    y = H(q.quarot_linear_w8a8(T(x, dev), wq_d, sw_d, rotate=True, bits=8))
    rows = np.sort(np.random.default_rng(4).choice(wl.M, 12, replace=False))
    rows[0], rows[-1] = 0, wl.M - 1
    say(f"linear w8a8 full size {name}: oracle on {len(rows)} rows")
    rxq, rsx = orc.quant_int8(x[rows], rotate=True, clip=1.0, bits=8)
    ry = orc.dequant(orc.gemm_i8(rxq, rwq), rsx, rsw)
    assert_fp16_close(y[rows], ry, f"{name} int8 y rows")
