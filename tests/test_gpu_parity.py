"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer outputs (packed int4 codes, scales' bits, int32 accumulators, KV
codes) must match bit for bit.  fp16 outputs must satisfy the stated
tolerance max |gpu - oracle| <= 1e-2 * max |oracle|, and, because the kernels
perform the oracle's IEEE operations in the oracle's order, they are also
required to match bit for bit (the number of differing elements is printed).
"""
import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.gpu

FP_TOL = 1e-2


def say(*a):
    print("[gpu-parity]", *a, flush=True)


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_00456_amd as q
    q.lib()
    return torch.device("cuda:0")


def T(a, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def H(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_fp16_close(got, ref, what):
    got = np.asarray(got, np.float16)
    ref = np.asarray(ref, np.float16)
    assert got.shape == ref.shape
    g = got.astype(np.float64)
    r = ref.astype(np.float64)
    amax = np.abs(r).max() if r.size else 0.0
    err = np.abs(g - r).max() if r.size else 0.0
    ndiff = int((got.view(np.uint16) != ref.view(np.uint16)).sum())
    say(f"{what}: max|err|={err:.3g} max|ref|={amax:.3g} differing={ndiff}/{ref.size}")
    assert err <= FP_TOL * amax + 1e-30, what
    # the kernels perform the oracle's IEEE operations in the oracle's order,
    # so any differing element is a deviation from the defined arithmetic
    assert ndiff == 0, f"{what}: {ndiff} elements differ from the oracle"


def assert_same(got, ref, what):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    nd = int((got != ref).sum())
    if nd:
        idx = np.argwhere(got != ref)[:5]
        say(f"{what}: {nd} mismatches, first at {idx.tolist()}")
    assert nd == 0, what


# ----------------------------------------------------------- rotation ---

ROT_SIZES = [8, 64, 128, 512, 1024, 4096, 8192, 16384, 32768,     # m = 1
             24, 96, 3072, 6144, 24576,                             # m = 12
             40, 5120, 20480,                                       # m = 20
             56, 448, 3584, 7168, 14336, 28672,                     # m = 28
             216, 13824,                                            # m = 108
             344, 5504, 11008]                                      # m = 172


@pytest.mark.parametrize("n", ROT_SIZES)
def test_hadamard_fp16(dev, orc, n):
    import paper_2404_00456_amd as q
    rows = 37 if n <= 8192 else 9
    say(f"hadamard n={n} rows={rows}")
    x = workloads.random_rows(n, rows, n, "student_t3")
    y = H(q.quarot_hadamard(T(x, dev)))
    assert_fp16_close(y, orc.hadamard(x), f"hadamard n={n}")


@pytest.mark.parametrize("n", [8192, 28672, 11008])
def test_hadamard_fp16_many_rows(dev, orc, n):
    """The standalone rotation over 2048 rows (every block of the grid busy
    several times over): seeded sampled rows equal to the oracle's, the
    first and last included."""
    import paper_2404_00456_amd as q
    rows = 2048
    say(f"hadamard many rows n={n} rows={rows}")
    x = workloads.random_rows(n + 11, rows, n, "normal")
    y = H(q.quarot_hadamard(T(x, dev)))
    rng = np.random.default_rng(n)
    sel = np.unique(np.concatenate([[0, rows - 1], rng.integers(0, rows, 10)]))
    assert_fp16_close(y[sel], orc.hadamard(x[sel]), f"hadamard many rows n={n}")


@pytest.mark.parametrize("n", [8, 128, 1024, 8192, 32768, 24, 3072, 5120, 28672, 216, 11008])
def test_hadamard_in_place(dev, orc, n):
    """x == y is allowed: every kernel family (power of two, exact small m,
    fp64 large m) reads a row whole before writing it."""
    import paper_2404_00456_amd as q
    rows = 261 if n <= 1024 else 7
    say(f"hadamard in place n={n} rows={rows}")
    x = workloads.random_rows(n + 5, rows, n, "normal")
    xd = T(x, dev)
    q.quarot_hadamard(xd, y=xd)
    assert_fp16_close(H(xd), orc.hadamard(x), f"hadamard in place n={n}")


@pytest.mark.parametrize("n", ROT_SIZES)
def test_quant_int4_rotated(dev, orc, n):
    import paper_2404_00456_amd as q
    rows = 37 if n <= 8192 else 9
    say(f"quant_int4 rotate n={n} rows={rows}")
    x = workloads.random_rows(n + 1, rows, n, "normal", scale=3.0)
    x[0] = 0            # all-zero row -> scale 0, codes 0
    x[1, 0] = 100.0     # single spike
    codes, scale = q.quarot_quant_int4(T(x, dev), rotate=True, clip_ratio=1.0)
    rq, rs = orc.quant_int4(x, rotate=True, clip=1.0)
    assert_same(H(codes), rq, f"codes n={n}")
    assert_same(H(scale).view(np.uint16), rs.view(np.uint16), f"scales n={n}")


@pytest.mark.parametrize("n,clip", [(4096, 0.9), (11008, 0.9), (28672, 0.9), (128, 0.5)])
def test_quant_int4_clip(dev, orc, n, clip):
    import paper_2404_00456_amd as q
    x = workloads.random_rows(7 * n, 21, n, "student_t3")
    codes, scale = q.quarot_quant_int4(T(x, dev), rotate=True, clip_ratio=clip)
    rq, rs = orc.quant_int4(x, rotate=True, clip=clip)
    assert_same(H(codes), rq, f"codes n={n} clip={clip}")
    assert_same(H(scale).view(np.uint16), rs.view(np.uint16), f"scales n={n} clip={clip}")
    # with clip < 1 the code -8 appears
    assert (orc.unpack_int4(rq) == -8).any()


@pytest.mark.parametrize("n", [8, 200, 4096, 11008, 28672])
def test_quant_int4_plain(dev, orc, n):
    import paper_2404_00456_amd as q
    x = workloads.random_rows(3 * n, 13, n, "student_t3")
    # exact ties: row of k/2 values with amax 7 -> scale 1
    if n >= 16:
        x[2, :16] = np.array([7, 2.5, -2.5, 3.5, 0.5, 1.5, -1.5, -3.5, -0.5, 6.5, 5.5, 4.5,
                              0, 0, 0, 0], np.float16)
        x[2, 16:] = 0
    codes, scale = q.quarot_quant_int4(T(x, dev), rotate=False, clip_ratio=1.0)
    rq, rs = orc.quant_int4(x, rotate=False, clip=1.0)
    assert_same(H(codes), rq, f"plain codes n={n}")
    assert_same(H(scale).view(np.uint16), rs.view(np.uint16), f"plain scales n={n}")


def test_quant_ragged_rows(dev, orc):
    """Row counts that leave partial blocks (rows per block 4..256)."""
    import paper_2404_00456_amd as q
    for n in (8, 64, 128, 4096, 56):
        for rows in (1, 3, 255, 257):
            x = workloads.random_rows(rows + n, rows, n)
            codes, scale = q.quarot_quant_int4(T(x, dev), rotate=True)
            rq, rs = orc.quant_int4(x, rotate=True)
            assert_same(H(codes), rq, f"codes n={n} rows={rows}")
            assert_same(H(scale).view(np.uint16), rs.view(np.uint16), f"s n={n} rows={rows}")


# --------------------------------------------------------------- GEMM ---

def rand_codes(rng, rows, K):
    return rng.integers(0, 256, size=(rows, K // 2), dtype=np.uint8)


@pytest.mark.parametrize("M,N,K", [(1, 1, 64), (16, 256, 128), (255, 257, 192),
                                   (300, 520, 1024), (513, 100, 4096), (64, 1000, 11008),
                                   (256, 256, 28672), (2, 3, 65536)])
def test_gemm_exact(dev, orc, M, N, K):
    import paper_2404_00456_amd as q
    say(f"gemm M={M} N={N} K={K}")
    rng = np.random.default_rng(M * 7 + N * 3 + K)
    xq = rand_codes(rng, M, K)
    wq = rand_codes(rng, N, K)
    sx = rng.uniform(0.01, 2.0, M).astype(np.float16)
    sw = rng.uniform(0.0005, 0.05, N).astype(np.float16)
    args = (T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev))
    y, acc = q.quarot_w4a4_gemm(*args, want_acc=True)
    y_only = q.quarot_w4a4_gemm(*args)  # no int32 output: the fast epilogue on full tiles
    racc = orc.gemm_i32(xq, wq)
    assert_same(H(acc), racc, f"acc M={M} N={N} K={K}")
    ry = orc.dequant(racc, sx, sw)
    assert_fp16_close(H(y), ry, f"y M={M} N={N} K={K}")
    assert_fp16_close(H(y_only), ry, f"y (no acc) M={M} N={N} K={K}")


@pytest.mark.parametrize("M,N,K", [(2048, 8448, 128), (2048, 8448, 256), (2048, 8448, 384),
                                   (2048, 8448, 640), (2304, 8448, 512), (2200, 8400, 1024)])
def test_gemm_many_tiles(dev, orc, M, N, K):
    """More 256 x 256 tiles than one wave of blocks (264 and 297 tiles), so
    that blocks walk several tiles: k-step counts below, at and above the
    LDS ring depth, tile counts with and without a multiple of 8, ragged
    edges."""
    import paper_2404_00456_amd as q
    say(f"gemm many tiles M={M} N={N} K={K}")
    rng = np.random.default_rng(M + N + K)
    xq = rand_codes(rng, M, K)
    wq = rand_codes(rng, N, K)
    sx = rng.uniform(0.01, 2.0, M).astype(np.float16)
    sw = rng.uniform(0.0005, 0.05, N).astype(np.float16)
    args = (T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev))
    y, acc = q.quarot_w4a4_gemm(*args, want_acc=True)
    y_only = q.quarot_w4a4_gemm(*args)  # no int32 output: the fast epilogue on full tiles
    racc = orc.gemm_i32(xq, wq)
    assert_same(H(acc), racc, f"acc M={M} N={N} K={K}")
    ry = orc.dequant(racc, sx, sw)
    assert_fp16_close(H(y), ry, f"y M={M} N={N} K={K}")
    assert_fp16_close(H(y_only), ry, f"y (no acc) M={M} N={N} K={K}")


def test_gemm_tiny_scales(dev, orc):
    """Scales down to fp16 subnormals, so that y spans the fp16 subnormal
    range and underflows to zero: the conversions of both epilogues (full
    tiles without int32 output, and the general one) against the oracle."""
    import paper_2404_00456_amd as q
    M, N, K = 512, 768, 2048
    rng = np.random.default_rng(11)
    xq = rand_codes(rng, M, K)
    wq = rand_codes(rng, N, K)
    sx = (2.0 ** rng.uniform(-24, -10, M)).astype(np.float16)
    sw = (2.0 ** rng.uniform(-14, -6, N)).astype(np.float16)
    args = (T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev))
    y, acc = q.quarot_w4a4_gemm(*args, want_acc=True)
    y_only = q.quarot_w4a4_gemm(*args)
    racc = orc.gemm_i32(xq, wq)
    ry = orc.dequant(racc, sx, sw)
    sub = np.abs(ry.astype(np.float32)) < 2.0 ** -14
    assert sub.mean() > 0.2 and (ry == 0).any()  # the case is exercised
    assert_same(H(acc), racc, "tiny-scale acc")
    assert_fp16_close(H(y), ry, "tiny-scale y")
    assert_fp16_close(H(y_only), ry, "tiny-scale y (no acc)")


def test_gemm_extreme_codes(dev, orc):
    """All -8 codes: |acc| = 64 K, the largest magnitude (K = 65536: 2^22)."""
    import paper_2404_00456_amd as q
    M, N, K = 40, 300, 65536
    xq = np.full((M, K // 2), 0x88, np.uint8)
    wq = np.full((N, K // 2), 0x88, np.uint8)
    wq[1] = 0x77  # +7
    sx = np.ones(M, np.float16)
    sw = np.full(N, 2.0 ** -14, np.float16)
    y, acc = q.quarot_w4a4_gemm(T(xq, dev), T(sx, dev), T(wq, dev), T(sw, dev), want_acc=True)
    racc = orc.gemm_i32(xq, wq)
    assert racc[0, 0] == 64 * K and racc[0, 1] == -56 * K
    assert_same(H(acc), racc, "extreme acc")
    assert_fp16_close(H(y), orc.dequant(racc, sx, sw), "extreme y")


# ------------------------------------------------------ whole layer -----

def _layer_case(dev, orc, name, sample_rows):
    import paper_2404_00456_amd as q
    import torch
    wl = workloads.LINEAR[name]
    say(f"{name}: generating inputs M={wl.M} K={wl.K} N={wl.N}")
    x, w, _ = workloads.linear_inputs(wl)
    say(f"{name}: oracle weight prep")
    rwq, rsw = orc.prepare_weight(w, rotate=True)
    say(f"{name}: gpu weight prep")
    wq_d, sw_d = q.prepare_weight(T(w, dev), rotate=True)
    assert_same(H(wq_d), rwq, f"{name} weight codes")
    assert_same(H(sw_d).view(np.uint16), rsw.view(np.uint16), f"{name} weight scales")
    del w
    x_d = T(x, dev)
    say(f"{name}: gpu quarot_linear")
    y_d = q.quarot_linear(x_d, wq_d, sw_d, rotate=True, clip_ratio=1.0)
    xq_d, sx_d = q.quarot_quant_int4(x_d, rotate=True)
    y2_d, acc_d = q.quarot_w4a4_gemm(xq_d, sx_d, wq_d, sw_d, want_acc=True)
    torch.cuda.synchronize()
    if sample_rows is None:
        rows = np.arange(wl.M)
    else:
        rows = np.sort(np.random.default_rng(1).choice(wl.M, sample_rows, replace=False))
        rows[0] = 0
        rows[-1] = wl.M - 1
    say(f"{name}: oracle on {len(rows)} rows")
    xs = x[rows]
    rxq, rsx = orc.quant_int4(xs, rotate=True)
    assert_same(H(xq_d)[rows], rxq, f"{name} activation codes")
    assert_same(H(sx_d)[rows].view(np.uint16), rsx.view(np.uint16), f"{name} act scales")
    ry, racc = orc.linear(xs, rwq, rsw, rotate=True, want_acc=True)
    assert_same(H(acc_d)[rows], racc, f"{name} int32 acc")
    assert_fp16_close(H(y_d)[rows], ry, f"{name} y (quarot_linear)")
    assert_same(H(y2_d)[rows].view(np.uint16), H(y_d)[rows].view(np.uint16),
                f"{name} linear == quant + gemm")


def test_layer_tiny(dev, orc):
    _layer_case(dev, orc, "tiny", None)


# the full-size layer shapes: tests/test_gpu_fullsize.py


# ----------------------------------------------------------------- KV ---

@pytest.mark.parametrize("D,G,rotate", [(128, 128, True), (128, 32, True), (64, 64, True),
                                        (256, 128, True), (128, 128, False), (8, 8, True),
                                        (512, 64, True), (16, 8, False)])
def test_kv_quant_dequant(dev, orc, D, G, rotate):
    import paper_2404_00456_amd as q
    rng = np.random.default_rng(D + G)
    rows = 1000 + D
    x = (rng.standard_normal((rows, D)) * 2).astype(np.float16)
    x[3] = 0.25  # constant row: zero scale
    say(f"kv D={D} G={G} rotate={rotate}")
    cq, sc, ze = q.quarot_kv_quant(T(x, dev), group=G, rotate=rotate, clip_ratio=0.95)
    rq, rs, rz = orc.kv_quant(x, group=G, rotate=rotate, clip=0.95)
    assert_same(H(cq), rq, "kv codes")
    assert_same(H(sc).view(np.uint16), rs.view(np.uint16), "kv scales")
    assert_same(H(ze).view(np.uint16), rz.view(np.uint16), "kv zeros")
    for inv in ((False, True) if rotate else (False,)):
        out = q.quarot_kv_dequant(T(rq, dev), T(rs, dev), T(rz, dev), group=G,
                                  inverse_rotate=inv)
        assert_fp16_close(H(out), orc.kv_dequant(rq, rs, rz, group=G, inverse_rotate=inv),
                          f"kv dequant D={D} G={G} inv={inv}")


def assert_fp16_bits(got, ref, what):
    """Bit-for-bit fp16 equality for large arrays (no float64 copies);
    differing elements, if any, are reported against the fp tolerance."""
    gb, rb = np.asarray(got).view(np.uint16), np.asarray(ref).view(np.uint16)
    assert gb.shape == rb.shape, what
    bad = np.flatnonzero(gb.reshape(-1) != rb.reshape(-1))
    say(f"{what}: differing={bad.size}/{rb.size}")
    if bad.size:
        g = got.reshape(-1)[bad].astype(np.float64)
        r = ref.reshape(-1)[bad].astype(np.float64)
        say(f"{what}: max|err| on those {np.abs(g - r).max():.3g}")
    assert bad.size == 0, what


def test_kv_config_70b_heads(dev, orc):
    """The whole 4-bit KV workload the benchmark times: K and V fp16
    [16, 64, 4096, 128] (4 Mi head rows each), H_128 per row, asymmetric
    uint4 in groups of 128 with clip 0.95.  Codes, scales and zeros bit for
    bit; the dequantized cache bit for bit in the rotated basis (the
    benchmark's call) and rotated back."""
    import paper_2404_00456_amd as q
    import torch
    wl = workloads.KV["kv4_70b"]
    k, v = workloads.kv_inputs(wl)
    assert k.shape == (16, 64, 4096, 128)
    for name, t in (("K", k), ("V", v)):
        x = t.reshape(-1, wl.D)
        say(f"kv4 {name}: rows={x.shape[0]}")
        cq, sc, ze = q.quarot_kv_quant(T(x, dev), group=wl.group, rotate=True, clip_ratio=wl.clip)
        rq, rs, rz = orc.kv_quant(x, group=wl.group, rotate=True, clip=wl.clip)
        assert_same(H(cq), rq, f"kv4 {name} codes")
        assert_same(H(sc).view(np.uint16), rs.view(np.uint16), f"kv4 {name} scales")
        assert_same(H(ze).view(np.uint16), rz.view(np.uint16), f"kv4 {name} zeros")
        for inv in (False, True):
            out = q.quarot_kv_dequant(cq, sc, ze, group=wl.group, inverse_rotate=inv)
            assert_fp16_bits(H(out), orc.kv_dequant(rq, rs, rz, group=wl.group,
                                                    inverse_rotate=inv),
                             f"kv4 {name} dequant inverse_rotate={inv}")
            del out
        del cq, sc, ze, rq, rs, rz
        torch.cuda.empty_cache()


def test_deterministic(dev):
    import paper_2404_00456_amd as q
    x = workloads.random_rows(5, 300, 11008, "student_t3")
    xd = T(x, dev)
    a = [H(q.quarot_quant_int4(xd, rotate=True)[0]) for _ in range(3)]
    assert all(np.array_equal(a[0], b) for b in a[1:])
