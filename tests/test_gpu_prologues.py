"""GPU parity of the prologues of the two online-Hadamard sites (§4 Stage
1b: silu(gate) * up before the down-projection; §4 Stage 1c: the Hadamard
transform across heads before out_proj), through the C ABI, against the
CPU oracle.  Codes, scales and fp16 outputs must match bit for bit (the
fp16 tolerance of the other parity tests, max |err| <= 1e-2 max |oracle|,
is checked as well)."""
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


def test_swiglu_every_fp16_gate(dev, orc):
    """All 63488 finite fp16 gate values against three up values each."""
    import paper_2404_00456_amd as q
    h16 = np.arange(65536, dtype=np.uint32).astype(np.uint16).view(np.float16)
    g = h16[np.isfinite(h16)]
    g = g[: len(g) // 8 * 8]
    for up in (1.0, -0.7, 13.5):
        u = np.full_like(g, up)
        got = H(q.quarot_swiglu(T(g, dev), T(u, dev)))
        assert_same(got.view(np.uint16), orc.swiglu(g, u).view(np.uint16), f"swiglu up={up}")


def test_swiglu_random(dev, orc):
    import paper_2404_00456_amd as q
    rng = np.random.default_rng(2)
    g = (rng.standard_normal(1 << 20) * 4).astype(np.float16)
    u = (rng.standard_normal(1 << 20) * 3).astype(np.float16)
    got = H(q.quarot_swiglu(T(g, dev), T(u, dev)))
    assert_same(got.view(np.uint16), orc.swiglu(g, u).view(np.uint16), "swiglu random")


@pytest.mark.parametrize("n", [24, 40, 56, 128, 4096, 5120, 8192, 11008, 13824, 14336, 28672])
def test_swiglu_quant_int4(dev, orc, n):
    import paper_2404_00456_amd as q
    rows = 33 if n <= 8192 else 9
    say(f"swiglu_quant n={n} rows={rows}")
    g = workloads.random_rows(2 * n, rows, n, "normal", 3.0)
    u = workloads.random_rows(2 * n + 1, rows, n, "student_t3", 1.0)
    g[0] = -100.0      # silu underflows: an all-zero row
    g[1, :8] = 65504.0  # silu(g) = g
    u[1, :8] = 0.5
    for clip in (1.0, 0.9):
        codes, scale = q.quarot_swiglu_quant_int4(T(g, dev), T(u, dev), clip_ratio=clip)
        rq, rs = orc.swiglu_quant_int4(g, u, rotate=True, clip=clip)
        assert_same(H(codes), rq, f"swiglu codes n={n} clip={clip}")
        assert_same(H(scale).view(np.uint16), rs.view(np.uint16), f"swiglu scales n={n}")


def test_swiglu_quant_70b_down_rows(dev, orc):
    """The Llama-2-70B down-projection input width (28672 = 1024 x 28) on
    256 token rows, with the unfused chain (quarot_swiglu, then
    quarot_quant_int4) as a second GPU reference."""
    import paper_2404_00456_amd as q
    n, rows = 28672, 256
    g = workloads.random_rows(77, rows, n, "normal", 2.0)
    u = workloads.random_rows(78, rows, n, "normal", 1.0)
    gd, ud = T(g, dev), T(u, dev)
    codes, scale = q.quarot_swiglu_quant_int4(gd, ud)
    c2, s2 = q.quarot_quant_int4(q.quarot_swiglu(gd, ud), rotate=True)
    assert_same(H(codes), H(c2), "fused == unfused codes")
    assert_same(H(scale).view(np.uint16), H(s2).view(np.uint16), "fused == unfused scales")
    rq, rs = orc.swiglu_quant_int4(g, u, rotate=True, clip=1.0)
    assert_same(H(codes), rq, "swiglu 70b codes")
    assert_same(H(scale).view(np.uint16), rs.view(np.uint16), "swiglu 70b scales")


HEADS = [(2, 8), (8, 8), (4, 64), (32, 128), (64, 128), (8, 128), (128, 128),
         (64, 256), (256, 128), (16, 512), (2, 16384)]


@pytest.mark.parametrize("nh,dh", HEADS)
def test_hadamard_heads_fp16(dev, orc, nh, dh):
    import paper_2404_00456_amd as q
    n = nh * dh
    rows = 37 if n <= 8192 else 9
    z = workloads.random_rows(n + nh, rows, n, "student_t3")
    z[0] = 0
    z[1] = 0.5  # equal heads: all but head 0 cancel to +0
    y = H(q.quarot_hadamard_heads(T(z, dev), nh))
    assert_fp16_close(y, orc.hadamard_heads(z, nh), f"heads nh={nh} dh={dh}")


@pytest.mark.parametrize("nh,dh", HEADS)
def test_hadamard_heads_quant(dev, orc, nh, dh):
    import paper_2404_00456_amd as q
    n = nh * dh
    rows = 37 if n <= 8192 else 9
    z = workloads.random_rows(n + nh + 1, rows, n, "normal", 2.0)
    z[0] = 0
    for clip in (1.0, 0.9):
        codes, scale = q.quarot_hadamard_heads_quant_int4(T(z, dev), nh, clip_ratio=clip)
        rq, rs = orc.heads_quant_int4(z, nh, clip=clip)
        assert_same(H(codes), rq, f"heads codes nh={nh} dh={dh} clip={clip}")
        assert_same(H(scale).view(np.uint16), rs.view(np.uint16), f"heads scales nh={nh}")


def test_hadamard_heads_in_place_and_ragged_rows(dev, orc):
    import paper_2404_00456_amd as q
    nh, dh = 64, 128
    for rows in (1, 3, 255, 257):
        z = workloads.random_rows(rows, rows, nh * dh)
        zd = T(z, dev)
        q.quarot_hadamard_heads(zd, nh, y=zd)
        assert_fp16_close(H(zd), orc.hadamard_heads(z, nh), f"heads in place rows={rows}")
