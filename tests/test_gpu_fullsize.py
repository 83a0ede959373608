"""Full-size parity of the timed pipeline (App. A.10 4-bit linear layer on
the Llama-2 layer shapes; §4 Stage 1b/2b): the benchmark's own inputs,
weight preparation and launches, checked against the CPU oracle.

For every layer shape: the prepared weights (codes and scales of every
output channel) bit for bit; then, on the e3m2 path the benchmark times
(quarot_quant_int4_e3m2 + quarot_w4a4_gemm_e3m2) and on the int4 path
(quarot_quant_int4 + quarot_w4a4_gemm), and through both fused layer calls,
a seeded sample of token rows holding at least one row of every 256-row
tile of the GEMM (all N columns): activation codes (decoded from the e3m2
layout), scales, int32 accumulators and fp16 outputs bit for bit against
the oracle's quantizer, integer product and dequant.  All outputs of the
two GEMM paths are also compared with each other."""
import numpy as np
import pytest

import workloads
from test_gpu_e3m2 import decode_e3m2_layout
from test_gpu_parity import H, T, assert_same, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_00456_amd as q
    q.lib()
    return torch.device("cuda:0")


def sample_rows(M, per_tile, seed):
    """per_tile seeded rows from every 256-row tile, plus the first and last."""
    rng = np.random.default_rng(seed)
    rows = [t * 256 + int(r) for t in range((M + 255) // 256)
            for r in rng.choice(min(256, M - t * 256), per_tile, replace=False)]
    return np.unique(np.array(rows + [0, M - 1]))


@pytest.mark.parametrize("name,per_tile", [("llama2_70b_up", 1), ("llama2_70b_down", 1),
                                           ("llama2_7b_up", 8), ("llama2_7b_down", 8)])
def test_pipeline_full_size(dev, orc, name, per_tile):
    import torch
    import paper_2404_00456_amd as q
    wl = workloads.LINEAR[name]
    M, N, K = wl.M, wl.N, wl.K
    say(f"{name}: inputs M={M} K={K} N={N}")
    x, w, _ = workloads.linear_inputs(wl)
    say(f"{name}: weight prep (gpu, oracle)")
    wd = T(w, dev)
    wq, sw = q.prepare_weight(wd, rotate=True)
    del wd
    w6 = q.quarot_pack_e3m2(wq)
    rwq, rsw = orc.prepare_weight(w, rotate=True)
    del w
    assert_same(H(wq), rwq, f"{name} weight codes")
    assert_same(H(sw).view(np.uint16), rsw.view(np.uint16), f"{name} weight scales")
    wrows = sample_rows(N, 1, 7)
    assert_same(decode_e3m2_layout(H(w6), N, K, wrows),
                orc.unpack_int4(rwq[wrows]).astype(np.float64), f"{name} e3m2 weight layout")

    say(f"{name}: gpu e3m2 and int4 paths")
    xd = T(x, dev)
    x6, sx6 = q.quarot_quant_int4_e3m2(xd, rotate=True, clip_ratio=1.0)
    y6, acc6 = q.quarot_w4a4_gemm_e3m2(x6, sx6, w6, sw, want_acc=True)
    xq, sx = q.quarot_quant_int4(xd, rotate=True, clip_ratio=1.0)
    y4, acc4 = q.quarot_w4a4_gemm(xq, sx, wq, sw, want_acc=True)
    torch.cuda.synchronize()
    nd_acc = int((acc6 != acc4).sum().item())
    nd_y = int((y6.view(torch.int16) != y4.view(torch.int16)).sum().item())
    say(f"{name}: all {M}x{N} outputs, e3m2 vs int4 path: acc differ {nd_acc}, y differ {nd_y}")
    assert nd_acc == 0 and nd_y == 0
    assert torch.equal(sx6.view(torch.int16), sx.view(torch.int16))
    del acc4, y4
    yl6 = q.quarot_linear_e3m2(xd, w6, sw, rotate=True, clip_ratio=1.0)
    yl4 = q.quarot_linear(xd, wq, sw, rotate=True, clip_ratio=1.0)
    torch.cuda.synchronize()
    assert torch.equal(yl6.view(torch.int16), y6.view(torch.int16))
    assert torch.equal(yl4.view(torch.int16), y6.view(torch.int16))
    del yl6, yl4

    rows = sample_rows(M, per_tile, 11)
    say(f"{name}: oracle on {len(rows)} rows ({per_tile} per 256-row tile) x {N} columns")
    rxq, rsx = orc.quant_int4(x[rows], rotate=True, clip=1.0)
    ri = torch.from_numpy(rows).to(dev)
    assert_same(H(xq.index_select(0, ri)), rxq, f"{name} int4 activation codes")
    assert_same(H(sx6.index_select(0, ri)).view(np.uint16), rsx.view(np.uint16),
                f"{name} activation scales")
    assert_same(decode_e3m2_layout(H(x6), M, K, rows), orc.unpack_int4(rxq).astype(np.float64),
                f"{name} e3m2 activation codes")
    racc = orc.gemm_i32(rxq, rwq)
    ry = orc.dequant(racc, rsx, rsw)
    assert_same(H(acc6.index_select(0, ri)), racc, f"{name} int32 acc")
    assert_same(H(y6.index_select(0, ri)).view(np.uint16), ry.view(np.uint16), f"{name} y")
