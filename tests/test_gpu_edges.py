"""Edge cases of the C ABI on a device: empty inputs are no-ops, rejected
arguments leave the outputs untouched, misaligned and non-contiguous
buffers are refused, and a call enqueued on a side stream gives the same
bits as on the default stream."""
import numpy as np
import pytest

import workloads
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


def test_empty_inputs_are_no_ops(dev):
    import torch
    import paper_2404_00456_amd as q
    say("empty inputs")
    e16 = torch.empty((0, 128), dtype=torch.float16, device=dev)
    assert q.quarot_hadamard(e16).shape == (0, 128)
    codes, scale = q.quarot_quant_int4(e16, rotate=True)
    assert codes.shape == (0, 64) and scale.shape == (0,)
    codes8, _ = q.quarot_quant_int8(e16, rotate=True, bits=8)
    assert codes8.shape == (0, 128)
    gq, gs = q.quarot_quant_int4_grouped(e16, group=64, rotate=True)
    assert gq.shape == (0, 64) and gs.shape == (2, 0)
    assert q.quarot_hadamard_heads(torch.empty((0, 8192), dtype=torch.float16, device=dev),
                                   64).shape == (0, 8192)
    # M = 0 and N = 0 products
    wq = torch.zeros((256, 64), dtype=torch.uint8, device=dev)
    sw = torch.ones(256, dtype=torch.float16, device=dev)
    xq0 = torch.zeros((0, 64), dtype=torch.uint8, device=dev)
    sx0 = torch.ones(0, dtype=torch.float16, device=dev)
    assert q.quarot_w4a4_gemm(xq0, sx0, wq, sw).shape == (0, 256)
    xq = torch.zeros((16, 64), dtype=torch.uint8, device=dev)
    sx = torch.ones(16, dtype=torch.float16, device=dev)
    assert q.quarot_w4a4_gemm(xq, sx, wq[:0], sw[:0]).shape == (16, 0)
    assert q.quarot_linear(e16, wq, sw).shape == (0, 256)
    kq, ks, kz = q.quarot_kv_quant(e16, group=128, rotate=True)
    assert kq.shape == (0, 64)
    g = torch.empty(0, dtype=torch.float16, device=dev)
    assert q.quarot_swiglu(g, g).shape == (0,)
    torch.cuda.synchronize()


def test_rejected_arguments_leave_outputs_untouched(dev):
    import torch
    import paper_2404_00456_amd as q
    say("rejected arguments")
    x = T(workloads.random_rows(5, 32, 4096), dev)
    qbuf = torch.full((32, 2048), 0xAB, dtype=torch.uint8, device=dev)
    sbuf = torch.full((32,), 7.0, dtype=torch.float16, device=dev)
    for clip in (0.0, 1.5, float("nan")):
        with pytest.raises(q.QuarotError):
            q.quarot_quant_int4(x, rotate=True, clip_ratio=clip, q=qbuf, scale=sbuf)
    with pytest.raises(q.QuarotError):  # width 100 has no Hadamard factorization
        q.quarot_quant_int4(x[:, :100].contiguous(), rotate=True, q=qbuf[:, :50].contiguous())
    torch.cuda.synchronize()
    assert bool((qbuf == 0xAB).all()) and bool((sbuf == 7.0).all())
    # GEMM with an unsupported K (not a multiple of 64)
    xq = torch.zeros((8, 50), dtype=torch.uint8, device=dev)
    y = torch.full((8, 16), 3.0, dtype=torch.float16, device=dev)
    with pytest.raises(q.QuarotError):
        q.quarot_w4a4_gemm(xq, sbuf[:8].contiguous(), torch.zeros((16, 50), dtype=torch.uint8,
                                                                  device=dev),
                           torch.ones(16, dtype=torch.float16, device=dev), y=y)
    torch.cuda.synchronize()
    assert bool((y == 3.0).all())


def test_misaligned_and_strided_buffers_refused(dev):
    import torch
    import paper_2404_00456_amd as q
    say("misaligned / strided")
    base = torch.zeros(4 * 4096 + 8, dtype=torch.float16, device=dev)
    shifted = base[1:1 + 4 * 4096].view(4, 4096)  # 2-byte offset
    with pytest.raises(q.QuarotError) as ei:
        q.quarot_hadamard(shifted)
    assert ei.value.status == 3  # QUAROT_ERR_ALIGNMENT
    strided = torch.zeros((4, 8192), dtype=torch.float16, device=dev)[:, ::2]
    with pytest.raises(ValueError):
        q.quarot_hadamard(strided)


def test_side_stream_matches_default_stream(dev, orc):
    import torch
    import paper_2404_00456_amd as q
    say("side stream")
    x = workloads.random_rows(11, 300, 8192)
    xd = T(x, dev)
    codes0, scale0 = q.quarot_quant_int4(xd, rotate=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        codes1, scale1 = q.quarot_quant_int4(xd, rotate=True, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    assert_same(H(codes1), H(codes0), "codes on a side stream")
    assert_same(H(scale1).view(np.uint16), H(scale0).view(np.uint16), "scales on a side stream")
    rq, _ = orc.quant_int4(x, rotate=True)
    assert_same(H(codes1), rq, "side-stream codes vs oracle")


def test_e3m2_entry_points_edges(dev, orc):
    """The e3m2 operand path: empty inputs are no-ops, rejected arguments
    leave the outputs untouched, misaligned buffers are refused, and a side
    stream gives the default stream's bits."""
    import torch
    import paper_2404_00456_amd as q
    say("e3m2 edges")
    e16 = torch.empty((0, 8192), dtype=torch.float16, device=dev)
    q6, s6 = q.quarot_quant_int4_e3m2(e16, rotate=True)
    assert q6.shape == (64, 0) and s6.shape == (0,)
    assert q.quarot_pack_e3m2(torch.empty((0, 4096), dtype=torch.uint8, device=dev)).shape == (64, 0)
    w6 = torch.zeros((64, 256 * 96), dtype=torch.uint8, device=dev)
    sw = torch.ones(256, dtype=torch.float16, device=dev)
    x6 = torch.zeros((64, 0), dtype=torch.uint8, device=dev)
    assert q.quarot_w4a4_gemm_e3m2(x6, torch.ones(0, dtype=torch.float16, device=dev), w6,
                                   sw).shape == (0, 256)
    assert q.quarot_linear_e3m2(e16, w6, sw).shape == (0, 256)
    # rejected: clip out of range, width without an e3m2 epilogue
    x = T(workloads.random_rows(21, 32, 8192), dev)
    qbuf = torch.full((64, 32 * 96), 0xAB, dtype=torch.uint8, device=dev)
    sbuf = torch.full((32,), 7.0, dtype=torch.float16, device=dev)
    for clip in (0.0, 1.5):
        with pytest.raises(q.QuarotError):
            q.quarot_quant_int4_e3m2(x, rotate=True, clip_ratio=clip, q6=qbuf, scale=sbuf)
    with pytest.raises(q.QuarotError):  # 7168 = 2^8 * 28: refused, int4 + repack instead
        q.quarot_quant_int4_e3m2(torch.zeros((32, 7168), dtype=torch.float16, device=dev),
                                 rotate=True, q6=qbuf.view(-1)[:56 * 32 * 96].view(56, 32 * 96),
                                 scale=sbuf)
    with pytest.raises(ValueError):  # a code buffer smaller than rows x n needs
        q.quarot_quant_int4_e3m2(torch.zeros((32, 13824), dtype=torch.float16, device=dev),
                                 rotate=True, q6=qbuf, scale=sbuf)
    y = torch.full((32, 256), 3.0, dtype=torch.float16, device=dev)
    with pytest.raises(q.QuarotError):  # clip out of range
        q.quarot_linear_e3m2(x, w6, sw, clip_ratio=2.0, y=y)
    torch.cuda.synchronize()
    assert bool((qbuf == 0xAB).all()) and bool((sbuf == 7.0).all()) and bool((y == 3.0).all())
    # misaligned code buffer
    raw = torch.zeros(64 * 32 * 96 + 16, dtype=torch.uint8, device=dev)
    with pytest.raises(q.QuarotError) as ei:
        q.quarot_quant_int4_e3m2(x, rotate=True, q6=raw[8:8 + 64 * 32 * 96].view(64, 32 * 96),
                                 scale=sbuf)
    assert ei.value.status == 3
    # side stream
    xs = workloads.random_rows(23, 300, 8192)
    xd = T(xs, dev)
    a6, a_s = q.quarot_quant_int4_e3m2(xd, rotate=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        b6, b_s = q.quarot_quant_int4_e3m2(xd, rotate=True, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    assert_same(H(b6), H(a6), "e3m2 codes on a side stream")
    assert_same(H(b_s).view(np.uint16), H(a_s).view(np.uint16), "e3m2 scales on a side stream")


def test_fake_hip_error_leaves_outputs_untouched(dev, monkeypatch):
    """With QUAROT_FAKE_HIP_ERROR naming the call, the two-launch layer
    entry point reports QUAROT_ERR_HIP with hipErrorLaunchFailure and writes
    neither its output nor its workspace; with the variable cleared the
    same call runs."""
    import torch
    import paper_2404_00456_amd as q
    say("fake hip error")
    x = T(workloads.random_rows(31, 64, 8192), dev)
    w6 = torch.zeros((64, 256 * 96), dtype=torch.uint8, device=dev)
    sw = torch.ones(256, dtype=torch.float16, device=dev)
    y = torch.full((64, 256), 3.0, dtype=torch.float16, device=dev)
    ws = torch.full((q.quarot_linear_e3m2_workspace_size(64, 8192),), 0x5A, dtype=torch.uint8,
                    device=dev)
    monkeypatch.setenv("QUAROT_FAKE_HIP_ERROR", "quarot_linear_e3m2")
    with pytest.raises(q.QuarotError) as ei:
        q.quarot_linear_e3m2(x, w6, sw, y=y, workspace=ws)
    assert ei.value.status == 6 and ei.value.hip_error == 719
    torch.cuda.synchronize()
    assert bool((y == 3.0).all()) and bool((ws == 0x5A).all())
    monkeypatch.delenv("QUAROT_FAKE_HIP_ERROR")
    q.quarot_linear_e3m2(x, w6, sw, y=y, workspace=ws)
    torch.cuda.synchronize()
    assert bool((y == 0.0).all())  # zero weights
