"""The allocation-free linear layer (quarot_linear_e3m2_scratch, for callers
that cannot allocate device memory) through the C ABI: its output equals
quarot_linear_e3m2's (the workspace entry point) bit for bit on two calls
in a row, the second on a smaller input, so the fixed scratch array's
leftover contents from the first call cannot leak into the second; sizes
beyond the array are refused before any device work."""
import ctypes

import numpy as np
import pytest

import workloads
from test_gpu_parity import T, say

pytestmark = pytest.mark.gpu

WORKSPACE = 4


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_00456_amd as q
    q.lib()
    return torch.device("cuda:0")


def scratch_call(x, w6, sw, y, rotate=True, clip=1.0):
    import torch
    import paper_2404_00456_amd as q
    M, K = x.shape
    N = sw.numel()
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    return q.lib().quarot_linear_e3m2_scratch(
        p(x), p(w6), p(sw), p(y), M, N, K, int(rotate), float(clip),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


def test_scratch_entry_point_matches_workspace_entry_point(dev):
    import torch
    import paper_2404_00456_amd as q
    # the first call the largest (44 MB of codes and scales), then smaller
    for M, N, K, clip, seed in ((2048, 4096, 28672, 1.0, 1), (300, 520, 11008, 0.9, 2),
                                (64, 256, 8192, 1.0, 3)):
        say(f"scratch linear M={M} N={N} K={K}")
        assert q.quarot_linear_e3m2_workspace_size(M, K) <= q.SCRATCH_BYTES
        x = T(workloads.random_rows(seed, M, K, "student_t3", 2.0), dev)
        w = T(workloads.random_rows(seed + 100, N, K, "normal", 0.02), dev)
        w6, sw = q.prepare_weight_e3m2(w, rotate=True)
        ref = q.quarot_linear_e3m2(x, w6, sw, rotate=True, clip_ratio=clip)
        y = torch.full((M, N), 7.0, dtype=torch.float16, device=dev)
        assert scratch_call(x, w6, sw, y, clip=clip) == 0
        torch.cuda.synchronize()
        nd = int((y.view(torch.int16) != ref.view(torch.int16)).sum().item())
        say(f"scratch linear M={M} N={N} K={K}: {nd} differing of {M * N}")
        assert nd == 0


def test_scratch_entry_point_refuses_oversize(dev):
    import torch
    import paper_2404_00456_amd as q
    M, N, K = 16384, 256, 8192  # 100 MB of codes: beyond the 64 MiB array
    assert q.quarot_linear_e3m2_workspace_size(M, K) > q.SCRATCH_BYTES
    x = torch.zeros((M, K), dtype=torch.float16, device=dev)
    w6 = torch.zeros((K // 128, N * 96), dtype=torch.uint8, device=dev)
    sw = torch.ones(N, dtype=torch.float16, device=dev)
    y = torch.full((M, N), 3.0, dtype=torch.float16, device=dev)
    assert scratch_call(x, w6, sw, y) == WORKSPACE
    torch.cuda.synchronize()
    assert bool((y == 3.0).all())
