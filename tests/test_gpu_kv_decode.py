"""GPU parity of the 4-bit KV cache decode path (App. A.10 Append and
Decode; §4 Stage 2c) through the C ABI, against the CPU oracle.  Append
writes codes, scales and zeros bit for bit; the attention output is a
floating-point result and must satisfy max |gpu - oracle| <= 1e-2 *
max |oracle| (the measured error is printed; binary32 accumulation keeps
it within about one fp16 ulp of the fp64 oracle)."""
import numpy as np
import pytest

import workloads
from test_gpu_parity import H, T, assert_same, say

pytestmark = pytest.mark.gpu

FP_TOL = 1e-2


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2404_00456_amd as q
    q.lib()
    return torch.device("cuda:0")


def rand_cache(rng, nkv, s_max, D, G):
    codes = rng.integers(0, 256, size=(nkv, s_max, D // 2), dtype=np.uint8)
    scale = rng.uniform(0.05, 0.6, size=(nkv, s_max, D // G)).astype(np.float16)
    zero = rng.uniform(-3, 0, size=(nkv, s_max, D // G)).astype(np.float16)
    return codes, scale, zero


def check_attention(dev, orc, q, k, v, seq, G, what):
    import paper_2404_00456_amd as qq
    kd = tuple(T(x, dev) for x in k)
    vd = tuple(T(x, dev) for x in v)
    got = H(qq.quarot_kv_decode_attention(T(q, dev), kd, vd, seq, group=G)).astype(np.float64)
    ref = orc.kv_attention(q, k, v, seq, group=G).astype(np.float64)
    err = np.abs(got - ref).max()
    amax = np.abs(ref).max()
    ulp = np.abs(got - ref) / np.maximum(np.abs(ref) * 2.0 ** -10, 2.0 ** -24)
    say(f"{what}: max|err|={err:.3g} max|ref|={amax:.3g} max err in fp16 ulps={ulp.max():.2f}")
    assert err <= FP_TOL * amax, what


@pytest.mark.parametrize("nkv,rep,s_max,seq,D,G", [
    (1, 1, 1, 1, 128, 128), (3, 1, 40, 17, 128, 128), (16, 1, 300, 300, 128, 64),
    (4, 8, 512, 511, 128, 128), (8, 1, 2048, 1500, 64, 32), (2, 2, 1000, 999, 256, 128),
    (64, 1, 4096, 4096, 128, 128), (1, 1, 9000, 8191, 128, 128),
    # the benchmarked decode step: 16 x 64 query rows over 4096 cached tokens
    (1024, 1, 4096, 4096, 128, 128)])
def test_decode_attention_random_cache(dev, orc, nkv, rep, s_max, seq, D, G):
    rng = np.random.default_rng(nkv * 7 + s_max + D + G)
    k = rand_cache(rng, nkv, s_max, D, G)
    v = rand_cache(rng, nkv, s_max, D, G)
    q = (rng.standard_normal((nkv * rep, D)) * 0.5).astype(np.float16)
    check_attention(dev, orc, q, k, v, seq, G, f"attn nkv={nkv} rep={rep} seq={seq} D={D} G={G}")


def test_decode_attention_peaked_scores(dev, orc):
    """Large scores (one token dominates): the running max must rescale."""
    rng = np.random.default_rng(9)
    k = rand_cache(rng, 4, 1024, 128, 128)
    v = rand_cache(rng, 4, 1024, 128, 128)
    q = (rng.standard_normal((4, 128)) * 20).astype(np.float16)
    check_attention(dev, orc, q, k, v, 1024, 128, "attn peaked")


def test_append_then_decode_on_quantized_heads(dev, orc):
    """The config-5 head shape (head_dim 128, group 128, clip 0.95): fill a
    cache with quarot_kv_append one token at a time for 2 batch x 64 heads,
    compare it bit for bit with the oracle, then decode."""
    import paper_2404_00456_amd as qq
    import torch
    wl = workloads.KV["kv4_70b"]
    B, Hh, S, D, G = 2, wl.H, 48, wl.D, wl.group
    k, v = workloads.kv_inputs(wl, B=B, S=S)
    k = k.reshape(B * Hh, S, D)
    v = v.reshape(B * Hh, S, D)
    rows = B * Hh
    caches = []
    for t_np in (k, v):
        qc = torch.zeros((rows, S, D // 2), dtype=torch.uint8, device=dev)
        sc = torch.zeros((rows, S, D // G), dtype=torch.float16, device=dev)
        zc = torch.zeros_like(sc)
        td = T(t_np, dev)
        for pos in range(S):
            qq.quarot_kv_append(td[:, pos].contiguous(), qc, sc, zc, pos, group=G,
                                rotate=True, clip_ratio=wl.clip)
        rq, rs, rz = orc.kv_quant(t_np.reshape(-1, D), group=G, rotate=True, clip=wl.clip)
        assert_same(H(qc).reshape(-1, D // 2), rq, "appended codes")
        assert_same(H(sc).reshape(-1).view(np.uint16), rs.reshape(-1).view(np.uint16), "scales")
        assert_same(H(zc).reshape(-1).view(np.uint16), rz.reshape(-1).view(np.uint16), "zeros")
        caches.append((H(qc), H(sc), H(zc)))
    rng = np.random.default_rng(0)
    qv = rng.standard_normal((rows, D)).astype(np.float16)
    qrot = H(qq.quarot_hadamard(T(qv, dev)))  # queries rotated like the keys
    check_attention(dev, orc, qrot, caches[0], caches[1], S, G, "append+decode")
