"""Pins for the oracle's 4-bit KV decode path (App. A.10 Append / Decode,
§4 Stage 2c): attention over the dequantized cache against torch's
scaled_dot_product_attention (a library routine) in float64, closed forms
(one token, uniform scores), invariants (tokens past seq_len are ignored,
grouped queries equal repeated caches), and Append against kv_quant."""
import numpy as np
import pytest
import torch

F16_ULP = 2.0 ** -10


def make_cache(rng, nkv, s_max, D, G):
    codes = rng.integers(0, 256, size=(nkv, s_max, D // 2), dtype=np.uint8)
    scale = rng.uniform(0.05, 0.6, size=(nkv, s_max, D // G)).astype(np.float16)
    zero = rng.uniform(-3, 0, size=(nkv, s_max, D // G)).astype(np.float16)
    return codes, scale, zero


def dequant_exact(orc, cache, G):
    codes, scale, zero = cache
    c = orc.unpack_uint4(codes).astype(np.float64)
    s = np.repeat(scale.astype(np.float64), G, axis=-1)
    z = np.repeat(zero.astype(np.float64), G, axis=-1)
    return c * s + z


@pytest.mark.parametrize("nkv,rep,s_max,seq,D,G", [(3, 1, 40, 40, 128, 128), (2, 4, 64, 37, 64, 32),
                                                   (4, 1, 300, 257, 128, 64), (1, 8, 17, 1, 256, 128)])
def test_attention_matches_sdpa(orc, nkv, rep, s_max, seq, D, G):
    rng = np.random.default_rng(nkv * 1000 + s_max + D)
    k = make_cache(rng, nkv, s_max, D, G)
    v = make_cache(rng, nkv, s_max, D, G)
    q = rng.standard_normal((nkv * rep, D)).astype(np.float16)
    out = orc.kv_attention(q, k, v, seq, group=G).astype(np.float64)
    K = torch.from_numpy(dequant_exact(orc, k, G)[:, :seq]).repeat_interleave(rep, 0)
    V = torch.from_numpy(dequant_exact(orc, v, G)[:, :seq]).repeat_interleave(rep, 0)
    Q = torch.from_numpy(q.astype(np.float64))[:, None, :]
    ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V)[:, 0, :].numpy()
    assert np.all(np.abs(out - ref) <= F16_ULP * np.abs(ref) + 2.0 ** -24)


def test_one_token_returns_its_value_row(orc):
    rng = np.random.default_rng(1)
    k = make_cache(rng, 2, 8, 128, 128)
    v = make_cache(rng, 2, 8, 128, 128)
    q = rng.standard_normal((2, 128)).astype(np.float16)
    out = orc.kv_attention(q, k, v, 1)
    ref = dequant_exact(orc, v, 128)[:, 0].astype(np.float16)  # numpy rounds fp64 once
    assert np.array_equal(out, ref)


def test_output_rounded_once_from_fp64(orc):
    """Two tokens with equal scores average their value rows.  Token 0's
    row is 1 (code 0, zero 1); token 1's is 1 + 2^-10 + 2^-24 (code 1,
    scale 1 + 2^-10, zero 2^-24, both fp16).  The exact output
    1 + 2^-11 + 2^-25 lies just above the fp16 midpoint 1 + 2^-11: rounded
    once it is 1 + 2^-10, while a detour through binary32 lands on the
    midpoint and ties to even, 1."""
    D = G = 8
    q = np.zeros((1, D), np.float16)
    kc = np.zeros((1, 2, D // 2), np.uint8)
    ks = np.ones((1, 2, 1), np.float16)
    kz = np.zeros((1, 2, 1), np.float16)
    vc = np.zeros((1, 2, D // 2), np.uint8)
    vc[0, 1] = 0x11  # code 1 everywhere
    vs = np.array([[[1.0], [1.0 + 2.0 ** -10]]], np.float16)
    vz = np.array([[[1.0], [2.0 ** -24]]], np.float16)
    out = orc.kv_attention(q, (kc, ks, kz), (vc, vs, vz), 2, group=G)
    exact = 1.0 + 2.0 ** -11 + 2.0 ** -25
    assert np.float64(exact).astype(np.float32) == np.float32(1.0 + 2.0 ** -11)
    assert np.all(out.view(np.uint16) == np.float16(1.0 + 2.0 ** -10).view(np.uint16))


def test_zero_query_averages_values(orc):
    rng = np.random.default_rng(2)
    k = make_cache(rng, 1, 50, 64, 64)
    v = make_cache(rng, 1, 50, 64, 64)
    q = np.zeros((1, 64), np.float16)
    out = orc.kv_attention(q, k, v, 33, group=64).astype(np.float64)
    ref = dequant_exact(orc, v, 64)[0, :33].mean(axis=0)
    assert np.all(np.abs(out[0] - ref) <= F16_ULP * np.abs(ref) + 2.0 ** -24)


def test_tokens_past_seq_len_ignored(orc):
    rng = np.random.default_rng(3)
    k = make_cache(rng, 2, 64, 128, 128)
    v = make_cache(rng, 2, 64, 128, 128)
    q = rng.standard_normal((2, 128)).astype(np.float16)
    a = orc.kv_attention(q, k, v, 40)
    k2 = tuple(x.copy() for x in k)
    v2 = tuple(x.copy() for x in v)
    k2[0][:, 40:] = 0xFF
    v2[1][:, 40:] = 7.0
    assert np.array_equal(a, orc.kv_attention(q, k2, v2, 40))


def test_grouped_queries_equal_repeated_cache(orc):
    rng = np.random.default_rng(4)
    k = make_cache(rng, 2, 30, 128, 128)
    v = make_cache(rng, 2, 30, 128, 128)
    q = rng.standard_normal((8, 128)).astype(np.float16)
    grouped = orc.kv_attention(q, k, v, 30)
    rep = tuple(np.repeat(x, 4, axis=0) for x in k), tuple(np.repeat(x, 4, axis=0) for x in v)
    assert np.array_equal(grouped, orc.kv_attention(q, rep[0], rep[1], 30))


def test_append_writes_one_position(orc):
    rng = np.random.default_rng(5)
    rows, s_max, D, G = 6, 10, 128, 64
    cache = make_cache(rng, rows, s_max, D, G)
    kv_new = rng.standard_normal((rows, D)).astype(np.float16)
    qc, sc, zc = orc.kv_append(kv_new, *cache, pos=7, group=G)
    rq, rs, rz = orc.kv_quant(kv_new, group=G, rotate=True, clip=0.95)
    assert np.array_equal(qc[:, 7], rq) and np.array_equal(sc[:, 7], rs) and np.array_equal(zc[:, 7], rz)
    keep = [t for t in range(s_max) if t != 7]
    assert np.array_equal(qc[:, keep], cache[0][:, keep])
    assert np.array_equal(sc[:, keep], cache[1][:, keep])
