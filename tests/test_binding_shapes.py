"""The Python binding checks every tensor against the sizes it hands to the
C ABI (the library trusts its pointers), and raises ValueError before
anything is launched.  CPU tensors suffice: the shape checks come first,
so no device is touched."""
import pytest
import torch

import paper_2404_00456_amd as q

SHAPE = "must have shape|must hold|must be [0-9]-D|must be a positive divisor|rows must hold|do not match"


def f16(*s):
    return torch.zeros(s, dtype=torch.float16)


def u8(*s):
    return torch.zeros(s, dtype=torch.uint8)


def i8(*s):
    return torch.zeros(s, dtype=torch.int8)


CASES = {
    "hadamard y": lambda: q.quarot_hadamard(f16(4, 128), y=f16(4, 64)),
    "quant_int4 q": lambda: q.quarot_quant_int4(f16(4, 128), q=u8(4, 63)),
    "quant_int4 scale": lambda: q.quarot_quant_int4(f16(4, 128), scale=f16(3)),
    "gemm wq K": lambda: q.quarot_w4a4_gemm(u8(8, 64), f16(8), u8(16, 32), f16(16)),
    "gemm sx": lambda: q.quarot_w4a4_gemm(u8(8, 64), f16(7), u8(16, 64), f16(16)),
    "gemm sw": lambda: q.quarot_w4a4_gemm(u8(8, 64), f16(8), u8(16, 64), f16(15)),
    "gemm y": lambda: q.quarot_w4a4_gemm(u8(8, 64), f16(8), u8(16, 64), f16(16), y=f16(8, 15)),
    "gemm acc": lambda: q.quarot_w4a4_gemm(u8(8, 64), f16(8), u8(16, 64), f16(16),
                                           acc_out=torch.zeros((7, 16), dtype=torch.int32)),
    "gemm 1-D": lambda: q.quarot_w4a4_gemm(u8(512), f16(8), u8(16, 64), f16(16)),
    "pack out": lambda: q.quarot_pack_e3m2(u8(4, 64), out=u8(1, 4 * 95)),
    "gemm e3m2 operands": lambda: q.quarot_w4a4_gemm_e3m2(u8(1, 8 * 96), f16(8), u8(1, 15 * 96),
                                                          f16(16)),
    "gemm e3m2 y": lambda: q.quarot_w4a4_gemm_e3m2(u8(1, 8 * 96), f16(8), u8(1, 16 * 96), f16(16),
                                                   y=f16(16, 8)),
    "quant e3m2 q6": lambda: q.quarot_quant_int4_e3m2(f16(8, 128), q6=u8(1, 7 * 96)),
    "quant e3m2 scale": lambda: q.quarot_quant_int4_e3m2(f16(8, 128), scale=f16(9)),
    "linear e3m2 wq6": lambda: q.quarot_linear_e3m2(f16(8, 128), u8(1, 15 * 96), f16(16)),
    "linear e3m2 y": lambda: q.quarot_linear_e3m2(f16(8, 128), u8(1, 16 * 96), f16(16),
                                                  y=f16(8, 17)),
    "swiglu e3m2 up": lambda: q.quarot_swiglu_quant_e3m2(f16(8, 128), f16(8, 64)),
    "linear wq": lambda: q.quarot_linear(f16(8, 128), u8(16, 32), f16(16)),
    "linear sw": lambda: q.quarot_linear(f16(8, 128), u8(16, 64), f16(17)),
    "linear y": lambda: q.quarot_linear(f16(8, 128), u8(16, 64), f16(16), y=f16(16, 8)),
    "quant_int8 q": lambda: q.quarot_quant_int8(f16(4, 128), q=i8(4, 127)),
    "w8a8 wq": lambda: q.quarot_w8a8_gemm(i8(8, 64), f16(8), i8(16, 32), f16(16)),
    "w8a8 acc": lambda: q.quarot_w8a8_gemm(i8(8, 64), f16(8), i8(16, 64), f16(16),
                                           acc_out=torch.zeros((8, 15), dtype=torch.int32)),
    "linear w8a8 sw": lambda: q.quarot_linear_w8a8(f16(8, 64), i8(16, 64), f16(8)),
    "grouped quant scale": lambda: q.quarot_quant_int4_grouped(f16(8, 256), group=128,
                                                               scale=f16(8, 2)),
    "grouped quant group": lambda: q.quarot_quant_int4_grouped(f16(8, 256), group=96),
    "grouped gemm sx": lambda: q.quarot_w4a4_gemm_grouped(u8(8, 128), f16(8, 2), u8(16, 128),
                                                          f16(2, 16), group=128),
    "grouped gemm wq": lambda: q.quarot_w4a4_gemm_grouped(u8(8, 128), f16(2, 8), u8(16, 64),
                                                          f16(2, 16), group=128),
    "grouped linear sw": lambda: q.quarot_linear_w4a4_grouped(f16(8, 256), u8(16, 128),
                                                              f16(16, 2), group=128),
    "swiglu h": lambda: q.quarot_swiglu(f16(64), f16(64), h=f16(32)),
    "swiglu quant q": lambda: q.quarot_swiglu_quant_int4(f16(4, 128), f16(4, 128), q=u8(4, 32)),
    "heads y": lambda: q.quarot_hadamard_heads(f16(4, 1024), 8, y=f16(4, 512)),
    "heads count": lambda: q.quarot_hadamard_heads(f16(4, 1000), 16),
    "heads quant scale": lambda: q.quarot_hadamard_heads_quant_int4(f16(4, 1024), 8, scale=f16(5)),
    "kv quant zero": lambda: q.quarot_kv_quant(f16(16, 128), group=64, zero=f16(16, 1)),
    "kv quant group": lambda: q.quarot_kv_quant(f16(16, 128), group=0),
    "kv dequant scale": lambda: q.quarot_kv_dequant(u8(16, 64), f16(16, 1), f16(16, 2), group=64),
    "kv dequant out": lambda: q.quarot_kv_dequant(u8(16, 64), f16(16, 1), f16(16, 1),
                                                  out=f16(16, 64)),
    "kv append cache rows": lambda: q.quarot_kv_append(f16(4, 128), u8(3, 10, 64), f16(4, 10, 1),
                                                       f16(4, 10, 1), pos=0),
    "kv append scale": lambda: q.quarot_kv_append(f16(4, 128), u8(4, 10, 64), f16(4, 9, 1),
                                                  f16(4, 10, 1), pos=0),
    "kv append width": lambda: q.quarot_kv_append(f16(4, 128), u8(4, 20, 32), f16(4, 10, 1),
                                                  f16(4, 10, 1), pos=0),
    "decode v_codes": lambda: q.quarot_kv_decode_attention(
        f16(8, 128), (u8(2, 16, 64), f16(2, 16, 1), f16(2, 16, 1)),
        (u8(2, 15, 64), f16(2, 16, 1), f16(2, 16, 1)), 16),
    "decode k_scale": lambda: q.quarot_kv_decode_attention(
        f16(8, 128), (u8(2, 16, 64), f16(2, 16, 2), f16(2, 16, 1)),
        (u8(2, 16, 64), f16(2, 16, 1), f16(2, 16, 1)), 16),
    "decode q width": lambda: q.quarot_kv_decode_attention(
        f16(8, 64), (u8(2, 16, 64), f16(2, 16, 1), f16(2, 16, 1)),
        (u8(2, 16, 64), f16(2, 16, 1), f16(2, 16, 1)), 16, group=64),
    "decode out": lambda: q.quarot_kv_decode_attention(
        f16(8, 128), (u8(2, 16, 64), f16(2, 16, 1), f16(2, 16, 1)),
        (u8(2, 16, 64), f16(2, 16, 1), f16(2, 16, 1)), 16, out=f16(4, 128)),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_mismatched_shape_raises_before_launch(case):
    with pytest.raises(ValueError, match=SHAPE):
        CASES[case]()
