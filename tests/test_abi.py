"""C-ABI checks that need no GPU: the library loads, exports every symbol
that include/quarot.h declares (and the measurement library every symbol of
include/quarot_probe.h, which libquarot itself does not export), answers
host-only queries, and rejects bad arguments before touching any device.
No kernel is launched here."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2404_00456_amd as q

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
HEADER = os.path.join(INCLUDE, "quarot.h")
PROBE_HEADER = os.path.join(INCLUDE, "quarot_probe.h")

OK, INVALID, UNSUPPORTED, ALIGN, WORKSPACE, NODEV, HIP = range(7)

# fake, aligned, never dereferenced device addresses for validation tests
P = ctypes.c_void_p(1 << 20)
P2 = ctypes.c_void_p((1 << 20) + 4096)
UNALIGNED = ctypes.c_void_p((1 << 20) + 8)


def declared_functions(header=HEADER):
    src = open(header).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(quarot_[a-z0-9_]+)\s*\(", src)))


def has_gpu():
    import torch
    return torch.cuda.device_count() > 0


@pytest.fixture(scope="module")
def L():
    return q.lib()


@pytest.fixture(scope="module")
def PL():
    return q.probe_lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(L, name), name
    # and the binding declares exactly those signatures
    assert sorted(q.SIGNATURES) == names


def test_probe_library_is_apart(L, PL):
    names = declared_functions(PROBE_HEADER)
    assert len(names) == 4
    for name in names:
        assert hasattr(PL, name), name
        assert not hasattr(L, name), name  # measurement tools stay out of libquarot
    assert sorted(q.PROBE_SIGNATURES) == names


def test_status_strings(L):
    for code, name in q.STATUS.items():
        assert L.quarot_status_string(code).decode() == name
    assert L.quarot_status_string(99).decode() == "QUAROT_ERR_UNKNOWN"
    assert q.quarot_version() == 100


def test_hadamard_factor_matches_oracle(orc):
    for n in (8, 16, 128, 1024, 4096, 8192, 16384, 32768, 11008, 28672, 5120, 13824, 14336,
              24, 40, 56, 344, 216, 20480, 24576):
        assert q.quarot_hadamard_factor(n) == orc.hadamard_factor(n), n
    for bad in (0, -8, 4, 12, 100, 65536, 172 * 128, 28 * 2048, 72, 20 * 2048):
        assert q.quarot_hadamard_factor(bad) is None, bad


@pytest.mark.parametrize("m", [12, 20, 28, 108, 172])
def test_library_tables_match_oracle(orc, m):
    """The library and the oracle build H_m independently from the same
    published constructions; they must agree entry for entry."""
    lib_t = q.quarot_hadamard_factor_table(m)
    assert np.array_equal(lib_t, orc.hm_table(m))
    H = lib_t.astype(np.int64)
    assert np.array_equal(H @ H.T, m * np.eye(m, dtype=np.int64))


def test_workspace_size(L):
    assert q.quarot_linear_workspace_size(16384, 8192) == 16384 * 4096 + 32768
    assert q.quarot_linear_workspace_size(3, 128) == 256 + 256
    assert q.quarot_linear_workspace_size(0, 128) == 256 * 0 + 0
    assert q.quarot_linear_workspace_size(-1, 128) == 0
    assert q.quarot_linear_workspace_size(4, 0) == 0
    assert q.quarot_linear_workspace_size(4, 7) == 0


def test_invalid_arguments_rejected_before_device(L):
    # Every call here must be invalid: the pointers are fake, and a call
    # with valid arguments would launch a kernel on them where a device is
    # present.  Valid arguments are exercised only without a device
    # (test_no_device_reported) and with real buffers in the GPU tests.
    S = None  # null stream
    # hadamard
    assert L.quarot_hadamard(P, P2, -1, 128, S) == INVALID
    assert L.quarot_hadamard(P, P2, 4, 0, S) == INVALID
    assert L.quarot_hadamard(P, P2, 4, 100, S) == UNSUPPORTED
    assert L.quarot_hadamard(P, P2, 4, 65536, S) == UNSUPPORTED
    assert L.quarot_hadamard(None, P2, 4, 128, S) == INVALID
    assert L.quarot_hadamard(UNALIGNED, P2, 4, 128, S) == ALIGN
    assert L.quarot_hadamard(None, None, 0, 128, S) == OK  # empty is a no-op
    # quant
    assert L.quarot_quant_int4(P, P2, P2, 4, 128, 1, 0.0, S) == INVALID
    assert L.quarot_quant_int4(P, P2, P2, 4, 128, 1, 1.5, S) == INVALID
    assert L.quarot_quant_int4(P, P2, P2, 4, 12, 0, 1.0, S) == UNSUPPORTED
    assert L.quarot_quant_int4(P, P2, P2, 4, 11008 * 3, 1, 1.0, S) == UNSUPPORTED
    assert L.quarot_quant_int4(P, None, P2, 4, 128, 1, 1.0, S) == INVALID
    assert L.quarot_quant_int4(P, P2, UNALIGNED, 4, 128, 1, 1.0, S) == ALIGN
    assert L.quarot_quant_int4(None, None, None, 0, 128, 1, 1.0, S) == OK
    # gemm
    assert L.quarot_w4a4_gemm(P, P, P, P, P, None, 4, 4, 100, S) == UNSUPPORTED
    assert L.quarot_w4a4_gemm(P, P, P, P, P, None, -1, 4, 128, S) == INVALID
    assert L.quarot_w4a4_gemm(P, P, P, P, P, None, 4, 4, 0, S) == INVALID
    assert L.quarot_w4a4_gemm(P, P, P, P, P, None, 4, 4, 65536 + 64, S) == UNSUPPORTED
    assert L.quarot_w4a4_gemm(P, None, P, P, P, None, 4, 4, 128, S) == INVALID
    assert L.quarot_w4a4_gemm(P, P, P, P, P, UNALIGNED, 4, 4, 128, S) == ALIGN
    assert L.quarot_w4a4_gemm(None, None, None, None, None, None, 0, 4, 128, S) == OK
    # linear
    assert L.quarot_linear(P, P, P, P, 4, 4, 128, 1, 1.0, None, 0, S) == WORKSPACE
    assert L.quarot_linear(P, P, P, P, 4, 4, 128, 1, 1.0, P, 10, S) == WORKSPACE
    assert L.quarot_linear(P, P, P, P, 4, 4, 128, 1, 1.0, ctypes.c_void_p((1 << 20) + 16),
                           4096, S) == ALIGN
    assert L.quarot_linear(P, P, P, P, 4, 4, 96, 1, 1.0, P, 4096, S) == UNSUPPORTED
    assert L.quarot_linear(P, P, P, P, 4, 4, 128, 1, -0.5, P, 4096, S) == INVALID
    # kv
    assert L.quarot_kv_quant(P, P, P, P, 4, 128, 256, 1, 0.95, S) == UNSUPPORTED
    assert L.quarot_kv_quant(P, P, P, P, 4, 96, 32, 1, 0.95, S) == UNSUPPORTED
    assert L.quarot_kv_quant(P, P, P, P, 4, 128, 4, 1, 0.95, S) == UNSUPPORTED
    assert L.quarot_kv_quant(P, P, P, P, 4, 1024, 128, 1, 0.95, S) == UNSUPPORTED
    assert L.quarot_kv_quant(P, P, P, None, 4, 128, 128, 1, 0.95, S) == INVALID
    assert L.quarot_kv_dequant(P, P, P, P, 4, 128, 0, 0, S) == INVALID
    assert L.quarot_kv_dequant(P, P, UNALIGNED, P, 4, 128, 128, 0, S) == ALIGN
    # 6/8-bit
    assert L.quarot_quant_int8(P, P2, P2, 4, 128, 1, 1.0, 4, S) == INVALID   # bits
    assert L.quarot_quant_int8(P, P2, P2, 4, 128, 1, 0.0, 8, S) == INVALID
    assert L.quarot_quant_int8(P, P2, P2, 4, 100, 1, 1.0, 8, S) == UNSUPPORTED
    assert L.quarot_quant_int8(P, UNALIGNED, P2, 4, 128, 1, 1.0, 8, S) == ALIGN
    assert L.quarot_quant_int8(None, None, None, 0, 128, 1, 1.0, 6, S) == OK
    assert L.quarot_w8a8_gemm(P, P, P, P, P, None, 4, 4, 96, S) == UNSUPPORTED
    assert L.quarot_w8a8_gemm(P, None, P, P, P, None, 4, 4, 128, S) == INVALID
    assert L.quarot_linear_w8a8_workspace_size(3, 128) == 512 + 256
    assert L.quarot_linear_w8a8(P, P, P, P, 4, 4, 128, 1, 1.0, 8, P, 10, S) == WORKSPACE
    assert L.quarot_linear_w8a8(P, P, P, P, 4, 4, 128, 1, 1.0, 5, P, 4096, S) == INVALID
    # clip search
    assert L.quarot_quant_search(P, P, P, P, 4, 128, 1, 5, 20, P, 1 << 20, S) == INVALID
    assert L.quarot_quant_search(P, P, P, P, 4, 128, 1, 4, 0, P, 1 << 20, S) == INVALID
    assert L.quarot_quant_search(P, P, P, P, 4, 128, 1, 4, 101, P, 1 << 20, S) == INVALID
    assert L.quarot_quant_search(P, P, P, P, 4, 100, 1, 4, 20, P, 1 << 20, S) == UNSUPPORTED
    assert L.quarot_quant_search(P, P, P, P, 4, 128, 1, 4, 20, P, 100, S) == WORKSPACE
    assert L.quarot_quant_search(P, P, P, None, 4, 128, 1, 4, 20, P, 1 << 20, S) == INVALID
    assert L.quarot_quant_search_workspace_size(4, 128, 1) == 4 * 128 * 4
    assert L.quarot_quant_search_workspace_size(4, 128, 0) == 0
    # kv append / decode attention
    assert L.quarot_kv_append(P, P, P, P, 4, 16, 16, 128, 128, 1, 0.95, S) == INVALID  # pos
    assert L.quarot_kv_append(P, P, P, P, 4, 16, -1, 128, 128, 1, 0.95, S) == INVALID
    assert L.quarot_kv_append(P, P, P, P, 4, 16, 3, 96, 32, 1, 0.95, S) == UNSUPPORTED
    assert L.quarot_kv_append(P, None, P, P, 4, 16, 3, 128, 128, 1, 0.95, S) == INVALID
    assert L.quarot_kv_append(None, None, None, None, 0, 16, 3, 128, 128, 1, 0.95, S) == OK
    A = (P, P, P, P, P, P, P, P2)
    assert L.quarot_kv_decode_attention(*A, 8, 3, 64, 64, 128, 128, 0.1, P, 1 << 20, S) == INVALID
    assert L.quarot_kv_decode_attention(*A, 8, 8, 64, 65, 128, 128, 0.1, P, 1 << 20, S) == INVALID
    assert L.quarot_kv_decode_attention(*A, 8, 8, 64, 0, 128, 128, 0.1, P, 1 << 20, S) == INVALID
    assert L.quarot_kv_decode_attention(*A, 8, 8, 64, 64, 96, 32, 0.1, P, 1 << 20, S) == UNSUPPORTED
    assert L.quarot_kv_decode_attention(*A, 8, 8, 64, 64, 128, 16, 0.1, P, 1 << 20, S) == UNSUPPORTED
    assert L.quarot_kv_decode_attention(*A, 8, 8, 64, 64, 128, 128, 0.0, P, 1 << 20, S) == INVALID
    assert L.quarot_kv_decode_attention(P, None, P, P, P, P, P, P2, 8, 8, 64, 64, 128, 128, 0.1,
                                        P, 1 << 20, S) == INVALID
    assert L.quarot_kv_decode_attention(*A, 0, 8, 64, 64, 128, 128, 0.1, None, 0, S) == OK
    need = L.quarot_kv_attention_workspace_size(64, 4096, 128)
    assert need == 64 * 16 * (128 + 2) * 4  # 16 chunks of 256 tokens per row
    assert L.quarot_kv_decode_attention(*A, 64, 64, 4096, 4096, 128, 128, 0.1, P, need - 4,
                                        S) == WORKSPACE
    assert L.quarot_kv_attention_workspace_size(4096, 4096, 128) == 0  # one chunk per row
    # swiglu prologue
    assert L.quarot_swiglu(P, P2, P, 12, S) == UNSUPPORTED
    assert L.quarot_swiglu(P, P2, P, -8, S) == INVALID
    assert L.quarot_swiglu(P, None, P, 16, S) == INVALID
    assert L.quarot_swiglu(P, P2, UNALIGNED, 16, S) == ALIGN
    assert L.quarot_swiglu(None, None, None, 0, S) == OK
    assert L.quarot_swiglu_quant_int4(P, P2, P, P2, -1, 128, 1.0, S) == INVALID
    assert L.quarot_swiglu_quant_int4(P, P2, P, P2, 4, 128, 0.0, S) == INVALID
    assert L.quarot_swiglu_quant_int4(P, P2, P, P2, 4, 100, 1.0, S) == UNSUPPORTED
    assert L.quarot_swiglu_quant_int4(P, None, P, P2, 4, 128, 1.0, S) == INVALID
    assert L.quarot_swiglu_quant_int4(P, UNALIGNED, P, P2, 4, 128, 1.0, S) == ALIGN
    assert L.quarot_swiglu_quant_int4(None, None, None, None, 0, 11008, 1.0, S) == OK
    # heads
    assert L.quarot_hadamard_heads(P, P2, 4, 48, 128, S) == UNSUPPORTED   # 48 heads
    assert L.quarot_hadamard_heads(P, P2, 4, 64, 96, S) == UNSUPPORTED    # head_dim 96
    assert L.quarot_hadamard_heads(P, P2, 4, 512, 128, S) == UNSUPPORTED  # n > 32768
    assert L.quarot_hadamard_heads(P, P2, 4, 1, 128, S) == UNSUPPORTED
    assert L.quarot_hadamard_heads(P, P2, 4, 0, 128, S) == INVALID
    assert L.quarot_hadamard_heads(P, None, 4, 64, 128, S) == INVALID
    assert L.quarot_hadamard_heads(P, UNALIGNED, 4, 64, 128, S) == ALIGN
    assert L.quarot_hadamard_heads(None, None, 0, 64, 128, S) == OK
    assert L.quarot_hadamard_heads_quant_int4(P, P2, None, 4, 64, 128, 1.0, S) == INVALID
    assert L.quarot_hadamard_heads_quant_int4(P, P2, P, 4, 64, 128, 2.0, S) == INVALID
    # group-wise
    G = L.quarot_quant_int4_grouped
    assert G(P, P2, P, 4, 128, 0, 1, 1.0, P, 1 << 20, S) == INVALID
    assert G(P, P2, P, 4, 128, 48, 1, 1.0, P, 1 << 20, S) == UNSUPPORTED   # not a power of two
    assert G(P, P2, P, 4, 128, 4, 1, 1.0, P, 1 << 20, S) == UNSUPPORTED    # below 8
    assert G(P, P2, P, 4, 1024, 1024, 1, 1.0, P, 1 << 20, S) == UNSUPPORTED  # above 512
    assert G(P, P2, P, 4, 384, 256, 0, 1.0, P, 1 << 20, S) == UNSUPPORTED  # does not divide n
    assert G(P, P2, P, 4, 128, 64, 1, 0.0, P, 1 << 20, S) == INVALID
    assert G(P, P2, P, 4, 128, 64, 1, 1.0, P, 100, S) == WORKSPACE
    assert G(P, P2, P, 4, 128, 64, 1, 1.0, None, 0, S) == WORKSPACE
    assert G(P, None, P, 4, 128, 64, 1, 1.0, P, 1 << 20, S) == INVALID
    assert G(P, P2, UNALIGNED, 4, 128, 64, 1, 1.0, P, 1 << 20, S) == ALIGN
    assert G(None, None, None, 0, 128, 64, 1, 1.0, None, 0, S) == OK
    assert L.quarot_quant_int4_grouped_workspace_size(4, 128, 1) == 4 * 128 * 4
    assert L.quarot_quant_int4_grouped_workspace_size(4, 128, 0) == 0
    GG = L.quarot_w4a4_gemm_grouped
    assert GG(P, P, P, P, P, 4, 4, 256, 32, S) == UNSUPPORTED
    assert GG(P, P, P, P, P, 4, 4, 256, 512, S) == UNSUPPORTED
    assert GG(P, P, P, P, P, 4, 4, 256, 0, S) == INVALID
    assert GG(P, P, P, P, P, 4, 4, 192, 64, S) == UNSUPPORTED   # K not a multiple of 128
    assert GG(P, P, P, P, P, 4, 4, 384, 256, S) == UNSUPPORTED  # K not a multiple of 256
    assert GG(P, None, P, P, P, 4, 4, 256, 128, S) == INVALID
    assert GG(P, P, P, P, UNALIGNED, 4, 4, 256, 128, S) == ALIGN
    assert GG(None, None, None, None, None, 0, 4, 256, 128, S) == OK
    G6 = L.quarot_w4a4_gemm_grouped_e3m2
    assert G6(P, P, P, P, P, 8, 8, 256, 64, S) == UNSUPPORTED    # one instruction spans 128 k
    assert G6(P, P, P, P, P, 12, 8, 256, 128, S) == UNSUPPORTED  # M not a multiple of 8
    assert G6(P, P, P, P, P, 8, 20, 256, 128, S) == UNSUPPORTED  # N not a multiple of 8
    assert G6(P, P, P, P, P, 8, 8, 384, 256, S) == UNSUPPORTED   # K not a multiple of 256
    assert G6(P, P, P, P, P, 8, 8, 256, 0, S) == INVALID
    assert G6(P, None, P, P, P, 8, 8, 256, 128, S) == INVALID
    assert G6(P, P, P, P, UNALIGNED, 8, 8, 256, 128, S) == ALIGN
    assert G6(None, None, None, None, None, 0, 8, 256, 128, S) == OK
    LG = L.quarot_linear_w4a4_grouped
    need = L.quarot_linear_w4a4_grouped_workspace_size(3, 256, 128, 1)
    assert need == 512 + 256 + 3 * 256 * 4  # codes, scales, binary32 rows (256-B rounded)
    assert L.quarot_linear_w4a4_grouped_workspace_size(3, 256, 128, 0) == 512 + 256
    assert LG(P, P, P, P, 4, 4, 256, 128, 1, 1.0, P, 10, S) == WORKSPACE
    assert LG(P, P, P, P, 4, 4, 256, 128, 1, 1.0, ctypes.c_void_p((1 << 20) + 16), 1 << 20,
              S) == ALIGN
    assert LG(P, P, P, P, 4, 4, 256, 96, 1, 1.0, P, 1 << 20, S) == UNSUPPORTED
    assert LG(P, P, P, P, 4, 4, 256, 128, 1, 1.5, P, 1 << 20, S) == INVALID
    assert LG(None, None, None, None, 0, 4, 256, 128, 1, 1.0, None, 0, S) == OK
    # e3m2 operand path
    assert L.quarot_pack_e3m2(P, P2, -1, 128, S) == INVALID
    assert L.quarot_pack_e3m2(P, P2, 4, 0, S) == INVALID
    assert L.quarot_pack_e3m2(P, P2, 4, 192, S) == UNSUPPORTED      # not a multiple of 128
    assert L.quarot_pack_e3m2(P, P2, 4, 65536 + 128, S) == UNSUPPORTED
    assert L.quarot_pack_e3m2(None, P2, 4, 128, S) == INVALID
    assert L.quarot_pack_e3m2(P, UNALIGNED, 4, 128, S) == ALIGN
    assert L.quarot_pack_e3m2(None, None, 0, 128, S) == OK
    E = L.quarot_w4a4_gemm_e3m2
    assert E(P, P, P, P, P, None, 4, 4, 192, S) == UNSUPPORTED       # K not a multiple of 128
    assert E(P, P, P, P, P, None, -1, 4, 128, S) == INVALID
    assert E(P, P, P, P, P, None, 4, 4, 0, S) == INVALID
    assert E(P, None, P, P, P, None, 4, 4, 128, S) == INVALID
    assert E(P, P, P, P, P, UNALIGNED, 4, 4, 128, S) == ALIGN
    assert E(None, None, None, None, None, None, 0, 4, 128, S) == OK
    QE = L.quarot_quant_int4_e3m2
    assert QE(P, P2, P2, 4, 128, 1, 0.0, S) == INVALID
    assert QE(P, P2, P2, 4, 64, 1, 1.0, S) == UNSUPPORTED           # not a multiple of 128
    assert QE(P, P2, P2, 4, 28 * 256, 1, 1.0, S) == UNSUPPORTED      # m = 28 needs 2^9 or 2^10
    assert QE(P, P2, P2, 4, 108 * 16, 1, 1.0, S) == UNSUPPORTED      # m = 108 needs 2^5 .. 2^7
    assert QE(P, P2, P2, 4, 172 * 128, 1, 1.0, S) == UNSUPPORTED     # m = 172 needs 2^5 or 2^6
    assert QE(P, None, P2, 4, 128, 1, 1.0, S) == INVALID
    assert QE(P, P2, UNALIGNED, 4, 128, 1, 1.0, S) == ALIGN
    assert QE(None, None, None, 0, 128, 1, 1.0, S) == OK
    LE = L.quarot_linear_e3m2
    assert L.quarot_linear_e3m2_workspace_size(3, 256) == 768 + 256
    assert L.quarot_linear_e3m2_workspace_size(3, 192) == 0
    assert LE(P, P, P, P, 4, 4, 128, 1, 1.0, P, 10, S) == WORKSPACE
    assert LE(P, P, P, P, 4, 4, 128, 1, 1.0, ctypes.c_void_p((1 << 20) + 16), 1 << 20,
              S) == ALIGN
    assert LE(P, P, P, P, 4, 4, 192, 1, 1.0, P, 1 << 20, S) == UNSUPPORTED
    assert LE(P, P, P, P, 4, 4, 128, 1, 1.5, P, 1 << 20, S) == INVALID
    assert LE(None, None, None, None, 0, 4, 128, 1, 1.0, None, 0, S) == OK
    SE = L.quarot_swiglu_quant_e3m2
    assert SE(P, P2, P, P2, 4, 8192 + 128, 1.0, S) == UNSUPPORTED
    assert SE(P, P2, P, P2, 4, 28672, 0.0, S) == INVALID
    assert SE(P, None, P, P2, 4, 28672, 1.0, S) == INVALID


def test_probe_arguments_rejected_before_device(PL):
    S = None
    assert PL.quarot_device_peaks(None, None) == INVALID
    for probe in (PL.quarot_mfma_probe, PL.quarot_mfma_probe_fp6):
        assert probe(P, 0, 10, S) == INVALID
        assert probe(P, 4, 0, S) == INVALID
        assert probe(P, (1 << 20) + 1, 10, S) == INVALID
        assert probe(None, 4, 10, S) == INVALID
        assert probe(UNALIGNED, 4, 10, S) == ALIGN


@pytest.mark.skipif(has_gpu(), reason="valid arguments would reach a real device")
def test_probe_no_device_reported(PL):
    cus, clk = ctypes.c_int(), ctypes.c_int()
    assert PL.quarot_device_peaks(ctypes.byref(cus), ctypes.byref(clk)) == NODEV
    assert PL.quarot_mfma_probe(P, 4, 10, None) == NODEV
    assert PL.quarot_mfma_probe_fp6(P, 4, 10, None) == NODEV


@pytest.mark.skipif(has_gpu(), reason="valid arguments would reach a real device")
def test_no_device_reported(L):
    """With valid arguments and no GPU the call stops at the device check
    (fake pointers are never dereferenced because nothing launches)."""
    assert L.quarot_quant_int4(P, P2, P2, 4, 128, 1, 1.0, None) == NODEV
    assert L.quarot_w4a4_gemm(P, P, P, P, P, None, 4, 4, 128, None) == NODEV
    assert L.quarot_swiglu_quant_int4(P, P2, P, P2, 4, 28672, 1.0, None) == NODEV
    assert L.quarot_hadamard_heads_quant_int4(P, P2, P, 4, 64, 128, 1.0, None) == NODEV
    assert L.quarot_quant_int4_grouped(P, P2, P, 4, 128, 128, 1, 1.0, P, 1 << 20,
                                       None) == NODEV
    assert L.quarot_w4a4_gemm_grouped(P, P, P, P, P, 4, 4, 256, 64, None) == NODEV
    assert L.quarot_w4a4_gemm_grouped_e3m2(P, P, P, P, P, 8, 8, 256, 128, None) == NODEV
    assert L.quarot_linear_w4a4_grouped(P, P, P, P, 4, 4, 256, 256, 1, 1.0, P, 1 << 20,
                                        None) == NODEV
    assert L.quarot_pack_e3m2(P, P2, 4, 128, None) == NODEV
    assert L.quarot_w4a4_gemm_e3m2(P, P, P, P, P, None, 4, 4, 128, None) == NODEV
    assert L.quarot_quant_int4_e3m2(P, P2, P2, 4, 28672, 1, 1.0, None) == NODEV
    assert L.quarot_quant_int4_e3m2(P, P2, P2, 4, 11008, 1, 1.0, None) == NODEV
    assert L.quarot_quant_int4_e3m2(P, P2, P2, 4, 13824, 1, 1.0, None) == NODEV
    assert L.quarot_linear_e3m2(P, P, P, P, 4, 4, 8192, 1, 1.0, P, 1 << 20, None) == NODEV
    assert L.quarot_swiglu_quant_e3m2(P, P2, P, P2, 4, 28672, 1.0, None) == NODEV
    assert L.quarot_linear_e3m2_scratch(P, P, P, P, 2048, 4, 28672, 1, 1.0, None) == NODEV


def test_binding_rejects_host_tensors():
    import torch
    x = torch.zeros(4, 128, dtype=torch.float16)
    with pytest.raises(ValueError):
        q.quarot_hadamard(x, y=torch.zeros_like(x))
    with pytest.raises(TypeError):
        q.quarot_hadamard(x.float(), y=torch.zeros_like(x))


HIP_ERROR_LAUNCH_FAILURE = 719  # hipErrorLaunchFailure


@pytest.fixture
def fake_hip_error(monkeypatch):
    def arm(call):
        monkeypatch.setenv("QUAROT_FAKE_HIP_ERROR", call)
    yield arm
    monkeypatch.delenv("QUAROT_FAKE_HIP_ERROR", raising=False)


def test_fake_hip_error_hook(L, fake_hip_error):
    """QUAROT_FAKE_HIP_ERROR=<entry point> makes exactly that entry point
    report QUAROT_ERR_HIP after its argument checks and before any device
    work; quarot_last_hip_error() returns the code; other entry points and
    invalid arguments are unaffected.  Host-only: nothing launches."""
    nodev_or_ok = (NODEV, OK)
    fake_hip_error("quarot_linear")
    assert L.quarot_linear(P, P, P, P, 4, 4, 128, 1, 1.0, P, 1 << 20, None) == HIP
    assert L.quarot_last_hip_error() == HIP_ERROR_LAUNCH_FAILURE
    assert L.quarot_linear(P, P, P, P, 4, 4, 128, 1, 0.0, P, 1 << 20, None) == INVALID
    assert L.quarot_linear(P, P, P, P, 4, 4, 128, 1, 1.0, P, 16, None) == WORKSPACE
    if not has_gpu():
        assert L.quarot_quant_int4(P, P2, P2, 4, 128, 1, 1.0, None) in nodev_or_ok
    for call, invoke in (
            ("quarot_hadamard", lambda: L.quarot_hadamard(P, P2, 4, 128, None)),
            ("quarot_w4a4_gemm_e3m2",
             lambda: L.quarot_w4a4_gemm_e3m2(P, P, P, P, P, None, 4, 4, 128, None)),
            ("quarot_hadamard_heads_quant_int4",
             lambda: L.quarot_hadamard_heads_quant_int4(P, P2, P, 4, 64, 128, 1.0, None)),
            ("quarot_kv_decode_attention",
             lambda: L.quarot_kv_decode_attention(P, P, P, P, P, P, P, P2, 4, 4, 64, 64, 128,
                                                  128, 0.1, P, 1 << 24, None))):
        fake_hip_error(call)
        assert invoke() == HIP, call
        assert L.quarot_last_hip_error() == HIP_ERROR_LAUNCH_FAILURE
    # the binding turns it into QuarotError carrying both codes
    fake_hip_error("quarot_quant_int4")
    with pytest.raises(q.QuarotError) as ei:
        q._check("quarot_quant_int4", L.quarot_quant_int4(P, P2, P2, 4, 128, 1, 1.0, None))
    assert ei.value.status == HIP and ei.value.hip_error == HIP_ERROR_LAUNCH_FAILURE


def test_last_hip_error_is_per_thread(L, fake_hip_error):
    import threading
    fake_hip_error("quarot_hadamard")
    assert L.quarot_hadamard(P, P2, 4, 128, None) == HIP
    seen = []
    t = threading.Thread(target=lambda: seen.append(L.quarot_last_hip_error()))
    t.start()
    t.join()
    assert seen == [0] and L.quarot_last_hip_error() == HIP_ERROR_LAUNCH_FAILURE


def test_scratch_entry_point_limits(L):
    """The allocation-free layer refuses sizes beyond its fixed array
    (64 MiB of codes and scales) before any device work, and otherwise
    validates like quarot_linear_e3m2."""
    SE = L.quarot_linear_e3m2_scratch
    assert q.SCRATCH_BYTES == 64 << 20
    assert L.quarot_linear_e3m2_workspace_size(16384, 8192) > q.SCRATCH_BYTES
    assert SE(P, P, P, P, 16384, 4, 8192, 1, 1.0, None) == WORKSPACE
    assert SE(P, P, P, P, 4, 4, 8192, 1, 0.0, None) == INVALID
    assert SE(P, P, P, P, 4, 4, 192, 1, 1.0, None) == UNSUPPORTED
    assert SE(None, P, P, P, 4, 4, 8192, 1, 1.0, None) == INVALID
    assert SE(UNALIGNED, P, P, P, 4, 4, 8192, 1, 1.0, None) == ALIGN
    assert SE(None, None, None, None, 0, 4, 8192, 1, 1.0, None) == OK
