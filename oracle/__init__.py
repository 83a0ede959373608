"""CPU oracle for the QuaRot W4A4 linear-layer hot path.

TEST INFRASTRUCTURE ONLY.  The oracle is a plain C implementation
(``quarot_oracle.c``) of what the GPU path computes, loaded here with ctypes.
Only the test suite, the smoke check and the bench's CPU-baseline leg may
import this package; the product path never does.

Every function takes and returns numpy arrays.  fp16 data travels as numpy
``float16`` (its bits are passed to C as ``uint16``); rotations stay fp32.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "quarot_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liborc.so")

# -ffp-contract=off: every written a*b+c stays two rounded operations.
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
          "-fPIC", "-shared", "-Wall", "-Wextra"]


def build(force: bool = True) -> str:
    """Compile the oracle into ``oracle/liborc.so`` with gcc."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.run(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I = ctypes.c_int
_F = ctypes.c_float

_SIGS = {
    "orc_f16_to_f32_array": (None, [_P, _P, _I64]),
    "orc_f32_to_f16_array": (None, [_P, _P, _I64]),
    "orc_f64_to_f16_array": (None, [_P, _P, _I64]),
    "orc_sylvester_entry": (_I, [_I64, _I64]),
    "orc_hm_table": (_I, [_I, _P]),
    "orc_hadamard_factor": (_I, [_I64, _P, _P]),
    "orc_rotation_scale": (_F, [_I64]),
    "orc_rotate_f32": (_I, [_P, _P, _I64, _I64]),
    "orc_rotate_f16": (_I, [_P, _P, _I64, _I64]),
    "orc_hadamard_f16": (_I, [_P, _P, _I64, _I64]),
    "orc_quant_sym_f32": (_I, [_P, _P, _P, _I64, _I64, _F]),
    "orc_quant_int4": (_I, [_P, _P, _P, _I64, _I64, _I, _F]),
    "orc_gemm_i32": (_I, [_P, _P, _P, _I64, _I64, _I64]),
    "orc_dequant": (_I, [_P, _P, _P, _P, _I64, _I64]),
    "orc_linear": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I64, _I, _F]),
    "orc_kv_quant": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _F]),
    "orc_kv_dequant": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I]),
    "orc_silu_f32": (_F, [_F]),
    "orc_swiglu_f16": (_I, [_P, _P, _P, _I64]),
    "orc_swiglu_quant_int4": (_I, [_P, _P, _P, _P, _I64, _I64, _I, _F]),
    "orc_heads_f16": (_I, [_P, _P, _I64, _I64, _I64]),
    "orc_heads_quant_int4": (_I, [_P, _P, _P, _I64, _I64, _I64, _F]),
    "orc_kv_append": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I64, _I64, _I, _F]),
    "orc_kv_attention": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _I64,
                              _I64, _F]),
    "orc_quant_sym8_f32": (_I, [_P, _P, _P, _I64, _I64, _F, _I]),
    "orc_quant_int8": (_I, [_P, _P, _P, _I64, _I64, _I, _F, _I]),
    "orc_gemm_i8": (_I, [_P, _P, _P, _I64, _I64, _I64]),
    "orc_quant_search": (_I, [_P, _P, _P, _P, _I64, _I64, _I, _I, _I]),
    "orc_quant_int4_grouped": (_I, [_P, _P, _P, _I64, _I64, _I64, _I, _F]),
    "orc_gemm_grouped": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I64, _I64]),
    "orc_set_threads": (None, [_I]),
    "orc_max_threads": (_I, []),
}


def lib():
    """Load (building first if needed) the oracle shared library.  The
    environment variable QUAROT_ORACLE_LIB names another build of the same
    source to load instead (the sanitizer test uses it)."""
    global _lib
    if _lib is None:
        path = os.environ.get("QUAROT_ORACLE_LIB")
        if not path:
            path = _LIB_PATH
            if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
                build()
        L = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(st: int, what: str):
    if st != 0:
        raise OracleError(f"{what} failed with status {st}")


def _f16(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float16))


def _u16(a16: np.ndarray) -> np.ndarray:
    return a16.view(np.uint16)


# -- number formats ---------------------------------------------------------

def f16_to_f32(h: np.ndarray) -> np.ndarray:
    h = _f16(h)
    out = np.empty(h.shape, np.float32)
    lib().orc_f16_to_f32_array(_ptr(_u16(h)), _ptr(out), h.size)
    return out


def f32_to_f16(f: np.ndarray) -> np.ndarray:
    f = np.ascontiguousarray(np.asarray(f, dtype=np.float32))
    out = np.empty(f.shape, np.uint16)
    lib().orc_f32_to_f16_array(_ptr(f), _ptr(out), f.size)
    return out.view(np.float16)


def f64_to_f16(d: np.ndarray) -> np.ndarray:
    """binary64 -> binary16 rounded once (nearest even)."""
    d = np.ascontiguousarray(np.asarray(d, dtype=np.float64))
    out = np.empty(d.shape, np.uint16)
    lib().orc_f64_to_f16_array(_ptr(d), _ptr(out), d.size)
    return out.view(np.float16)


# -- Hadamard matrices ------------------------------------------------------

def hadamard_factor(n: int):
    """(k, m) with n = 2**k * m, or None if n has no compiled factorization."""
    k = ctypes.c_int()
    m = ctypes.c_int()
    st = lib().orc_hadamard_factor(n, ctypes.byref(k), ctypes.byref(m))
    return None if st else (k.value, m.value)


def hm_table(m: int) -> np.ndarray:
    out = np.empty((m, m), np.int8)
    _check(lib().orc_hm_table(m, _ptr(out)), f"hm_table({m})")
    return out


def sylvester_entry(i: int, j: int) -> int:
    return lib().orc_sylvester_entry(i, j)


def rotation_scale(n: int) -> np.float32:
    return np.float32(lib().orc_rotation_scale(n))


# -- rotation ---------------------------------------------------------------

def rotate_f32(t: np.ndarray) -> np.ndarray:
    t = np.ascontiguousarray(t, dtype=np.float32)
    rows, n = t.shape
    y = np.empty_like(t)
    _check(lib().orc_rotate_f32(_ptr(t), _ptr(y), rows, n), "rotate_f32")
    return y


def rotate_f16(x: np.ndarray) -> np.ndarray:
    x = _f16(x)
    rows, n = x.shape
    y = np.empty((rows, n), np.float32)
    _check(lib().orc_rotate_f16(_ptr(_u16(x)), _ptr(y), rows, n), "rotate_f16")
    return y


def hadamard(x: np.ndarray) -> np.ndarray:
    """Standalone online Hadamard: fp16 rows in, RN16 of the rotation out."""
    x = _f16(x)
    rows, n = x.shape
    y = np.empty((rows, n), np.uint16)
    _check(lib().orc_hadamard_f16(_ptr(_u16(x)), _ptr(y), rows, n), "hadamard")
    return y.view(np.float16)


# -- quantization -----------------------------------------------------------

def quant_sym_f32(y: np.ndarray, clip: float = 1.0):
    y = np.ascontiguousarray(y, dtype=np.float32)
    rows, n = y.shape
    q = np.empty((rows, n // 2), np.uint8)
    s = np.empty(rows, np.uint16)
    _check(lib().orc_quant_sym_f32(_ptr(y), _ptr(q), _ptr(s), rows, n, clip),
           "quant_sym_f32")
    return q, s.view(np.float16)


def quant_int4(x: np.ndarray, rotate: bool = True, clip: float = 1.0):
    """fp16 rows -> (packed codes uint8 [rows, n/2], fp16 scales [rows])."""
    x = _f16(x)
    rows, n = x.shape
    q = np.empty((rows, n // 2), np.uint8)
    s = np.empty(rows, np.uint16)
    _check(lib().orc_quant_int4(_ptr(_u16(x)), _ptr(q), _ptr(s), rows, n,
                                int(rotate), clip), "quant_int4")
    return q, s.view(np.float16)


def quant_sym8_f32(y: np.ndarray, clip: float = 1.0, bits: int = 8):
    y = np.ascontiguousarray(y, dtype=np.float32)
    rows, n = y.shape
    q = np.empty((rows, n), np.int8)
    s = np.empty(rows, np.uint16)
    _check(lib().orc_quant_sym8_f32(_ptr(y), _ptr(q), _ptr(s), rows, n, clip, bits),
           "quant_sym8_f32")
    return q, s.view(np.float16)


def quant_int8(x: np.ndarray, rotate: bool = True, clip: float = 1.0, bits: int = 8):
    """fp16 rows -> (int8 codes [rows, n] with 2^(bits-1) - 1 levels a side,
    fp16 scales [rows])."""
    x = _f16(x)
    rows, n = x.shape
    q = np.empty((rows, n), np.int8)
    s = np.empty(rows, np.uint16)
    _check(lib().orc_quant_int8(_ptr(_u16(x)), _ptr(q), _ptr(s), rows, n, int(rotate), clip,
                                bits), "quant_int8")
    return q, s.view(np.float16)


def quant_search(w: np.ndarray, rotate: bool = True, bits: int = 4, n_candidates: int = 20):
    """Per-row clip search: (codes, scales, chosen clip per row).  Codes are
    packed nibbles [rows, n/2] for bits = 4, int8 [rows, n] for 6 and 8."""
    w = _f16(w)
    rows, n = w.shape
    q = np.empty((rows, n // 2), np.uint8) if bits == 4 else np.empty((rows, n), np.int8)
    s = np.empty(rows, np.uint16)
    c = np.empty(rows, np.float32)
    _check(lib().orc_quant_search(_ptr(_u16(w)), _ptr(q), _ptr(s), _ptr(c), rows, n,
                                  int(rotate), bits, n_candidates), "quant_search")
    return q, s.view(np.float16), c


def quant_int4_grouped(x: np.ndarray, group: int = 128, rotate: bool = True, clip: float = 1.0):
    """Group-wise int4: (codes [rows, n/2], scales fp16 group-major [n/group, rows])."""
    x = _f16(x)
    rows, n = x.shape
    q = np.empty((rows, n // 2), np.uint8)
    s = np.empty((n // group, rows), np.uint16)
    _check(lib().orc_quant_int4_grouped(_ptr(_u16(x)), _ptr(q), _ptr(s), rows, n, group,
                                        int(rotate), clip), "quant_int4_grouped")
    return q, s.view(np.float16)


def gemm_grouped(xq: np.ndarray, sx: np.ndarray, wq: np.ndarray, sw: np.ndarray,
                 group: int = 128) -> np.ndarray:
    """Group-wise W4A4 product with per-group dequant; sx [K/G, M], sw [K/G, N]."""
    xq = np.ascontiguousarray(xq, dtype=np.uint8)
    wq = np.ascontiguousarray(wq, dtype=np.uint8)
    sx = _f16(sx)
    sw = _f16(sw)
    M, Kh = xq.shape
    N = wq.shape[0]
    y = np.empty((M, N), np.uint16)
    _check(lib().orc_gemm_grouped(_ptr(xq), _ptr(_u16(sx)), _ptr(wq), _ptr(_u16(sw)), _ptr(y),
                                  M, N, 2 * Kh, group), "gemm_grouped")
    return y.view(np.float16)


def gemm_i8(xq: np.ndarray, wq: np.ndarray) -> np.ndarray:
    xq = np.ascontiguousarray(xq, dtype=np.int8)
    wq = np.ascontiguousarray(wq, dtype=np.int8)
    M, K = xq.shape
    N, K2 = wq.shape
    assert K == K2
    acc = np.empty((M, N), np.int32)
    _check(lib().orc_gemm_i8(_ptr(xq), _ptr(wq), _ptr(acc), M, N, K), "gemm_i8")
    return acc


def gemm_i32(xq: np.ndarray, wq: np.ndarray) -> np.ndarray:
    xq = np.ascontiguousarray(xq, dtype=np.uint8)
    wq = np.ascontiguousarray(wq, dtype=np.uint8)
    M, Kh = xq.shape
    N, Kh2 = wq.shape
    assert Kh == Kh2
    acc = np.empty((M, N), np.int32)
    _check(lib().orc_gemm_i32(_ptr(xq), _ptr(wq), _ptr(acc), M, N, 2 * Kh), "gemm_i32")
    return acc


def dequant(acc: np.ndarray, sx: np.ndarray, sw: np.ndarray) -> np.ndarray:
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    sx = _f16(sx)
    sw = _f16(sw)
    M, N = acc.shape
    y = np.empty((M, N), np.uint16)
    _check(lib().orc_dequant(_ptr(acc), _ptr(_u16(sx)), _ptr(_u16(sw)), _ptr(y), M, N),
           "dequant")
    return y.view(np.float16)


def linear(x: np.ndarray, wq: np.ndarray, sw: np.ndarray, rotate: bool = True,
           clip: float = 1.0, want_acc: bool = False):
    """The whole W4A4 layer; returns y (and the int32 accumulators)."""
    x = _f16(x)
    wq = np.ascontiguousarray(wq, dtype=np.uint8)
    sw = _f16(sw)
    M, K = x.shape
    N = wq.shape[0]
    y = np.empty((M, N), np.uint16)
    acc = np.empty((M, N), np.int32) if want_acc else None
    _check(lib().orc_linear(_ptr(_u16(x)), _ptr(wq), _ptr(_u16(sw)), _ptr(y),
                            _ptr(acc) if want_acc else None, M, N, K, int(rotate), clip),
           "linear")
    y = y.view(np.float16)
    return (y, acc) if want_acc else y


def prepare_weight(w: np.ndarray, rotate: bool = True, clip: float = 1.0):
    """Offline weight prep: rotate each output-channel row like an activation
    row and quantize it per row (per output channel)."""
    return quant_int4(w, rotate=rotate, clip=clip)


# -- KV cache ---------------------------------------------------------------

def kv_quant(kv: np.ndarray, group: int = 128, rotate: bool = True, clip: float = 0.95):
    """kv [rows, D] fp16 -> (codes uint8 [rows, D/2], scale, zero fp16 [rows, D/group])."""
    kv = _f16(kv)
    rows, D = kv.shape
    q = np.empty((rows, D // 2), np.uint8)
    sc = np.empty((rows, D // group), np.uint16)
    ze = np.empty((rows, D // group), np.uint16)
    _check(lib().orc_kv_quant(_ptr(_u16(kv)), _ptr(q), _ptr(sc), _ptr(ze), rows, D, group,
                              int(rotate), clip), "kv_quant")
    return q, sc.view(np.float16), ze.view(np.float16)


def kv_dequant(q: np.ndarray, scale: np.ndarray, zero: np.ndarray, group: int = 128,
               inverse_rotate: bool = False) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.uint8)
    scale = _f16(scale)
    zero = _f16(zero)
    rows, Dh = q.shape
    D = 2 * Dh
    out = np.empty((rows, D), np.uint16)
    _check(lib().orc_kv_dequant(_ptr(q), _ptr(_u16(scale)), _ptr(_u16(zero)), _ptr(out),
                                rows, D, group, int(inverse_rotate)), "kv_dequant")
    return out.view(np.float16)


def kv_append(kv_new: np.ndarray, q_cache: np.ndarray, scale_cache: np.ndarray,
              zero_cache: np.ndarray, pos: int, group: int = 128, rotate: bool = True,
              clip: float = 0.95):
    """Quantize kv_new [rows, D] into caches [rows, s_max, ...] at token pos
    (in place on copies, which are returned)."""
    kv_new = _f16(kv_new)
    rows, D = kv_new.shape
    qc = np.ascontiguousarray(q_cache, dtype=np.uint8).copy()
    sc = _f16(scale_cache).copy()
    zc = _f16(zero_cache).copy()
    s_max = qc.shape[1]
    _check(lib().orc_kv_append(_ptr(_u16(kv_new)), _ptr(qc), _ptr(_u16(sc)), _ptr(_u16(zc)),
                               rows, s_max, pos, D, group, int(rotate), clip), "kv_append")
    return qc, sc, zc


def kv_attention(q: np.ndarray, k: tuple, v: tuple, seq_len: int, group: int = 128,
                 sm_scale: float = None) -> np.ndarray:
    """Decode attention of q [nq, D] over 4-bit caches k = (codes [nkv, s_max,
    D/2], scale, zero [nkv, s_max, D/group]) and v alike; fp64 inside."""
    q = _f16(q)
    nq, D = q.shape
    kc, ks, kz = (np.ascontiguousarray(k[0], dtype=np.uint8), _f16(k[1]), _f16(k[2]))
    vc, vs, vz = (np.ascontiguousarray(v[0], dtype=np.uint8), _f16(v[1]), _f16(v[2]))
    nkv, s_max = kc.shape[0], kc.shape[1]
    if sm_scale is None:
        sm_scale = 1.0 / np.sqrt(D)
    out = np.empty((nq, D), np.uint16)
    _check(lib().orc_kv_attention(_ptr(_u16(q)), _ptr(kc), _ptr(_u16(ks)), _ptr(_u16(kz)),
                                  _ptr(vc), _ptr(_u16(vs)), _ptr(_u16(vz)), _ptr(out), nq, nkv,
                                  s_max, seq_len, D, group, float(sm_scale)), "kv_attention")
    return out.view(np.float16)


# -- prologues of the two online-Hadamard sites -----------------------------

def silu_f32(g: float) -> np.float32:
    """The binary32 SiLU recipe (scalar)."""
    return np.float32(lib().orc_silu_f32(float(np.float32(g))))


def swiglu(gate: np.ndarray, up: np.ndarray) -> np.ndarray:
    """h = RN16(RN(silu(gate) * up)), elementwise, fp16 in and out."""
    g = _f16(gate)
    u = _f16(up)
    assert g.shape == u.shape
    h = np.empty(g.shape, np.uint16)
    _check(lib().orc_swiglu_f16(_ptr(_u16(g)), _ptr(_u16(u)), _ptr(h), g.size), "swiglu")
    return h.view(np.float16)


def swiglu_quant_int4(gate: np.ndarray, up: np.ndarray, rotate: bool = True,
                      clip: float = 1.0):
    """quant_int4(swiglu(gate, up)) per row: the down-projection input."""
    g = _f16(gate)
    u = _f16(up)
    rows, n = g.shape
    q = np.empty((rows, n // 2), np.uint8)
    s = np.empty(rows, np.uint16)
    _check(lib().orc_swiglu_quant_int4(_ptr(_u16(g)), _ptr(_u16(u)), _ptr(q), _ptr(s), rows,
                                       n, int(rotate), clip), "swiglu_quant_int4")
    return q, s.view(np.float16)


def heads_f32(z: np.ndarray, n_heads: int) -> np.ndarray:
    """Rows z [rows, n_heads * head_dim] (head-major) -> binary32
    z (H_nh (x) I) / sqrt(nh)."""
    z = _f16(z)
    rows, n = z.shape
    y = np.empty((rows, n), np.float32)
    _check(lib().orc_heads_f16(_ptr(_u16(z)), _ptr(y), rows, n_heads, n // n_heads), "heads")
    return y


def hadamard_heads(z: np.ndarray, n_heads: int) -> np.ndarray:
    """fp16 rows in, RN16 of the head-wise rotation out."""
    return f32_to_f16(heads_f32(z, n_heads))


def heads_quant_int4(z: np.ndarray, n_heads: int, clip: float = 1.0):
    z = _f16(z)
    rows, n = z.shape
    q = np.empty((rows, n // 2), np.uint8)
    s = np.empty(rows, np.uint16)
    _check(lib().orc_heads_quant_int4(_ptr(_u16(z)), _ptr(q), _ptr(s), rows, n_heads,
                                      n // n_heads, clip), "heads_quant_int4")
    return q, s.view(np.float16)


# -- packing helpers (test-side views of the packed format) -----------------

def unpack_int4(q: np.ndarray) -> np.ndarray:
    """Packed signed nibbles [rows, n/2] -> int8 codes [rows, n]."""
    q = np.asarray(q, dtype=np.uint8)
    lo = (q & 0xF).astype(np.int8)
    hi = (q >> 4).astype(np.int8)
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(q.shape[:-1] + (q.shape[-1] * 2,), np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


def unpack_uint4(q: np.ndarray) -> np.ndarray:
    q = np.asarray(q, dtype=np.uint8)
    out = np.empty(q.shape[:-1] + (q.shape[-1] * 2,), np.uint8)
    out[..., 0::2] = q & 0xF
    out[..., 1::2] = q >> 4
    return out


def set_threads(n: int):
    lib().orc_set_threads(n)


def max_threads() -> int:
    return lib().orc_max_threads()
