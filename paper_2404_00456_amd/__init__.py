"""MI355X (gfx950) QuaRot W4A4 rotated-linear hot path.

A thin ctypes binding over ``libquarot.so`` (HIP kernels behind the C ABI in
``include/quarot.h``).  Every function here only marshals arguments: torch
tensors provide device memory and the current stream, and every step of the
path runs in the library's kernels.  There is no CPU fallback; if the
library is missing or no gfx950 device is present the calls raise.

Paper: Ashkboos et al., "QuaRot: Outlier-Free 4-Bit Inference in Rotated
LLMs", arXiv 2404.00456 (§3.1 Hadamard construction, §4 Stage 1b/1d/2b,
§5 Setup, App. A.10 4-bit linear layer).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch  # first: the library then binds to torch's HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libquarot.so")
# the measurement library beside it (include/quarot_probe.h)
PROBE_LIB_PATH = os.path.join(_HERE, "libquarot_probe.so")

STATUS = {
    0: "QUAROT_OK",
    1: "QUAROT_ERR_INVALID_ARG",
    2: "QUAROT_ERR_UNSUPPORTED_SIZE",
    3: "QUAROT_ERR_ALIGNMENT",
    4: "QUAROT_ERR_WORKSPACE",
    5: "QUAROT_ERR_NO_DEVICE",
    6: "QUAROT_ERR_HIP",
}

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I = ctypes.c_int
_F = ctypes.c_float

# name -> (restype, argtypes), exactly the declarations of include/quarot.h
SIGNATURES = {
    "quarot_status_string": (ctypes.c_char_p, [_I]),
    "quarot_last_hip_error": (_I, []),
    "quarot_version": (_I, []),
    "quarot_hadamard_factor": (_I, [_I64, _P, _P]),
    "quarot_hadamard_factor_table": (_I, [_I, _P]),
    "quarot_hadamard": (_I, [_P, _P, _I64, _I64, _P]),
    "quarot_quant_int4": (_I, [_P, _P, _P, _I64, _I64, _I, _F, _P]),
    "quarot_w4a4_gemm": (_I, [_P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P]),
    "quarot_pack_e3m2": (_I, [_P, _P, _I64, _I64, _P]),
    "quarot_w4a4_gemm_e3m2": (_I, [_P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P]),
    "quarot_quant_int4_e3m2": (_I, [_P, _P, _P, _I64, _I64, _I, _F, _P]),
    "quarot_linear_e3m2_workspace_size": (ctypes.c_size_t, [_I64, _I64]),
    "quarot_linear_e3m2": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _F, _P, ctypes.c_size_t,
                                _P]),
    "quarot_linear_e3m2_scratch": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _F, _P]),
    "quarot_swiglu_quant_e3m2": (_I, [_P, _P, _P, _P, _I64, _I64, _F, _P]),
    "quarot_linear_workspace_size": (ctypes.c_size_t, [_I64, _I64]),
    "quarot_linear": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _F, _P, ctypes.c_size_t, _P]),
    "quarot_quant_int8": (_I, [_P, _P, _P, _I64, _I64, _I, _F, _I, _P]),
    "quarot_w8a8_gemm": (_I, [_P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P]),
    "quarot_linear_w8a8_workspace_size": (ctypes.c_size_t, [_I64, _I64]),
    "quarot_linear_w8a8": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _F, _I, _P,
                                ctypes.c_size_t, _P]),
    "quarot_quant_search_workspace_size": (ctypes.c_size_t, [_I64, _I64, _I]),
    "quarot_quant_search": (_I, [_P, _P, _P, _P, _I64, _I64, _I, _I, _I, _P, ctypes.c_size_t,
                                 _P]),
    "quarot_quant_int4_grouped_workspace_size": (ctypes.c_size_t, [_I64, _I64, _I]),
    "quarot_quant_int4_grouped": (_I, [_P, _P, _P, _I64, _I64, _I64, _I, _F, _P,
                                       ctypes.c_size_t, _P]),
    "quarot_w4a4_gemm_grouped": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _P]),
    "quarot_w4a4_gemm_grouped_e3m2": (_I, [_P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _P]),
    "quarot_linear_w4a4_grouped_workspace_size": (ctypes.c_size_t, [_I64, _I64, _I64, _I]),
    "quarot_linear_w4a4_grouped": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I64, _I, _F, _P,
                                        ctypes.c_size_t, _P]),
    "quarot_swiglu": (_I, [_P, _P, _P, _I64, _P]),
    "quarot_swiglu_quant_int4": (_I, [_P, _P, _P, _P, _I64, _I64, _F, _P]),
    "quarot_hadamard_heads": (_I, [_P, _P, _I64, _I64, _I64, _P]),
    "quarot_hadamard_heads_quant_int4": (_I, [_P, _P, _P, _I64, _I64, _I64, _F, _P]),
    "quarot_kv_quant": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _F, _P]),
    "quarot_kv_dequant": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I, _P]),
    "quarot_kv_append": (_I, [_P, _P, _P, _P, _I64, _I64, _I64, _I64, _I64, _I, _F, _P]),
    "quarot_kv_attention_workspace_size": (ctypes.c_size_t, [_I64, _I64, _I64]),
    "quarot_kv_decode_attention": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I64,
                                        _I64, _I64, _F, _P, ctypes.c_size_t, _P]),
}

# name -> (restype, argtypes), exactly the declarations of include/quarot_probe.h
PROBE_SIGNATURES = {
    "quarot_device_peaks": (_I, [_P, _P]),
    "quarot_mfma_probe": (_I, [_P, _I64, _I, _P]),
    "quarot_mfma_probe_fp6": (_I, [_P, _I64, _I, _P]),
    "quarot_probe_last_hip_error": (_I, []),
}

_lib = None
_probe_lib = None


class QuarotError(RuntimeError):
    def __init__(self, call: str, status: int, hip_error: int = 0):
        self.status = status
        self.hip_error = hip_error
        msg = f"{call} failed: {STATUS.get(status, status)}"
        if hip_error:
            msg += f" (hipError {hip_error})"
        super().__init__(msg)


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2404_00456_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def probe_lib() -> ctypes.CDLL:
    """The loaded measurement library; raises if it has not been built."""
    global _probe_lib
    if _probe_lib is None:
        if not os.path.exists(PROBE_LIB_PATH):
            raise RuntimeError(f"{PROBE_LIB_PATH} is missing: build it with "
                               "`python -m paper_2404_00456_amd.build`")
        L = ctypes.CDLL(PROBE_LIB_PATH)
        for name, (res, args) in PROBE_SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _probe_lib = L
    return _probe_lib


def _check(call: str, st: int):
    if st != 0:
        raise QuarotError(call, st, lib().quarot_last_hip_error() if st == 6 else 0)


def _check_probe(call: str, st: int):
    if st != 0:
        raise QuarotError(call, st, probe_lib().quarot_probe_last_hip_error() if st == 6 else 0)


def _ptr(t: Optional[torch.Tensor], dtype: torch.dtype, name: str):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream: Optional[torch.cuda.Stream]):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _rows(t: torch.Tensor, n: int) -> int:
    return t.numel() // n if n else 0


# Shape checks against the sizes a call is given: the library trusts its
# pointers, so a tensor smaller than the sizes say would be read or written
# past its end.  They raise before anything is launched.

def _shape(t: Optional[torch.Tensor], shape, name: str):
    if t is not None and tuple(t.shape) != tuple(int(d) for d in shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _numel(t: Optional[torch.Tensor], n: int, name: str):
    if t is not None and t.numel() != n:
        raise ValueError(f"{name} must hold {n} elements, got {t.numel()}")


def _ndim(t: torch.Tensor, d: int, name: str):
    if t.dim() != d:
        raise ValueError(f"{name} must be {d}-D, got shape {tuple(t.shape)}")


def _group(group: int, D: int, name: str = "group"):
    if group <= 0 or D % group:
        raise ValueError(f"{name} must be a positive divisor of {D}, got {group}")


# -- host-side queries ------------------------------------------------------

def quarot_version() -> int:
    return lib().quarot_version()


def quarot_hadamard_factor(n: int) -> Optional[Tuple[int, int]]:
    k = ctypes.c_int()
    m = ctypes.c_int()
    st = lib().quarot_hadamard_factor(n, ctypes.byref(k), ctypes.byref(m))
    return None if st else (k.value, m.value)


def quarot_device_peaks() -> Tuple[int, int]:
    """(compute units, peak shader clock in kHz) of the current device."""
    cus = ctypes.c_int()
    clk = ctypes.c_int()
    _check_probe("quarot_device_peaks",
                 probe_lib().quarot_device_peaks(ctypes.byref(cus), ctypes.byref(clk)))
    return cus.value, clk.value


def quarot_mfma_probe(out: torch.Tensor, blocks: int, iters: int,
                      stream: Optional[torch.cuda.Stream] = None) -> int:
    """Enqueue the int8-MFMA-only probe; returns its number of int ops
    (2 per multiply-add).  out: int32 device tensor of blocks * 512."""
    if out.numel() < blocks * 512:
        raise ValueError("out must hold blocks * 512 int32")
    _check_probe("quarot_mfma_probe", probe_lib().quarot_mfma_probe(
        _ptr(out, torch.int32, "out"), int(blocks), int(iters), _stream(stream)))
    return blocks * 8 * iters * 32 * 16384 * 2  # waves x MFMAs x multiply-adds x 2


def quarot_mfma_probe_fp6(out: torch.Tensor, blocks: int, iters: int,
                          stream: Optional[torch.cuda.Stream] = None) -> int:
    """Enqueue the e3m2 fp6-MFMA-only probe; returns its number of ops (2
    per multiply-add).  out: int32 device tensor of blocks * 512."""
    if out.numel() < blocks * 512:
        raise ValueError("out must hold blocks * 512 int32")
    _check_probe("quarot_mfma_probe_fp6", probe_lib().quarot_mfma_probe_fp6(
        _ptr(out, torch.int32, "out"), int(blocks), int(iters), _stream(stream)))
    return blocks * 8 * iters * 32 * 32768 * 2


def quarot_hadamard_factor_table(m: int):
    import numpy as np
    out = np.empty((m, m), np.int8)
    _check("quarot_hadamard_factor_table",
           lib().quarot_hadamard_factor_table(m, out.ctypes.data_as(ctypes.c_void_p)))
    return out


def quarot_linear_workspace_size(M: int, K: int) -> int:
    return int(lib().quarot_linear_workspace_size(M, K))


# -- device calls -----------------------------------------------------------

def quarot_hadamard(x: torch.Tensor, y: Optional[torch.Tensor] = None,
                    stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """y = RN16(x . H_n / sqrt(n)) row by row; x fp16 [..., n]."""
    n = x.shape[-1]
    _shape(y, x.shape, "y")
    if y is None:
        y = torch.empty_like(x)
    _check("quarot_hadamard", lib().quarot_hadamard(
        _ptr(x, torch.float16, "x"), _ptr(y, torch.float16, "y"), _rows(x, n), n,
        _stream(stream)))
    return y


def quarot_quant_int4(x: torch.Tensor, rotate: bool = True, clip_ratio: float = 1.0,
                      q: Optional[torch.Tensor] = None, scale: Optional[torch.Tensor] = None,
                      stream: Optional[torch.cuda.Stream] = None):
    """Per-row symmetric int4 (optionally of the rotated row).
    Returns (codes uint8 [..., n/2], scale fp16 [...])."""
    n = x.shape[-1]
    rows = _rows(x, n)
    _numel(q, rows * (n // 2), "q")
    _numel(scale, rows, "scale")
    if q is None:
        q = torch.empty(x.shape[:-1] + (n // 2,), dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty(x.shape[:-1], dtype=torch.float16, device=x.device)
    _check("quarot_quant_int4", lib().quarot_quant_int4(
        _ptr(x, torch.float16, "x"), _ptr(q, torch.uint8, "q"),
        _ptr(scale, torch.float16, "scale"), rows, n, int(bool(rotate)), float(clip_ratio),
        _stream(stream)))
    return q, scale


def quarot_w4a4_gemm(xq: torch.Tensor, sx: torch.Tensor, wq: torch.Tensor, sw: torch.Tensor,
                     y: Optional[torch.Tensor] = None, acc_out: Optional[torch.Tensor] = None,
                     want_acc: bool = False, stream: Optional[torch.cuda.Stream] = None):
    """y = dequant(Xq Wq^T); returns y, or (y, acc) with want_acc."""
    _ndim(xq, 2, "xq")
    _ndim(wq, 2, "wq")
    M, Kh = xq.shape
    N = wq.shape[0]
    _shape(wq, (N, Kh), "wq")
    _numel(sx, M, "sx")
    _numel(sw, N, "sw")
    _shape(y, (M, N), "y")
    _shape(acc_out, (M, N), "acc_out")
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=xq.device)
    if want_acc and acc_out is None:
        acc_out = torch.empty((M, N), dtype=torch.int32, device=xq.device)
    _check("quarot_w4a4_gemm", lib().quarot_w4a4_gemm(
        _ptr(xq, torch.uint8, "xq"), _ptr(sx, torch.float16, "sx"), _ptr(wq, torch.uint8, "wq"),
        _ptr(sw, torch.float16, "sw"), _ptr(y, torch.float16, "y"),
        _ptr(acc_out, torch.int32, "acc_out"), M, N, 2 * Kh, _stream(stream)))
    return (y, acc_out) if (want_acc or acc_out is not None) else y


def quarot_pack_e3m2(q4: torch.Tensor, out: Optional[torch.Tensor] = None,
                     stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """int4 codes [rows, k/2] -> the tiled e3m2 operand layout, as uint8
    [k/128, rows*96] (one row per 128-wide k block)."""
    _ndim(q4, 2, "q4")
    rows, kh = q4.shape
    k = 2 * kh
    _numel(out, rows * k * 3 // 4, "out")
    if out is None:
        out = torch.empty((k // 128 if k % 128 == 0 else 0, rows * 96), dtype=torch.uint8,
                          device=q4.device)
    _check("quarot_pack_e3m2", lib().quarot_pack_e3m2(
        _ptr(q4, torch.uint8, "q4"), _ptr(out, torch.uint8, "out"), rows, k, _stream(stream)))
    return out


def quarot_w4a4_gemm_e3m2(xq6: torch.Tensor, sx: torch.Tensor, wq6: torch.Tensor,
                          sw: torch.Tensor, y: Optional[torch.Tensor] = None,
                          acc_out: Optional[torch.Tensor] = None, want_acc: bool = False,
                          stream: Optional[torch.cuda.Stream] = None):
    """quarot_w4a4_gemm on operands in the tiled e3m2 layout
    (xq6 [K/128, M*96], wq6 [K/128, N*96])."""
    M, N = sx.shape[0], sw.shape[0]
    K = 128 * xq6.shape[0]
    _ndim(xq6, 2, "xq6")
    if xq6.shape[1] != M * 96 or tuple(wq6.shape) != (xq6.shape[0], N * 96):
        raise ValueError("quarot_w4a4_gemm_e3m2: operand shapes do not match sx, sw")
    _shape(y, (M, N), "y")
    _shape(acc_out, (M, N), "acc_out")
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=xq6.device)
    if want_acc and acc_out is None:
        acc_out = torch.empty((M, N), dtype=torch.int32, device=xq6.device)
    _check("quarot_w4a4_gemm_e3m2", lib().quarot_w4a4_gemm_e3m2(
        _ptr(xq6, torch.uint8, "xq6"), _ptr(sx, torch.float16, "sx"),
        _ptr(wq6, torch.uint8, "wq6"), _ptr(sw, torch.float16, "sw"), _ptr(y, torch.float16, "y"),
        _ptr(acc_out, torch.int32, "acc_out"), M, N, K, _stream(stream)))
    return (y, acc_out) if (want_acc or acc_out is not None) else y


def quarot_quant_int4_e3m2(x: torch.Tensor, rotate: bool = True, clip_ratio: float = 1.0,
                           q6: Optional[torch.Tensor] = None,
                           scale: Optional[torch.Tensor] = None,
                           stream: Optional[torch.cuda.Stream] = None):
    """quarot_quant_int4 with the codes in the tiled e3m2 layout
    ([n/128, rows*96] uint8); returns (q6, scale)."""
    _ndim(x, 2, "x")
    rows, n = x.shape
    _numel(q6, rows * n * 3 // 4, "q6")
    _numel(scale, rows, "scale")
    if q6 is None:
        q6 = torch.empty((n // 128 if n % 128 == 0 else 0, rows * 96), dtype=torch.uint8,
                         device=x.device)
    if scale is None:
        scale = torch.empty((rows,), dtype=torch.float16, device=x.device)
    _check("quarot_quant_int4_e3m2", lib().quarot_quant_int4_e3m2(
        _ptr(x, torch.float16, "x"), _ptr(q6, torch.uint8, "q6"),
        _ptr(scale, torch.float16, "scale"), rows, n, int(bool(rotate)), float(clip_ratio),
        _stream(stream)))
    return q6, scale


def quarot_linear_e3m2_workspace_size(M: int, K: int) -> int:
    return int(lib().quarot_linear_e3m2_workspace_size(M, K))


def quarot_linear_e3m2(x: torch.Tensor, wq6: torch.Tensor, sw: torch.Tensor,
                       rotate: bool = True, clip_ratio: float = 1.0,
                       y: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None,
                       stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """The 4-bit linear layer on the e3m2 path (weights from
    prepare_weight_e3m2); y equals quarot_linear's bit for bit."""
    _ndim(x, 2, "x")
    M, K = x.shape
    N = sw.numel()
    _numel(wq6, N * K * 3 // 4, "wq6")
    _shape(y, (M, N), "y")
    need = quarot_linear_e3m2_workspace_size(M, K)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    _check("quarot_linear_e3m2", lib().quarot_linear_e3m2(
        _ptr(x, torch.float16, "x"), _ptr(wq6, torch.uint8, "wq6"), _ptr(sw, torch.float16, "sw"),
        _ptr(y, torch.float16, "y"), M, N, K, int(bool(rotate)), float(clip_ratio),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream)))
    return y


SCRATCH_BYTES = 64 << 20  # QUAROT_SCRATCH_BYTES


def quarot_linear_e3m2_scratch(x: torch.Tensor, wq6: torch.Tensor, sw: torch.Tensor,
                               rotate: bool = True, clip_ratio: float = 1.0,
                               y: Optional[torch.Tensor] = None,
                               stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """quarot_linear_e3m2 with the codes and scales in the library's fixed
    device scratch array instead of a workspace (the C call allocates
    nothing; pass y to keep this wrapper from allocating it).  Calls that
    overlap in time on one device share that array and race."""
    _ndim(x, 2, "x")
    M, K = x.shape
    N = sw.numel()
    _numel(wq6, N * K * 3 // 4, "wq6")
    _shape(y, (M, N), "y")
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    _check("quarot_linear_e3m2_scratch", lib().quarot_linear_e3m2_scratch(
        _ptr(x, torch.float16, "x"), _ptr(wq6, torch.uint8, "wq6"), _ptr(sw, torch.float16, "sw"),
        _ptr(y, torch.float16, "y"), M, N, K, int(bool(rotate)), float(clip_ratio),
        _stream(stream)))
    return y


def quarot_swiglu_quant_e3m2(gate: torch.Tensor, up: torch.Tensor, clip_ratio: float = 1.0,
                             stream: Optional[torch.cuda.Stream] = None):
    """quarot_swiglu_quant_int4 with the codes in the tiled e3m2 layout."""
    _ndim(gate, 2, "gate")
    _shape(up, gate.shape, "up")
    rows, n = gate.shape
    q6 = torch.empty((n // 128 if n % 128 == 0 else 0, rows * 96), dtype=torch.uint8,
                     device=gate.device)
    scale = torch.empty((rows,), dtype=torch.float16, device=gate.device)
    _check("quarot_swiglu_quant_e3m2", lib().quarot_swiglu_quant_e3m2(
        _ptr(gate, torch.float16, "gate"), _ptr(up, torch.float16, "up"),
        _ptr(q6, torch.uint8, "q6"), _ptr(scale, torch.float16, "scale"), rows, n,
        float(clip_ratio), _stream(stream)))
    return q6, scale


def prepare_weight_e3m2(w: torch.Tensor, rotate: bool = True, clip_ratio: float = 1.0,
                        stream: Optional[torch.cuda.Stream] = None):
    """prepare_weight, then the codes repacked into the tiled e3m2 layout."""
    wq, sw = quarot_quant_int4(w, rotate=rotate, clip_ratio=clip_ratio, stream=stream)
    return quarot_pack_e3m2(wq, stream=stream), sw


def quarot_linear(x: torch.Tensor, wq: torch.Tensor, sw: torch.Tensor, rotate: bool = True,
                  clip_ratio: float = 1.0, y: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None,
                  stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """The 4-bit linear layer: rotate+quantize x, W4A4 GEMM, dequant."""
    _ndim(x, 2, "x")
    _ndim(wq, 2, "wq")
    M, K = x.shape
    N = wq.shape[0]
    _shape(wq, (N, K // 2), "wq")
    _numel(sw, N, "sw")
    _shape(y, (M, N), "y")
    need = quarot_linear_workspace_size(M, K)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    _check("quarot_linear", lib().quarot_linear(
        _ptr(x, torch.float16, "x"), _ptr(wq, torch.uint8, "wq"), _ptr(sw, torch.float16, "sw"),
        _ptr(y, torch.float16, "y"), M, N, K, int(bool(rotate)), float(clip_ratio),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream)))
    return y


def prepare_weight(w: torch.Tensor, rotate: bool = True, clip_ratio: float = 1.0,
                   stream: Optional[torch.cuda.Stream] = None):
    """Offline weight prep: each output-channel row of W [N, K] rotated like
    an activation row, then quantized per row (per output channel)."""
    return quarot_quant_int4(w, rotate=rotate, clip_ratio=clip_ratio, stream=stream)


def quarot_quant_int8(x: torch.Tensor, rotate: bool = True, clip_ratio: float = 1.0,
                      bits: int = 8, q: Optional[torch.Tensor] = None,
                      scale: Optional[torch.Tensor] = None,
                      stream: Optional[torch.cuda.Stream] = None):
    """Per-row symmetric 6/8-bit codes, one int8 per element.
    Returns (codes int8 [..., n], scale fp16 [...])."""
    n = x.shape[-1]
    rows = _rows(x, n)
    _numel(q, rows * n, "q")
    _numel(scale, rows, "scale")
    if q is None:
        q = torch.empty(x.shape, dtype=torch.int8, device=x.device)
    if scale is None:
        scale = torch.empty(x.shape[:-1], dtype=torch.float16, device=x.device)
    _check("quarot_quant_int8", lib().quarot_quant_int8(
        _ptr(x, torch.float16, "x"), _ptr(q, torch.int8, "q"),
        _ptr(scale, torch.float16, "scale"), rows, n, int(bool(rotate)), float(clip_ratio),
        int(bits), _stream(stream)))
    return q, scale


def quarot_w8a8_gemm(xq: torch.Tensor, sx: torch.Tensor, wq: torch.Tensor, sw: torch.Tensor,
                     y: Optional[torch.Tensor] = None, acc_out: Optional[torch.Tensor] = None,
                     want_acc: bool = False, stream: Optional[torch.cuda.Stream] = None):
    """y = dequant(Xq Wq^T) over int8 codes; returns y, or (y, acc)."""
    _ndim(xq, 2, "xq")
    _ndim(wq, 2, "wq")
    M, K = xq.shape
    N = wq.shape[0]
    _shape(wq, (N, K), "wq")
    _numel(sx, M, "sx")
    _numel(sw, N, "sw")
    _shape(y, (M, N), "y")
    _shape(acc_out, (M, N), "acc_out")
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=xq.device)
    if want_acc and acc_out is None:
        acc_out = torch.empty((M, N), dtype=torch.int32, device=xq.device)
    _check("quarot_w8a8_gemm", lib().quarot_w8a8_gemm(
        _ptr(xq, torch.int8, "xq"), _ptr(sx, torch.float16, "sx"), _ptr(wq, torch.int8, "wq"),
        _ptr(sw, torch.float16, "sw"), _ptr(y, torch.float16, "y"),
        _ptr(acc_out, torch.int32, "acc_out"), M, N, K, _stream(stream)))
    return (y, acc_out) if (want_acc or acc_out is not None) else y


def quarot_linear_w8a8(x: torch.Tensor, wq: torch.Tensor, sw: torch.Tensor, rotate: bool = True,
                       clip_ratio: float = 1.0, bits: int = 8,
                       y: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None,
                       stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    _ndim(x, 2, "x")
    _ndim(wq, 2, "wq")
    M, K = x.shape
    N = wq.shape[0]
    _shape(wq, (N, K), "wq")
    _numel(sw, N, "sw")
    _shape(y, (M, N), "y")
    need = int(lib().quarot_linear_w8a8_workspace_size(M, K))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    _check("quarot_linear_w8a8", lib().quarot_linear_w8a8(
        _ptr(x, torch.float16, "x"), _ptr(wq, torch.int8, "wq"), _ptr(sw, torch.float16, "sw"),
        _ptr(y, torch.float16, "y"), M, N, K, int(bool(rotate)), float(clip_ratio), int(bits),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream)))
    return y


def quarot_quant_search(w: torch.Tensor, rotate: bool = True, bits: int = 4,
                        n_candidates: int = 20, stream: Optional[torch.cuda.Stream] = None):
    """Offline weight quantization with a per-row clip search.
    Returns (codes, scale fp16 [rows], chosen clip float32 [rows]); codes are
    packed nibbles uint8 [rows, n/2] for bits = 4, int8 [rows, n] otherwise."""
    _ndim(w, 2, "w")
    rows, n = w.shape
    dev = w.device
    if bits == 4:
        q = torch.empty((rows, n // 2), dtype=torch.uint8, device=dev)
    else:
        q = torch.empty((rows, n), dtype=torch.int8, device=dev)
    scale = torch.empty(rows, dtype=torch.float16, device=dev)
    clip = torch.empty(rows, dtype=torch.float32, device=dev)
    need = int(lib().quarot_quant_search_workspace_size(rows, n, int(bool(rotate))))
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check("quarot_quant_search", lib().quarot_quant_search(
        _ptr(w, torch.float16, "w"), ctypes.c_void_p(q.data_ptr()),
        _ptr(scale, torch.float16, "scale"), _ptr(clip, torch.float32, "clip"), rows, n,
        int(bool(rotate)), int(bits), int(n_candidates), _ptr(ws, torch.uint8, "workspace"),
        ws.numel(), _stream(stream)))
    return q, scale, clip


def quarot_quant_int4_grouped(x: torch.Tensor, group: int = 128, rotate: bool = True,
                              clip_ratio: float = 1.0, q: Optional[torch.Tensor] = None,
                              scale: Optional[torch.Tensor] = None,
                              workspace: Optional[torch.Tensor] = None,
                              stream: Optional[torch.cuda.Stream] = None):
    """Group-wise symmetric int4 of x [rows, n] (optionally rotated first).
    Returns (codes uint8 [rows, n/2], scale fp16 [n/group, rows])."""
    _ndim(x, 2, "x")
    rows, n = x.shape
    dev = x.device
    _group(group, n)
    _shape(q, (rows, n // 2), "q")
    _shape(scale, (n // group, rows), "scale")
    if q is None:
        q = torch.empty((rows, n // 2), dtype=torch.uint8, device=dev)
    if scale is None:
        scale = torch.empty((n // group if group > 0 else 0, rows), dtype=torch.float16,
                            device=dev)
    need = int(lib().quarot_quant_int4_grouped_workspace_size(rows, n, int(bool(rotate))))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check("quarot_quant_int4_grouped", lib().quarot_quant_int4_grouped(
        _ptr(x, torch.float16, "x"), _ptr(q, torch.uint8, "q"),
        _ptr(scale, torch.float16, "scale"), rows, n, int(group), int(bool(rotate)),
        float(clip_ratio), _ptr(workspace, torch.uint8, "workspace"), workspace.numel(),
        _stream(stream)))
    return q, scale


def quarot_w4a4_gemm_grouped(xq: torch.Tensor, sx: torch.Tensor, wq: torch.Tensor,
                             sw: torch.Tensor, group: int = 128,
                             y: Optional[torch.Tensor] = None,
                             stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Group-wise W4A4 product; sx [K/group, M], sw [K/group, N] group-major."""
    _ndim(xq, 2, "xq")
    _ndim(wq, 2, "wq")
    M, Kh = xq.shape
    N = wq.shape[0]
    _group(group, 2 * Kh)
    _shape(wq, (N, Kh), "wq")
    _shape(sx, (2 * Kh // group, M), "sx")
    _shape(sw, (2 * Kh // group, N), "sw")
    _shape(y, (M, N), "y")
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=xq.device)
    _check("quarot_w4a4_gemm_grouped", lib().quarot_w4a4_gemm_grouped(
        _ptr(xq, torch.uint8, "xq"), _ptr(sx, torch.float16, "sx"), _ptr(wq, torch.uint8, "wq"),
        _ptr(sw, torch.float16, "sw"), _ptr(y, torch.float16, "y"), M, N, 2 * Kh, int(group),
        _stream(stream)))
    return y


def quarot_w4a4_gemm_grouped_e3m2(xq6: torch.Tensor, sx: torch.Tensor, wq6: torch.Tensor,
                                  sw: torch.Tensor, group: int = 128,
                                  y: Optional[torch.Tensor] = None,
                                  stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """quarot_w4a4_gemm_grouped on operands in the tiled e3m2 layout
    (xq6 [K/128, M*96], wq6 [K/128, N*96]); sx [K/group, M], sw [K/group, N]."""
    _ndim(xq6, 2, "xq6")
    _ndim(sx, 2, "sx")
    _ndim(sw, 2, "sw")
    M, N = sx.shape[1], sw.shape[1]
    K = 128 * xq6.shape[0]
    _group(group, K)
    if xq6.shape[1] != M * 96 or tuple(wq6.shape) != (xq6.shape[0], N * 96):
        raise ValueError("quarot_w4a4_gemm_grouped_e3m2: operand shapes do not match sx, sw")
    _shape(sx, (K // group, M), "sx")
    _shape(sw, (K // group, N), "sw")
    _shape(y, (M, N), "y")
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=xq6.device)
    _check("quarot_w4a4_gemm_grouped_e3m2", lib().quarot_w4a4_gemm_grouped_e3m2(
        _ptr(xq6, torch.uint8, "xq6"), _ptr(sx, torch.float16, "sx"),
        _ptr(wq6, torch.uint8, "wq6"), _ptr(sw, torch.float16, "sw"), _ptr(y, torch.float16, "y"),
        M, N, K, int(group), _stream(stream)))
    return y


def quarot_linear_w4a4_grouped(x: torch.Tensor, wq: torch.Tensor, sw: torch.Tensor,
                               group: int = 128, rotate: bool = True, clip_ratio: float = 1.0,
                               y: Optional[torch.Tensor] = None,
                               workspace: Optional[torch.Tensor] = None,
                               stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """The group-wise 4-bit linear layer (quantize x per group, grouped GEMM)."""
    _ndim(x, 2, "x")
    _ndim(wq, 2, "wq")
    M, K = x.shape
    N = wq.shape[0]
    _group(group, K)
    _shape(wq, (N, K // 2), "wq")
    _shape(sw, (K // group, N), "sw")
    _shape(y, (M, N), "y")
    need = int(lib().quarot_linear_w4a4_grouped_workspace_size(M, K, int(group),
                                                               int(bool(rotate))))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    _check("quarot_linear_w4a4_grouped", lib().quarot_linear_w4a4_grouped(
        _ptr(x, torch.float16, "x"), _ptr(wq, torch.uint8, "wq"), _ptr(sw, torch.float16, "sw"),
        _ptr(y, torch.float16, "y"), M, N, K, int(group), int(bool(rotate)), float(clip_ratio),
        _ptr(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream)))
    return y


def quarot_swiglu(gate: torch.Tensor, up: torch.Tensor, h: Optional[torch.Tensor] = None,
                  stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """h = RN16(silu(gate) * up) elementwise (binary32 silu recipe)."""
    if tuple(up.shape) != tuple(gate.shape):
        raise ValueError("gate and up must have the same shape")
    _shape(h, gate.shape, "h")
    if h is None:
        h = torch.empty_like(gate)
    _check("quarot_swiglu", lib().quarot_swiglu(
        _ptr(gate, torch.float16, "gate"), _ptr(up, torch.float16, "up"),
        _ptr(h, torch.float16, "h"), gate.numel(), _stream(stream)))
    return h


def quarot_swiglu_quant_int4(gate: torch.Tensor, up: torch.Tensor, clip_ratio: float = 1.0,
                             q: Optional[torch.Tensor] = None,
                             scale: Optional[torch.Tensor] = None,
                             stream: Optional[torch.cuda.Stream] = None):
    """Down-projection input: int4 codes of the rotated RN16(silu(gate) * up).
    Returns (codes uint8 [..., n/2], scale fp16 [...])."""
    n = gate.shape[-1]
    if tuple(up.shape) != tuple(gate.shape):
        raise ValueError("gate and up must have the same shape")
    rows = _rows(gate, n)
    _numel(q, rows * (n // 2), "q")
    _numel(scale, rows, "scale")
    if q is None:
        q = torch.empty(gate.shape[:-1] + (n // 2,), dtype=torch.uint8, device=gate.device)
    if scale is None:
        scale = torch.empty(gate.shape[:-1], dtype=torch.float16, device=gate.device)
    _check("quarot_swiglu_quant_int4", lib().quarot_swiglu_quant_int4(
        _ptr(gate, torch.float16, "gate"), _ptr(up, torch.float16, "up"),
        _ptr(q, torch.uint8, "q"), _ptr(scale, torch.float16, "scale"), rows, n,
        float(clip_ratio), _stream(stream)))
    return q, scale


def quarot_hadamard_heads(z: torch.Tensor, n_heads: int, y: Optional[torch.Tensor] = None,
                          stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """y = RN16(z (H_nh (x) I_dh) / sqrt(nh)); z fp16 [..., n_heads * head_dim]."""
    n = z.shape[-1]
    _group(n_heads, n, "n_heads")
    _shape(y, z.shape, "y")
    if y is None:
        y = torch.empty_like(z)
    _check("quarot_hadamard_heads", lib().quarot_hadamard_heads(
        _ptr(z, torch.float16, "z"), _ptr(y, torch.float16, "y"), _rows(z, n), n_heads,
        n // n_heads if n_heads > 0 else 0, _stream(stream)))
    return y


def quarot_hadamard_heads_quant_int4(z: torch.Tensor, n_heads: int, clip_ratio: float = 1.0,
                                     q: Optional[torch.Tensor] = None,
                                     scale: Optional[torch.Tensor] = None,
                                     stream: Optional[torch.cuda.Stream] = None):
    """out_proj input: per-token int4 codes of the head-wise rotation."""
    n = z.shape[-1]
    rows = _rows(z, n)
    _group(n_heads, n, "n_heads")
    _numel(q, rows * (n // 2), "q")
    _numel(scale, rows, "scale")
    if q is None:
        q = torch.empty(z.shape[:-1] + (n // 2,), dtype=torch.uint8, device=z.device)
    if scale is None:
        scale = torch.empty(z.shape[:-1], dtype=torch.float16, device=z.device)
    _check("quarot_hadamard_heads_quant_int4", lib().quarot_hadamard_heads_quant_int4(
        _ptr(z, torch.float16, "z"), _ptr(q, torch.uint8, "q"),
        _ptr(scale, torch.float16, "scale"), rows, n_heads,
        n // n_heads if n_heads > 0 else 0, float(clip_ratio), _stream(stream)))
    return q, scale


def quarot_kv_quant(kv: torch.Tensor, group: int = 128, rotate: bool = True,
                    clip_ratio: float = 0.95, q: Optional[torch.Tensor] = None,
                    scale: Optional[torch.Tensor] = None, zero: Optional[torch.Tensor] = None,
                    stream: Optional[torch.cuda.Stream] = None):
    """4-bit asymmetric KV cache: kv fp16 [..., head_dim] ->
    (codes uint8 [..., head_dim/2], scale, zero fp16 [..., head_dim/group])."""
    D = kv.shape[-1]
    rows = _rows(kv, D)
    lead = kv.shape[:-1]
    _group(group, D)
    _numel(q, rows * (D // 2), "q")
    _numel(scale, rows * (D // group), "scale")
    _numel(zero, rows * (D // group), "zero")
    if q is None:
        q = torch.empty(lead + (D // 2,), dtype=torch.uint8, device=kv.device)
    if scale is None:
        scale = torch.empty(lead + (D // group,), dtype=torch.float16, device=kv.device)
    if zero is None:
        zero = torch.empty(lead + (D // group,), dtype=torch.float16, device=kv.device)
    _check("quarot_kv_quant", lib().quarot_kv_quant(
        _ptr(kv, torch.float16, "kv"), _ptr(q, torch.uint8, "q"),
        _ptr(scale, torch.float16, "scale"), _ptr(zero, torch.float16, "zero"), rows, D, group,
        int(bool(rotate)), float(clip_ratio), _stream(stream)))
    return q, scale, zero


def quarot_kv_dequant(q: torch.Tensor, scale: torch.Tensor, zero: torch.Tensor,
                      group: int = 128, inverse_rotate: bool = False,
                      out: Optional[torch.Tensor] = None,
                      stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    D = 2 * q.shape[-1]
    rows = _rows(q, D // 2)
    _group(group, D)
    _numel(scale, rows * (D // group), "scale")
    _numel(zero, rows * (D // group), "zero")
    _numel(out, rows * D, "out")
    if out is None:
        out = torch.empty(q.shape[:-1] + (D,), dtype=torch.float16, device=q.device)
    _check("quarot_kv_dequant", lib().quarot_kv_dequant(
        _ptr(q, torch.uint8, "q"), _ptr(scale, torch.float16, "scale"),
        _ptr(zero, torch.float16, "zero"), _ptr(out, torch.float16, "out"), rows, D, group,
        int(bool(inverse_rotate)), _stream(stream)))
    return out


def quarot_kv_append(kv_new: torch.Tensor, q_cache: torch.Tensor, scale_cache: torch.Tensor,
                     zero_cache: torch.Tensor, pos: int, group: int = 128, rotate: bool = True,
                     clip_ratio: float = 0.95, stream: Optional[torch.cuda.Stream] = None):
    """Quantize kv_new [rows, D] into token position pos of the caches
    q_cache [rows, s_max, D/2], scale/zero_cache [rows, s_max, D/group]."""
    D = kv_new.shape[-1]
    rows = _rows(kv_new, D)
    _group(group, D)
    if q_cache.dim() < 2:
        raise ValueError("q_cache must be [rows, s_max, head_dim/2]")
    s_max = q_cache.shape[-2]
    _numel(q_cache, rows * s_max * (D // 2), "q_cache")
    if q_cache.shape[-1] != D // 2:
        raise ValueError(f"q_cache rows must hold {D // 2} bytes, got {q_cache.shape[-1]}")
    _numel(scale_cache, rows * s_max * (D // group), "scale_cache")
    _numel(zero_cache, rows * s_max * (D // group), "zero_cache")
    _check("quarot_kv_append", lib().quarot_kv_append(
        _ptr(kv_new, torch.float16, "kv_new"), _ptr(q_cache, torch.uint8, "q_cache"),
        _ptr(scale_cache, torch.float16, "scale_cache"),
        _ptr(zero_cache, torch.float16, "zero_cache"), rows, s_max, pos, D, group,
        int(bool(rotate)), float(clip_ratio), _stream(stream)))


def quarot_kv_attention_workspace_size(nq: int, seq_len: int, head_dim: int) -> int:
    return int(lib().quarot_kv_attention_workspace_size(nq, seq_len, head_dim))


def quarot_kv_decode_attention(q: torch.Tensor, k_cache, v_cache, seq_len: int,
                               group: int = 128, sm_scale: Optional[float] = None,
                               out: Optional[torch.Tensor] = None,
                               workspace: Optional[torch.Tensor] = None,
                               stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Decode attention of rotated queries q [nq, D] over 4-bit caches
    k_cache = (codes [nkv, s_max, D/2], scale, zero [nkv, s_max, D/group]),
    v_cache alike.  Returns fp16 [nq, D]."""
    _ndim(q, 2, "q")
    nq, D = q.shape
    kc, ks, kz = k_cache
    vc, vs, vz = v_cache
    _ndim(kc, 3, "k_codes")
    nkv, s_max = kc.shape[0], kc.shape[1]
    _group(group, D)
    for t, nm in ((kc, "k_codes"), (vc, "v_codes")):
        _shape(t, (nkv, s_max, D // 2), nm)
    for t, nm in ((ks, "k_scale"), (kz, "k_zero"), (vs, "v_scale"), (vz, "v_zero")):
        _shape(t, (nkv, s_max, D // group), nm)
    _shape(out, (nq, D), "out")
    if sm_scale is None:
        sm_scale = D ** -0.5
    if out is None:
        out = torch.empty((nq, D), dtype=torch.float16, device=q.device)
    need = quarot_kv_attention_workspace_size(nq, seq_len, D)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    _check("quarot_kv_decode_attention", lib().quarot_kv_decode_attention(
        _ptr(q, torch.float16, "q"), _ptr(kc, torch.uint8, "k_codes"),
        _ptr(ks, torch.float16, "k_scale"), _ptr(kz, torch.float16, "k_zero"),
        _ptr(vc, torch.uint8, "v_codes"), _ptr(vs, torch.float16, "v_scale"),
        _ptr(vz, torch.float16, "v_zero"), _ptr(out, torch.float16, "out"), nq, nkv, s_max,
        seq_len, D, group, float(sm_scale),
        _ptr(workspace, torch.uint8, "workspace") if workspace is not None else None,
        workspace.numel() if workspace is not None else 0, _stream(stream)))
    return out


__all__ = [
    "QuarotError", "lib", "probe_lib", "quarot_version", "quarot_device_peaks", "quarot_mfma_probe",
    "quarot_hadamard_factor",
    "quarot_hadamard_factor_table", "quarot_linear_workspace_size", "quarot_hadamard",
    "quarot_quant_int4", "quarot_w4a4_gemm", "quarot_linear", "prepare_weight",
    "quarot_quant_int8", "quarot_w8a8_gemm", "quarot_linear_w8a8", "quarot_quant_search",
    "quarot_quant_int4_grouped", "quarot_w4a4_gemm_grouped",
    "quarot_w4a4_gemm_grouped_e3m2", "quarot_linear_w4a4_grouped",
    "quarot_swiglu", "quarot_swiglu_quant_int4", "quarot_hadamard_heads", "quarot_hadamard_heads_quant_int4",
    "quarot_kv_quant", "quarot_kv_dequant", "quarot_kv_append",
    "quarot_kv_attention_workspace_size", "quarot_kv_decode_attention",
    "quarot_mfma_probe_fp6", "quarot_pack_e3m2", "quarot_w4a4_gemm_e3m2",
    "quarot_quant_int4_e3m2", "quarot_linear_e3m2_workspace_size", "quarot_linear_e3m2",
    "quarot_swiglu_quant_e3m2", "prepare_weight_e3m2", "quarot_linear_e3m2_scratch",
]
