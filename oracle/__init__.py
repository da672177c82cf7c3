"""CPU oracle for deployment-aligned fake quantization and the STE linear layer.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package.  It shares no code with the
GPU library (``paper_2609_39223_amd``) and imports nothing from it.

Contents
--------
* ``qf_oracle.c`` (built to ``_build/liboracle.so`` by :func:`oracle.build.build`):
  plain C codecs for E2M1, E4M3, E8M0, bfloat16, float16 and the three quantizers
  NVFP4 / MXFP4 / Q4_K (QATFactory Sec. 3.2.3, Tab. formats; Eqs. nvfp4-dequant,
  mxfp4-dequant, q4k-dequant), plus Q4_K block packing (Sec. 3.5, engine-native export).
* FP64 linear-layer references in this module: the forward O = A_hat W_hat^T
  (Eq. fakequant, written for row-major activations) and the straight-through backward
  dA = dO W_hat (Eq. activation-ste), dW = dO^T A_hat (Eqs. ste, activation-gradient-error).
  A numpy float64 matmul is the only library primitive used.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_build", "liboracle.so")
_lib = None

_u16p = ctypes.POINTER(ctypes.c_uint16)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_f32p = ctypes.POINTER(ctypes.c_float)
_i64 = ctypes.c_int64


def lib():
    """Load (building on first use if needed) the oracle's shared library."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(_LIB_PATH)
        L.or_bf16_to_f32.argtypes = [ctypes.c_uint16]
        L.or_bf16_to_f32.restype = ctypes.c_float
        L.or_bf16_from_f32.argtypes = [ctypes.c_float]
        L.or_bf16_from_f32.restype = ctypes.c_uint16
        L.or_f16_to_f32.argtypes = [ctypes.c_uint16]
        L.or_f16_to_f32.restype = ctypes.c_float
        L.or_f16_from_f32.argtypes = [ctypes.c_float]
        L.or_f16_from_f32.restype = ctypes.c_uint16
        L.or_e2m1_value.argtypes = [ctypes.c_int]
        L.or_e2m1_value.restype = ctypes.c_double
        L.or_e2m1_encode.argtypes = [ctypes.c_double]
        L.or_e2m1_encode.restype = ctypes.c_int
        L.or_e4m3_decode.argtypes = [ctypes.c_int]
        L.or_e4m3_decode.restype = ctypes.c_double
        L.or_e4m3_encode.argtypes = [ctypes.c_double]
        L.or_e4m3_encode.restype = ctypes.c_int
        L.or_e8m0_decode.argtypes = [ctypes.c_int]
        L.or_e8m0_decode.restype = ctypes.c_double
        L.or_amax.argtypes = [_u16p, _i64, _i64, _i64]
        L.or_amax.restype = ctypes.c_float
        L.or_nvfp4_quant.argtypes = [_u16p, _i64, _i64, _i64, _f32p, _u8p, _u8p, _f32p, _u16p]
        L.or_nvfp4_quant.restype = None
        L.or_nvfp4_dequant.argtypes = [_u8p, _u8p, ctypes.c_float, _i64, _i64, _u16p]
        L.or_nvfp4_dequant.restype = None
        L.or_mxfp4_quant.argtypes = [_u16p, _i64, _i64, _i64, _u8p, _u8p, _u16p]
        L.or_mxfp4_quant.restype = None
        L.or_mxfp4_dequant.argtypes = [_u8p, _u8p, _i64, _i64, _u16p]
        L.or_mxfp4_dequant.restype = None
        L.or_q4k_quant.argtypes = [_u16p, _i64, _i64, _i64, _u8p, _u16p]
        L.or_q4k_quant.restype = None
        L.or_q4k_dequant.argtypes = [_u8p, _i64, _i64, _u16p]
        L.or_q4k_dequant.restype = None
        ip = ctypes.POINTER(ctypes.c_int)
        L.or_q4k_pack_block.argtypes = [_u8p, ctypes.c_uint16, ctypes.c_uint16, ip, ip, ip]
        L.or_q4k_pack_block.restype = None
        L.or_q4k_unpack_block.argtypes = [_u8p, ctypes.POINTER(ctypes.c_uint16),
                                          ctypes.POINTER(ctypes.c_uint16), ip, ip, ip]
        L.or_q4k_unpack_block.restype = None
        _lib = L
    return _lib


def _ptr(a, t):
    return a.ctypes.data_as(t) if a is not None else None


def _rows(x: np.ndarray):
    assert x.dtype == np.uint16 and x.ndim == 2
    x = np.ascontiguousarray(x)
    return x, x.shape[0], x.shape[1]


# --------------------------------------------------------------------------- codecs
def bf16_to_f32(h: int) -> float:
    return lib().or_bf16_to_f32(int(h))


def bf16_from_f32(v: float) -> int:
    return lib().or_bf16_from_f32(float(np.float32(v)))


def f16_to_f32(h: int) -> float:
    return lib().or_f16_to_f32(int(h))


def f16_from_f32(v: float) -> int:
    return lib().or_f16_from_f32(float(np.float32(v)))


def e2m1_value(code: int) -> float:
    return lib().or_e2m1_value(int(code))


def e2m1_encode(v: float) -> int:
    return lib().or_e2m1_encode(float(v))


def e4m3_decode(code: int) -> float:
    return lib().or_e4m3_decode(int(code))


def e4m3_encode(t: float) -> int:
    return lib().or_e4m3_encode(float(t))


def e8m0_decode(code: int) -> float:
    return lib().or_e8m0_decode(int(code))


# ------------------------------------------------------------------------ quantizers
def amax(x: np.ndarray) -> float:
    x, R, K = _rows(x)
    return float(lib().or_amax(_ptr(x, _u16p), R, K, K))


def nvfp4(x: np.ndarray, amax_in: float | None = None) -> dict:
    """NVFP4 fake quant of a bf16 [R, K] tensor (blocks of 16 along K)."""
    x, R, K = _rows(x)
    assert K % 16 == 0
    codes = np.zeros((R, K // 2), np.uint8)
    scales = np.zeros((R, K // 16), np.uint8)
    xhat = np.zeros((R, K), np.uint16)
    s = np.zeros(1, np.float32)
    g = None if amax_in is None else np.array([amax_in], np.float32)
    lib().or_nvfp4_quant(_ptr(x, _u16p), R, K, K, _ptr(g, _f32p), _ptr(codes, _u8p),
                         _ptr(scales, _u8p), _ptr(s, _f32p), _ptr(xhat, _u16p))
    return {"codes": codes, "scales": scales, "S": float(s[0]), "xhat": xhat}


def nvfp4_dequant(codes: np.ndarray, scales: np.ndarray, S: float, K: int) -> np.ndarray:
    R = codes.shape[0]
    codes = np.ascontiguousarray(codes)
    scales = np.ascontiguousarray(scales)
    out = np.zeros((R, K), np.uint16)
    lib().or_nvfp4_dequant(_ptr(codes, _u8p), _ptr(scales, _u8p), float(S), R, K,
                           _ptr(out, _u16p))
    return out


def mxfp4(x: np.ndarray) -> dict:
    """MXFP4 fake quant of a bf16 [R, K] tensor (blocks of 32 along K)."""
    x, R, K = _rows(x)
    assert K % 32 == 0
    codes = np.zeros((R, K // 2), np.uint8)
    scales = np.zeros((R, K // 32), np.uint8)
    xhat = np.zeros((R, K), np.uint16)
    lib().or_mxfp4_quant(_ptr(x, _u16p), R, K, K, _ptr(codes, _u8p), _ptr(scales, _u8p),
                         _ptr(xhat, _u16p))
    return {"codes": codes, "scales": scales, "xhat": xhat}


def mxfp4_dequant(codes: np.ndarray, scales: np.ndarray, K: int) -> np.ndarray:
    R = codes.shape[0]
    codes = np.ascontiguousarray(codes)
    scales = np.ascontiguousarray(scales)
    out = np.zeros((R, K), np.uint16)
    lib().or_mxfp4_dequant(_ptr(codes, _u8p), _ptr(scales, _u8p), R, K, _ptr(out, _u16p))
    return out


def q4k(x: np.ndarray) -> dict:
    """Q4_K fake quant + 144-byte packing of a bf16 [R, K] tensor (super-blocks of 256)."""
    x, R, K = _rows(x)
    assert K % 256 == 0
    packed = np.zeros((R, K // 256, 144), np.uint8)
    xhat = np.zeros((R, K), np.uint16)
    lib().or_q4k_quant(_ptr(x, _u16p), R, K, K, _ptr(packed, _u8p), _ptr(xhat, _u16p))
    return {"packed": packed, "xhat": xhat}


def q4k_dequant(packed: np.ndarray, K: int) -> np.ndarray:
    packed = np.ascontiguousarray(packed)
    R = packed.shape[0]
    out = np.zeros((R, K), np.uint16)
    lib().or_q4k_dequant(_ptr(packed, _u8p), R, K, _ptr(out, _u16p))
    return out


def q4k_pack_block(d: int, dmin: int, ls, lm, q) -> np.ndarray:
    out = np.zeros(144, np.uint8)
    ci = ctypes.c_int
    a_ls = (ci * 8)(*[int(v) for v in ls])
    a_lm = (ci * 8)(*[int(v) for v in lm])
    a_q = (ci * 256)(*[int(v) for v in q])
    lib().or_q4k_pack_block(_ptr(out, _u8p), int(d), int(dmin), a_ls, a_lm, a_q)
    return out


def q4k_unpack_block(block: np.ndarray):
    block = np.ascontiguousarray(block, dtype=np.uint8)
    ci = ctypes.c_int
    d = ctypes.c_uint16()
    m = ctypes.c_uint16()
    a_ls, a_lm, a_q = (ci * 8)(), (ci * 8)(), (ci * 256)()
    lib().or_q4k_unpack_block(_ptr(block, _u8p), ctypes.byref(d), ctypes.byref(m), a_ls, a_lm,
                              a_q)
    return d.value, m.value, list(a_ls), list(a_lm), list(a_q)


def fakequant(x: np.ndarray, fmt: str, amax_in: float | None = None) -> np.ndarray:
    """x_hat = Q^-1(Q(x)) for fmt in {none, nvfp4, mxfp4, q4k} (Eq. fakequant)."""
    if fmt == "none":
        return np.ascontiguousarray(x)
    if fmt == "nvfp4":
        return nvfp4(x, amax_in)["xhat"]
    if fmt == "mxfp4":
        return mxfp4(x)["xhat"]
    if fmt == "q4k":
        return q4k(x)["xhat"]
    raise ValueError(fmt)


# ------------------------------------------------------------------- FP64 linear layer
def bf16_array_to_f64(h: np.ndarray) -> np.ndarray:
    """Exact widening of raw bfloat16 bits to float64."""
    return (h.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def linear_fwd(ahat: np.ndarray, what: np.ndarray) -> np.ndarray:
    """O = A_hat W_hat^T in FP64 (Eq. fakequant with row-major activations [M, K] and
    nn.Linear weights [N, K])."""
    return bf16_array_to_f64(ahat) @ bf16_array_to_f64(what).T


def linear_dx(dy: np.ndarray, what: np.ndarray) -> np.ndarray:
    """dA = dO W_hat in FP64 (Eq. activation-ste: the STE passes dO through W_hat)."""
    return bf16_array_to_f64(dy) @ bf16_array_to_f64(what)


def linear_dw(dy: np.ndarray, aop: np.ndarray) -> np.ndarray:
    """dW = dO^T A_hat in FP64 (Eq. ste; A_hat = A when activations are not quantized)."""
    return bf16_array_to_f64(dy).T @ bf16_array_to_f64(aop)


def dot_rows(a: np.ndarray, ai, b: np.ndarray, bi) -> np.ndarray:
    """Sampled FP64 entries sum_k a[ai[t], k] * b[bi[t], k] (for full-size spot checks)."""
    A = bf16_array_to_f64(a[np.asarray(ai)])
    B = bf16_array_to_f64(b[np.asarray(bi)])
    return (A * B).sum(axis=1)
