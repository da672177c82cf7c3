"""CPU oracle for deployment-aligned fake quantization and the STE linear layer.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package.  It shares no code with the
GPU library (``paper_2609_39223_amd``) and imports nothing from it.

Contents
--------
* ``qf_oracle.c`` (built to ``_build/liboracle.so`` by :func:`oracle.build.build`):
  plain C codecs for E2M1, E4M3, E8M0, bfloat16, float16 and the three quantizers
  NVFP4 / MXFP4 / Q4_K (QATFactory Sec. 3.2.3, Tab. formats; Eqs. nvfp4-dequant,
  mxfp4-dequant, q4k-dequant), plus Q4_K block packing (Sec. 3.5, engine-native export)
  and the LoRA merge W + s B A in binary32 (Sec. 3.3, Eqs. qad-lora, export-lora), and a
  Q4_K quantizer whose sub-block steps come from a search minimizing ||W - W_q||^2 (Sec. 4).
* FP64 linear-layer references in this module: the forward O = A_hat W_hat^T
  (Eq. fakequant, written for row-major activations) and the straight-through backward
  dA = dO W_hat (Eq. activation-ste), dW = dO^T A_hat (Eqs. ste, activation-gradient-error).
  A numpy float64 matmul is the only library primitive used.
* LoRA-QAD (Sec. 3.3): the merged fake quant W_hat = Q^-1(Q(W + s B A)) (Eq. qad-lora), its
  export codes Q(W + s B A) (Eq. export-lora), and the FP64 STE gradients of the factors:
  with G = dO^T A_hat the straight-through gradient of the merged weight (Eq. ste),
  dB = s G A^T and dA = s B^T G (chain rule through W + s B A).  The MoE variants apply
  these per expert (Sec. 3.3 "Mixture-of-experts adaptation": unshared factors, or one
  factor shared by every expert, whose gradient is then the sum over experts).
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
        L.or_q4k_mse_quant.argtypes = [_u16p, _i64, _i64, _i64, _u8p, _u16p]
        L.or_q4k_mse_quant.restype = None
        L.or_q4k_mse_subblock.argtypes = [_f32p, _f32p, _f32p, ctypes.POINTER(ctypes.c_int)]
        L.or_q4k_mse_subblock.restype = None
        L.or_lora_merge.argtypes = [_u16p, _i64, _i64, _i64, _f32p, _f32p, _i64, ctypes.c_float,
                                    _u16p]
        L.or_lora_merge.restype = None
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


# ------------------------------------------------------------------------------ LoRA-QAD
def lora_merge(w: np.ndarray, B: np.ndarray, A: np.ndarray, scale: float = 1.0) -> np.ndarray:
    """bf16 bits of W + scale * B A (Sec. 3.3, Eq. qad-lora): binary32 merge, one fused
    multiply-add per rank term in increasing rank order, rounded once to bf16 (the C
    function or_lora_merge states the reading)."""
    w, N, K = _rows(w)
    B = np.ascontiguousarray(B, dtype=np.float32)
    A = np.ascontiguousarray(A, dtype=np.float32)
    r = A.shape[0]
    assert B.shape == (N, r) and A.shape == (r, K)
    out = np.zeros((N, K), np.uint16)
    lib().or_lora_merge(_ptr(w, _u16p), N, K, K, _ptr(B, _f32p), _ptr(A, _f32p), r,
                        float(np.float32(scale)), _ptr(out, _u16p))
    return out


def lora_quant(w: np.ndarray, B: np.ndarray, A: np.ndarray, scale: float, fmt: str,
               amax_in: float | None = None) -> dict:
    """Q(W + s B A) with its dequantization (Eqs. qad-lora, export-lora): the quantizer of
    `fmt` applied to the merged bf16 weight; for NVFP4 the tensor amax is that of the merged
    weight unless amax_in (a tied-group value) is given.  Returns the quantizer's dict plus
    'merged' (the bf16 merged weight)."""
    m = lora_merge(w, B, A, scale)
    if fmt == "nvfp4":
        out = nvfp4(m, amax_in)
        out["amax"] = amax(m) if amax_in is None else float(np.float32(amax_in))
    elif fmt == "mxfp4":
        out = mxfp4(m)
    elif fmt == "q4k":
        out = q4k(m)
    else:
        raise ValueError(fmt)
    out["merged"] = m
    return out


def lora_grads(dy: np.ndarray, aop: np.ndarray, B: np.ndarray, A: np.ndarray,
               scale: float = 1.0):
    """FP64 STE gradients of the LoRA factors (Sec. 3.3 with Eq. ste): G = dO^T A_hat is the
    straight-through gradient of the merged weight W + s B A, so dB = s G A^T [N, r] and
    dA = s B^T G [r, K].  Returns (dA, dB)."""
    G = linear_dw(dy, aop)
    B64 = np.asarray(B, np.float64)
    A64 = np.asarray(A, np.float64)
    s = float(np.float32(scale))
    return s * (B64.T @ G), s * (G @ A64.T)


def _expert_factor(F: np.ndarray, e: int, per_expert_ndim: int) -> np.ndarray:
    """Expert e's slice of an unshared factor stack, or the shared factor itself."""
    return F[e] if F.ndim == per_expert_ndim else F


def lora_grads_grouped(dy: np.ndarray, aop: np.ndarray, offsets, B: np.ndarray, A: np.ndarray,
                       scale: float = 1.0):
    """FP64 factor gradients of the MoE LoRA layer (Sec. 3.3 "Mixture-of-experts adaptation").
    Rows [off[e], off[e+1]) of dy [T, N] and aop [T, K] belong to expert e.  A is [E, r, K]
    (one factor per expert) or [r, K] (shared by all experts); B is [E, N, r] or [N, r].
    Expert e's merged-weight gradient is G_e = dO_e^T A_hat_e; an unshared factor gets its
    expert's term, a shared factor the sum of the terms over experts in expert order.
    Returns (dA, dB) shaped like A and B."""
    off = np.asarray(offsets, np.int64)
    E = len(off) - 1
    s = float(np.float32(scale))
    dA = np.zeros(A.shape, np.float64)
    dB = np.zeros(B.shape, np.float64)
    for e in range(E):
        G = linear_dw(dy[off[e]:off[e + 1]], aop[off[e]:off[e + 1]])
        Ae = np.asarray(_expert_factor(A, e, 3), np.float64)
        Be = np.asarray(_expert_factor(B, e, 3), np.float64)
        ga, gb = s * (Be.T @ G), s * (G @ Ae.T)
        if A.ndim == 3:
            dA[e] = ga
        else:
            dA += ga
        if B.ndim == 3:
            dB[e] = gb
        else:
            dB += gb
    return dA, dB


def lora_quant_grouped(w: np.ndarray, B: np.ndarray, A: np.ndarray, scale: float, fmt: str):
    """Per-expert W_hat_e = Q^-1(Q(W_e + s B_e A_e)) for W [E, N, K] (Sec. 3.3: each expert's
    merged weight is quantized on its own, with its own NVFP4 tensor amax).  A / B as in
    lora_grads_grouped.  Returns x_hat [E, N, K]."""
    E = w.shape[0]
    return np.stack([lora_quant(w[e], _expert_factor(B, e, 3), _expert_factor(A, e, 3), scale,
                                fmt)["xhat"] for e in range(E)])


# --------------------------------------------------------------------- QAD distillation loss
def _log_softmax_f64(z: np.ndarray) -> np.ndarray:
    m = z.max(axis=1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))


def qad_kl(zt: np.ndarray, zs: np.ndarray):
    """Token-averaged forward KL of Eq. qad-objective in FP64 from bf16 logits [L, V] of the
    teacher (zt) and the student (zs): p = softmax over the vocabulary per token,
    KL_t = sum_v p_T log(p_T / p_S), loss = mean_t KL_t.  Its gradient with respect to the
    student's logits is (p_S - p_T) / L (the softmax Jacobian applied to -p_T / p_S).
    Also returns the teacher-student top-1 agreement per token (first index among equal
    maxima, compared on the bf16 logits).  Returns (loss, kl [L], grad [L, V], agree [L])."""
    t = bf16_array_to_f64(zt)
    s = bf16_array_to_f64(zs)
    L = t.shape[0]
    lt, ls = _log_softmax_f64(t), _log_softmax_f64(s)
    pt, ps = np.exp(lt), np.exp(ls)
    kl = (pt * (lt - ls)).sum(axis=1)
    loss = float(kl.mean()) if L else 0.0
    grad = (ps - pt) / max(L, 1)
    agree = (t.argmax(axis=1) == s.argmax(axis=1)).astype(np.int32)
    return loss, kl, grad, agree


# ----------------------------------------------------------------- Q4_K with an MSE search
def q4k_mse(x: np.ndarray) -> dict:
    """Q4_K with searched sub-block steps (the scale search minimizes ||W - W_q||^2, the
    objective of the paper's Q4_K PTQ baseline, Sec. 4): same 144-byte blocks and x_hat as
    q4k(); the C function or_q4k_mse_quant states the search."""
    x, R, K = _rows(x)
    assert K % 256 == 0
    packed = np.zeros((R, K // 256, 144), np.uint8)
    xhat = np.zeros((R, K), np.uint16)
    lib().or_q4k_mse_quant(_ptr(x, _u16p), R, K, K, _ptr(packed, _u8p), _ptr(xhat, _u16p))
    return {"packed": packed, "xhat": xhat}


def q4k_mse_subblock(x32) -> tuple:
    """The search for one 32-element sub-block: (a, mu, codes)."""
    xv = np.ascontiguousarray(x32, np.float32)
    assert xv.shape == (32,)
    a = np.zeros(1, np.float32)
    mu = np.zeros(1, np.float32)
    q = (ctypes.c_int * 32)()
    lib().or_q4k_mse_subblock(_ptr(xv, _f32p), _ptr(a, _f32p), _ptr(mu, _f32p), q)
    return float(a[0]), float(mu[0]), np.array(list(q))


# ------------------------------------------------------------ engine-native export (NVFP4/MXFP4)
def export_fused(members, fmt: str, a_amax: float | None = None) -> dict:
    """Export of a fused projection (Sec. 3.2.3 "Engine-specific scale sharing", Sec. 3.5):
    the engine's fused weight is the row concatenation of the member weights (QKV, gate/up);
    NVFP4 uses one tensor scale for it, from the amax over all members, and exports the
    input-activation scale from the running activation amax (Sec. 3.2.3 NVFP4 paragraph:
    S_act = amax / (6 * 448), the decode scale the engine applies).  MXFP4 has block scales
    only.  Returns codes [N, K/2], scales, and for NVFP4 weight_scale_2 (S) and input_scale."""
    W = np.concatenate([np.ascontiguousarray(m) for m in members], axis=0)
    if fmt == "nvfp4":
        q = nvfp4(W)
        out = {"codes": q["codes"], "scales": q["scales"], "weight_scale_2": q["S"],
               "amax": amax(W)}
        out["input_scale"] = (float(np.float32(np.float32(a_amax) / np.float32(2688.0)))
                              if a_amax is not None else None)
        return out
    if fmt == "mxfp4":
        q = mxfp4(W)
        return {"codes": q["codes"], "scales": q["scales"]}
    raise ValueError(fmt)


PAYLOAD_MAGIC = 0x31504651          # bytes "QFP1"


def payload_layout(fmt: str, N: int, K: int) -> dict:
    """Weight-sync payload of one layer (this library's format): a 64-byte header, then the
    codes, the block scales and two FP32 scalars (weight_scale_2, input_scale; zeros for
    MXFP4), each section starting at a multiple of 256 bytes."""
    blk = {"nvfp4": 16, "mxfp4": 32}[fmt]
    up = lambda v: (v + 255) // 256 * 256
    off_codes = 256
    off_scales = off_codes + up(N * K // 2)
    off_scalars = off_scales + up(N * K // blk)
    return {"codes": off_codes, "scales": off_scales, "scalars": off_scalars,
            "total": off_scalars + 256, "blk": blk}


def parse_payload(buf: np.ndarray) -> dict:
    """Reads a payload back (header fields little-endian: u32 magic, u32 format, i64 N, i64 K,
    u64 codes / scales / scalars offsets, u64 total size)."""
    b = np.ascontiguousarray(buf, np.uint8)
    magic, fmt = (int(v) for v in b[0:8].view("<u4"))
    N, K = (int(v) for v in b[8:24].view("<i8"))
    oc, osc, osr, total = (int(v) for v in b[24:56].view("<u8"))
    name = {1: "nvfp4", 2: "mxfp4"}[int(fmt)]
    blk = 16 if name == "nvfp4" else 32
    return {"magic": int(magic), "fmt": name, "N": int(N), "K": int(K), "total": int(total),
            "codes": b[oc:oc + N * K // 2].reshape(N, K // 2),
            "scales": b[osc:osc + N * K // blk].reshape(N, K // blk),
            "scalars": b[osr:osr + 8].view("<f4")}
