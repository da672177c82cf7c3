"""Python binding of libqf (C ABI in include/qf.h): argument marshalling only.

Every function takes torch tensors that live on the GPU, passes their device pointers and
the current HIP stream to the C entry point of the same name, and raises ``QFError`` when
the call returns a non-OK status.  All arithmetic runs in the library's HIP kernels; there
is no fallback path.  bf16 tensors may be ``torch.bfloat16`` or raw 16-bit integer tensors.

Tensor conventions follow nn.Linear: X [M, K], W [N, K], Y [M, N]; dW is FP32 [N, K].
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqf.so")

FMT = {"none": 0, "nvfp4": 1, "mxfp4": 2, "q4k": 3}
AMAX_COMPUTE, AMAX_GIVEN = 0, 1
FLAG_REUSE_WS = 1
FLAG_DECODE_IN_GEMM = 2
STATUS = {0: "QF_OK", 1: "QF_EINVAL", 2: "QF_ESHAPE", 3: "QF_EALIGN", 4: "QF_ENOTSUP",
          5: "QF_EDEVICE"}


class QFError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class QLinearDesc(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("ldx", ctypes.c_int64), ("ldw", ctypes.c_int64), ("ldy", ctypes.c_int64),
                ("wfmt", ctypes.c_int32), ("afmt", ctypes.c_int32),
                ("w_amax", ctypes.c_void_p), ("a_amax", ctypes.c_void_p),
                ("flags", ctypes.c_uint32)]


class LoRA(ctypes.Structure):
    _fields_ = [("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("r", ctypes.c_int64),
                ("scale", ctypes.c_float), ("a_shared", ctypes.c_int32),
                ("b_shared", ctypes.c_int32)]


class Member(ctypes.Structure):
    _fields_ = [("W", ctypes.c_void_p), ("rows", ctypes.c_int64), ("ldw", ctypes.c_int64)]


class PayloadLayout(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_uint64), ("scales", ctypes.c_uint64),
                ("scalars", ctypes.c_uint64), ("total", ctypes.c_uint64)]


class GroupedDesc(ctypes.Structure):
    _fields_ = [("E", ctypes.c_int64), ("T", ctypes.c_int64), ("N", ctypes.c_int64),
                ("K", ctypes.c_int64), ("wfmt", ctypes.c_int32), ("afmt", ctypes.c_int32),
                ("w_amax", ctypes.c_void_p), ("flags", ctypes.c_uint32)]


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int64


def lib() -> ctypes.CDLL:
    """Load libqf.so (built in-tree by ``__graft_entry__.build()``); no fallback."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        torch.cuda.init()  # bind the process's HIP runtime before the library loads
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "qf_version": ([], ctypes.c_int),
            "qf_last_error": ([], ctypes.c_char_p),
            "qf_amax": ([_P, _I, _I, _I, _P, ctypes.c_int, _P], ctypes.c_int),
            "qf_fakequant_nvfp4": ([_P, _I, _I, _I, _P, ctypes.c_int, _P, _P, _P, _P, _P],
                                   ctypes.c_int),
            "qf_fakequant_mxfp4": ([_P, _I, _I, _I, _P, _P, _P, _P], ctypes.c_int),
            "qf_fakequant_q4k": ([_P, _I, _I, _I, _P, _P, _P], ctypes.c_int),
            "qf_fakequant_q4k_mse": ([_P, _I, _I, _I, _P, _P, _P], ctypes.c_int),
            "qf_workspace_size": ([ctypes.POINTER(QLinearDesc), ctypes.POINTER(ctypes.c_size_t)],
                                  ctypes.c_int),
            "qf_saved_size": ([ctypes.POINTER(QLinearDesc), ctypes.POINTER(ctypes.c_size_t)],
                              ctypes.c_int),
            "qf_qlinear_fwd": ([ctypes.POINTER(QLinearDesc), _P, _P, _P, _P, _P, ctypes.c_size_t,
                                _P], ctypes.c_int),
            "qf_qlinear_fwd_noalloc": ([ctypes.POINTER(QLinearDesc), _P, _P, _P, _P],
                                       ctypes.c_int),
            "qf_qlinear_bwd_ste": ([ctypes.POINTER(QLinearDesc), _P, _P, _P, _P, _P, _P, _P,
                                    ctypes.c_size_t, _P], ctypes.c_int),
            "qf_fragment_bytes": ([_I, _I, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
            "qf_pack_fragments": ([_P, _I, _I, _I, _P, _P], ctypes.c_int),
            "qf_gemm_bf16_fragb": ([_I, _I, _I, _P, _I, _P, _P, _I, ctypes.c_int, _P,
                                    ctypes.c_size_t, _P], ctypes.c_int),
            "qf_gemm_packed_b": ([_I, _I, _I, _P, _I, ctypes.c_int, _P, _P, _P, _P, _I, _P],
                                 ctypes.c_int),
            "qf_dequantize_transposed": ([ctypes.c_int, _P, _P, _P, _I, _I, _P, _I, _P],
                                         ctypes.c_int),
            "qf_validate_fakequant": ([ctypes.c_int, _P, _I, _I, _I], ctypes.c_int),
            "qf_validate_qlinear": ([ctypes.POINTER(QLinearDesc), _P, _P, _P, _P, _P,
                                     ctypes.c_size_t], ctypes.c_int),
            "qf_validate_grouped": ([ctypes.POINTER(GroupedDesc), _P, _P, _P, _P, _P,
                                     ctypes.c_size_t], ctypes.c_int),
            "qf_grouped_workspace_size": ([ctypes.POINTER(GroupedDesc),
                                           ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
            "qf_grouped_saved_size": ([ctypes.POINTER(GroupedDesc),
                                       ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
            "qf_qlinear_grouped_fwd": ([ctypes.POINTER(GroupedDesc), _P, _P, _P, _P, _P, _P,
                                        ctypes.c_size_t, _P], ctypes.c_int),
            "qf_qlinear_grouped_bwd_ste": ([ctypes.POINTER(GroupedDesc), _P, _P, _P, _P, _P, _P,
                                            _P, _P, ctypes.c_size_t, _P], ctypes.c_int),
            "qf_gemm_bf16": ([_I, _I, _I, _P, _I, ctypes.c_int, _P, _I, ctypes.c_int, _P, _I,
                              ctypes.c_int, _P], ctypes.c_int),
            "qf_transpose_bf16": ([_P, _I, _I, _I, _P, _I, _P], ctypes.c_int),
            "qf_gemm_workspace_size": ([_I, _I, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)],
                                       ctypes.c_int),
            "qf_gemm_bf16_ws": ([_I, _I, _I, _P, _I, ctypes.c_int, _P, _I, ctypes.c_int, _P, _I,
                                 ctypes.c_int, _P, ctypes.c_size_t, _P], ctypes.c_int),
            "qf_gemm_bf16_at": ([_I, _I, _I, _P, _I, _P, _I, _P, _I, _P, _I, _P], ctypes.c_int),
            "qf_fakequant_transposed": ([ctypes.c_int, _P, _I, _I, _I, _P, _P, _I, _P],
                                        ctypes.c_int),
            "qf_lora_amax": ([_P, _I, _I, _I, ctypes.POINTER(LoRA), _P, ctypes.c_int, _P],
                             ctypes.c_int),
            "qf_lora_fakequant": ([ctypes.c_int, _P, _I, _I, _I, ctypes.POINTER(LoRA), _P,
                                   ctypes.c_int, _P, _P, _P, _P, _P, _P], ctypes.c_int),
            "qf_lora_fakequant_transposed": ([ctypes.c_int, _P, _I, _I, _I, ctypes.POINTER(LoRA),
                                              _P, _P, _I, _P], ctypes.c_int),
            "qf_lora_workspace_size": ([ctypes.POINTER(QLinearDesc), ctypes.POINTER(LoRA),
                                        ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
            "qf_qlinear_lora_fwd": ([ctypes.POINTER(QLinearDesc), ctypes.POINTER(LoRA), _P, _P,
                                     _P, _P, ctypes.c_size_t, _P], ctypes.c_int),
            "qf_qlinear_lora_bwd_ste": ([ctypes.POINTER(QLinearDesc), ctypes.POINTER(LoRA), _P,
                                         _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P],
                                        ctypes.c_int),
            "qf_qad_kl": ([_P, _I, _P, _I, _I, _I, ctypes.c_float, _P, _P, _P, _I, _P, _P],
                          ctypes.c_int),
            "qf_export_fused": ([ctypes.c_int, ctypes.POINTER(Member), ctypes.c_int, _I, _P, _P,
                                 _P, _P, _P, _P, _P], ctypes.c_int),
            "qf_payload_layout_of": ([ctypes.c_int, _I, _I, ctypes.POINTER(PayloadLayout)],
                                     ctypes.c_int),
            "qf_payload_write_header": ([ctypes.c_int, _I, _I, _P, _P], ctypes.c_int),
            "qf_grouped_lora_workspace_size": ([ctypes.POINTER(GroupedDesc), ctypes.POINTER(LoRA),
                                                ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
            "qf_qlinear_grouped_lora_fwd": ([ctypes.POINTER(GroupedDesc), ctypes.POINTER(LoRA), _P,
                                             _P, _P, _P, _P, ctypes.c_size_t, _P], ctypes.c_int),
            "qf_qlinear_grouped_lora_bwd_ste": ([ctypes.POINTER(GroupedDesc), ctypes.POINTER(LoRA),
                                                 _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t,
                                                 _P], ctypes.c_int),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise QFError(status, lib().qf_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor")
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    return t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _bf16(t):
    if t is not None and t.element_size() != 2:
        raise TypeError("bf16 operand must have 2-byte elements")
    return t


def _rows(x):
    if x.dim() != 2:
        raise ValueError("expected a 2-D tensor")
    if x.stride(1) != 1:
        raise ValueError("rows must be contiguous")
    return x.shape[0], x.shape[1], x.stride(0)


def version() -> int:
    return lib().qf_version()


# ----------------------------------------------------------------------------- quantizers
def amax(x, out, accumulate: bool = False):
    R, K, ld = _rows(_bf16(x))
    _check(lib().qf_amax(_ptr(x), R, K, ld, _ptr(out), int(accumulate), _stream()))
    return out


def fakequant_nvfp4(x, amax, amax_mode=AMAX_COMPUTE, s_out=None, codes=None, scales=None,
                    xhat=None):
    R, K, ld = _rows(_bf16(x))
    _check(lib().qf_fakequant_nvfp4(_ptr(x), R, K, ld, _ptr(amax), int(amax_mode), _ptr(s_out),
                                    _ptr(codes), _ptr(scales), _ptr(xhat), _stream()))


def fakequant_mxfp4(x, codes=None, scales=None, xhat=None):
    R, K, ld = _rows(_bf16(x))
    _check(lib().qf_fakequant_mxfp4(_ptr(x), R, K, ld, _ptr(codes), _ptr(scales), _ptr(xhat),
                                    _stream()))


def fakequant_q4k(x, packed=None, xhat=None):
    R, K, ld = _rows(_bf16(x))
    _check(lib().qf_fakequant_q4k(_ptr(x), R, K, ld, _ptr(packed), _ptr(xhat), _stream()))


def fakequant_q4k_mse(x, packed=None, xhat=None):
    R, K, ld = _rows(_bf16(x))
    _check(lib().qf_fakequant_q4k_mse(_ptr(x), R, K, ld, _ptr(packed), _ptr(xhat), _stream()))


def fakequant_transposed(x, fmt, out, amax=None):
    """out[k][r] = x_hat[r][k] for x [R, K]; out is a [K, >=R] row-contiguous bf16 tensor."""
    R, K, ld = _rows(_bf16(x))
    if out.dim() != 2 or out.shape[0] != K or out.shape[1] < R or out.stride(1) != 1:
        raise ValueError("out must be a [K, >=R] row-contiguous tensor")
    _check(lib().qf_fakequant_transposed(FMT[fmt], _ptr(x), R, K, ld, _ptr(amax),
                                         _ptr(_bf16(out)), out.stride(0), _stream()))
    return out


# --------------------------------------------------------------------------- linear layer
def qlinear_desc(M, N, K, wfmt="nvfp4", afmt="none", w_amax=None, a_amax=None, flags=0,
                 ldx=0, ldw=0, ldy=0) -> QLinearDesc:
    return QLinearDesc(M, N, K, ldx, ldw, ldy, FMT[wfmt], FMT[afmt], _ptr(w_amax),
                       _ptr(a_amax), flags)


def workspace_size(desc: QLinearDesc) -> int:
    n = ctypes.c_size_t()
    _check(lib().qf_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def workspace(desc: QLinearDesc, device="cuda"):
    return torch.empty(max(workspace_size(desc), 256), dtype=torch.uint8, device=device)


def saved_size(desc: QLinearDesc) -> int:
    n = ctypes.c_size_t()
    _check(lib().qf_saved_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def saved_buffer(desc: QLinearDesc, device="cuda"):
    """A device buffer for the layer's saved (packed) operands, qf_saved_size bytes."""
    return torch.empty(max(saved_size(desc), 256), dtype=torch.uint8, device=device)


def qlinear_fwd(desc, X, W, Y, ws, saved=None):
    _check(lib().qf_qlinear_fwd(ctypes.byref(desc), _ptr(_bf16(X)), _ptr(_bf16(W)),
                                _ptr(_bf16(Y)), _ptr(saved), _ptr(ws), ws.numel(), _stream()))
    return Y


def qlinear_fwd_noalloc(desc, X, W, Y):
    """qf_qlinear_fwd_noalloc: the forward with the library's static device scratch."""
    _check(lib().qf_qlinear_fwd_noalloc(ctypes.byref(desc), _ptr(_bf16(X)), _ptr(_bf16(W)),
                                        _ptr(_bf16(Y)), _stream()))
    return Y


def qlinear_bwd_ste(desc, dY, X, W, dX, dW, ws, saved=None):
    _check(lib().qf_qlinear_bwd_ste(ctypes.byref(desc), _ptr(_bf16(dY)), _ptr(_bf16(X)),
                                    _ptr(_bf16(W)), _ptr(saved), _ptr(_bf16(dX)), _ptr(dW),
                                    _ptr(ws), ws.numel(), _stream()))


def grouped_desc(E, T, N, K, wfmt="nvfp4", afmt="none", w_amax=None, flags=0) -> GroupedDesc:
    return GroupedDesc(E, T, N, K, FMT[wfmt], FMT[afmt], _ptr(w_amax), flags)


def grouped_workspace(desc: GroupedDesc, device="cuda"):
    n = ctypes.c_size_t()
    _check(lib().qf_grouped_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return torch.empty(max(n.value, 256), dtype=torch.uint8, device=device)


def grouped_saved_size(desc: GroupedDesc) -> int:
    n = ctypes.c_size_t()
    _check(lib().qf_grouped_saved_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def grouped_saved_buffer(desc: GroupedDesc, device="cuda"):
    """A device buffer for the grouped layer's saved operand (the experts' packed W_hat)."""
    return torch.empty(max(grouped_saved_size(desc), 256), dtype=torch.uint8, device=device)


def qlinear_grouped_fwd(desc, offsets, X, W, Y, ws, saved=None):
    _check(lib().qf_qlinear_grouped_fwd(ctypes.byref(desc), _ptr(offsets), _ptr(_bf16(X)),
                                        _ptr(_bf16(W)), _ptr(_bf16(Y)), _ptr(saved), _ptr(ws),
                                        ws.numel(), _stream()))


def qlinear_grouped_bwd_ste(desc, offsets, dY, X, W, dX, dW, ws, saved=None):
    _check(lib().qf_qlinear_grouped_bwd_ste(ctypes.byref(desc), _ptr(offsets), _ptr(_bf16(dY)),
                                            _ptr(_bf16(X)), _ptr(_bf16(W)), _ptr(saved),
                                            _ptr(_bf16(dX)), _ptr(dW), _ptr(ws), ws.numel(),
                                            _stream()))


def gemm_bf16(M, N, K, A, lda, a_kmajor, B, ldb, b_kmajor, C, ldc, c_f32, ws=None):
    if ws is None:
        _check(lib().qf_gemm_bf16(M, N, K, _ptr(_bf16(A)), lda, int(a_kmajor), _ptr(_bf16(B)),
                                  ldb, int(b_kmajor), _ptr(C), ldc, int(c_f32), _stream()))
    else:
        _check(lib().qf_gemm_bf16_ws(M, N, K, _ptr(_bf16(A)), lda, int(a_kmajor), _ptr(_bf16(B)),
                                     ldb, int(b_kmajor), _ptr(C), ldc, int(c_f32), _ptr(ws),
                                     ws.numel() * ws.element_size(), _stream()))
    return C


def gemm_bf16_at(M, N, K, A, lda, B, ldb, C, ldc, at, ldat):
    _check(lib().qf_gemm_bf16_at(M, N, K, _ptr(_bf16(A)), lda, _ptr(_bf16(B)), ldb,
                                 _ptr(_bf16(C)), ldc, _ptr(_bf16(at)), ldat, _stream()))
    return C, at


def fragment_bytes(N, K) -> int:
    n = ctypes.c_size_t()
    _check(lib().qf_fragment_bytes(N, K, ctypes.byref(n)))
    return n.value


def pack_fragments(B, out):
    """qf_pack_fragments: out (a flat 16-bit tensor of fragment_bytes(N, K) bytes) from B [N, K]."""
    N, K, ld = _rows(_bf16(B))
    _check(lib().qf_pack_fragments(_ptr(_bf16(B)), N, K, ld, _ptr(out), _stream()))
    return out


def gemm_bf16_fragb(M, N, K, A, lda, Bf, C, ldc, c_f32, ws=None):
    """qf_gemm_bf16_fragb: C = A B^T with B in the fragment-major layout."""
    _check(lib().qf_gemm_bf16_fragb(M, N, K, _ptr(_bf16(A)), lda, _ptr(Bf), _ptr(C), ldc,
                                    int(c_f32), _ptr(ws), 0 if ws is None else ws.numel(),
                                    _stream()))
    return C


def gemm_packed_b(M, N, K, A, lda, fmt, codes, scales, S, C, ldc):
    """qf_gemm_packed_b: C = A W_hat^T with W_hat decoded inside the GEMM from packed codes."""
    _check(lib().qf_gemm_packed_b(M, N, K, _ptr(_bf16(A)), lda, FMT[fmt], _ptr(codes),
                                  _ptr(scales), _ptr(S), _ptr(_bf16(C)), ldc, _stream()))
    return C


def dequantize_transposed(fmt, codes, scales, S, R, K, out):
    """qf_dequantize_transposed: out[k][r] = x_hat[r][k] from packed codes (out [K, >=R])."""
    if out.dim() != 2 or out.shape[0] != K or out.shape[1] < R or out.stride(1) != 1:
        raise ValueError("out must be a [K, >=R] row-contiguous tensor")
    _check(lib().qf_dequantize_transposed(FMT[fmt], _ptr(codes), _ptr(scales), _ptr(S), R, K,
                                          _ptr(_bf16(out)), out.stride(0), _stream()))
    return out


def gemm_workspace(M, N, c_f32, device="cuda"):
    n = ctypes.c_size_t()
    _check(lib().qf_gemm_workspace_size(M, N, int(c_f32), ctypes.byref(n)))
    return torch.empty(max(n.value, 256), dtype=torch.uint8, device=device)


def transpose_bf16(x, out):
    """out[c][r] = x[r][c] (bf16, R and C multiples of 8)."""
    R, C, ld = _rows(_bf16(x))
    if out.dim() != 2 or out.shape[0] != C or out.shape[1] < R or out.stride(1) != 1:
        raise ValueError("out must be a [C, >=R] row-contiguous tensor")
    _check(lib().qf_transpose_bf16(_ptr(x), R, C, ld, _ptr(_bf16(out)), out.stride(0), _stream()))
    return out


# --------------------------------------------------------------------------- LoRA-QAD
def lora(A, B, scale=1.0, a_shared=False, b_shared=False) -> LoRA:
    """Adapter descriptor: A FP32 [r, K] (or [E, r, K]), B FP32 [N, r] (or [E, N, r]).
    The descriptor holds references to A and B, so the device memory it points to stays
    allocated while the descriptor is alive."""
    for t in (A, B):
        if t.dtype != torch.float32 or not t.is_contiguous():
            raise TypeError("LoRA factors must be contiguous float32 tensors")
    r = A.shape[-2]
    if B.shape[-1] != r:
        raise ValueError("A is [.., r, K] and B is [.., N, r]")
    lo = LoRA(_ptr(A), _ptr(B), r, float(scale), int(a_shared), int(b_shared))
    lo._factors = (A, B)
    return lo


def lora_amax(W, lo: LoRA, out, accumulate: bool = False):
    N, K, ld = _rows(_bf16(W))
    _check(lib().qf_lora_amax(_ptr(W), N, K, ld, ctypes.byref(lo), _ptr(out), int(accumulate),
                              _stream()))
    return out


def lora_fakequant(W, lo: LoRA, fmt, amax=None, amax_mode=AMAX_COMPUTE, s_out=None, codes=None,
                   scales=None, packed=None, xhat=None):
    N, K, ld = _rows(_bf16(W))
    _check(lib().qf_lora_fakequant(FMT[fmt], _ptr(W), N, K, ld, ctypes.byref(lo), _ptr(amax),
                                   amax_mode, _ptr(s_out), _ptr(codes), _ptr(scales),
                                   _ptr(packed), _ptr(_bf16(xhat)), _stream()))


def lora_fakequant_transposed(W, lo: LoRA, fmt, out, amax=None):
    N, K, ld = _rows(_bf16(W))
    if out.dim() != 2 or out.shape[0] != K or out.shape[1] < N or out.stride(1) != 1:
        raise ValueError("out must be a [K, >=N] row-contiguous tensor")
    _check(lib().qf_lora_fakequant_transposed(FMT[fmt], _ptr(W), N, K, ld, ctypes.byref(lo),
                                              _ptr(amax), _ptr(_bf16(out)), out.stride(0),
                                              _stream()))
    return out


def lora_workspace(desc: QLinearDesc, lo: LoRA, device="cuda"):
    n = ctypes.c_size_t()
    _check(lib().qf_lora_workspace_size(ctypes.byref(desc), ctypes.byref(lo), ctypes.byref(n)))
    return torch.empty(max(n.value, 256), dtype=torch.uint8, device=device)


def qlinear_lora_fwd(desc, lo: LoRA, X, W, Y, ws):
    _check(lib().qf_qlinear_lora_fwd(ctypes.byref(desc), ctypes.byref(lo), _ptr(_bf16(X)),
                                     _ptr(_bf16(W)), _ptr(_bf16(Y)), _ptr(ws), ws.numel(),
                                     _stream()))
    return Y


def qlinear_lora_bwd_ste(desc, lo: LoRA, dY, X, W, dX, dA, dB, ws):
    _check(lib().qf_qlinear_lora_bwd_ste(ctypes.byref(desc), ctypes.byref(lo), _ptr(_bf16(dY)),
                                         _ptr(_bf16(X)), _ptr(_bf16(W)), _ptr(_bf16(dX)),
                                         _ptr(dA), _ptr(dB), _ptr(ws), ws.numel(), _stream()))


def grouped_lora_workspace(desc: GroupedDesc, lo: LoRA, device="cuda"):
    n = ctypes.c_size_t()
    _check(lib().qf_grouped_lora_workspace_size(ctypes.byref(desc), ctypes.byref(lo),
                                                ctypes.byref(n)))
    return torch.empty(max(n.value, 256), dtype=torch.uint8, device=device)


def qlinear_grouped_lora_fwd(desc, lo: LoRA, offsets, X, W, Y, ws):
    _check(lib().qf_qlinear_grouped_lora_fwd(ctypes.byref(desc), ctypes.byref(lo), _ptr(offsets),
                                             _ptr(_bf16(X)), _ptr(_bf16(W)), _ptr(_bf16(Y)),
                                             _ptr(ws), ws.numel(), _stream()))


def qlinear_grouped_lora_bwd_ste(desc, lo: LoRA, offsets, dY, X, W, dX, dA, dB, ws):
    _check(lib().qf_qlinear_grouped_lora_bwd_ste(ctypes.byref(desc), ctypes.byref(lo),
                                                 _ptr(offsets), _ptr(_bf16(dY)), _ptr(_bf16(X)),
                                                 _ptr(_bf16(W)), _ptr(_bf16(dX)), _ptr(dA),
                                                 _ptr(dB), _ptr(ws), ws.numel(), _stream()))


# ------------------------------------------------------------------ QAD distillation loss
def qad_kl(zt, zs, row_kl, loss=None, grad=None, agree=None, grad_scale=None):
    """Forward KL of Eq. qad-objective per token (row_kl), its mean (loss), the student-logit
    gradient grad_scale * (p_S - p_T) (default grad_scale = 1/L) and top-1 agreement."""
    L, V, ldt = _rows(_bf16(zt))
    L2, V2, lds = _rows(_bf16(zs))
    if (L2, V2) != (L, V):
        raise ValueError("teacher and student logits must have the same shape")
    ldg = 0
    if grad is not None:
        _, _, ldg = _rows(_bf16(grad))
    gs = (1.0 / L if L else 1.0) if grad_scale is None else float(grad_scale)
    _check(lib().qf_qad_kl(_ptr(zt), ldt, _ptr(zs), lds, L, V, gs, _ptr(row_kl), _ptr(loss),
                           _ptr(grad), ldg, _ptr(agree), _stream()))


# --------------------------------------------------------------- engine-native export / sync
def export_fused(members, fmt, codes, scales, w_amax=None, weight_scale_2=None, a_amax=None,
                 input_scale=None):
    """Fused-projection export: members are bf16 [rows_i, K] tensors (row-contiguous)."""
    K = members[0].shape[1]
    arr = (Member * len(members))()
    for i, m in enumerate(members):
        R, Km, ld = _rows(_bf16(m))
        if Km != K:
            raise ValueError("members must share K")
        arr[i] = Member(_ptr(m), R, ld)
    _check(lib().qf_export_fused(FMT[fmt], arr, len(members), K, _ptr(codes), _ptr(scales),
                                 _ptr(w_amax), _ptr(weight_scale_2), _ptr(a_amax),
                                 _ptr(input_scale), _stream()))


def payload_layout(fmt, N, K) -> PayloadLayout:
    L = PayloadLayout()
    _check(lib().qf_payload_layout_of(FMT[fmt], N, K, ctypes.byref(L)))
    return L


def payload_write_header(fmt, N, K, payload):
    _check(lib().qf_payload_write_header(FMT[fmt], N, K, _ptr(payload), _stream()))
