"""Host-only checks of the C ABI library: it loads, exports every symbol include/qf.h
declares, and rejects invalid arguments before touching the GPU (no kernel is launched
by any call here: each one fails host validation)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qf.h")
LIB = os.path.join(ROOT, "paper_2609_39223_amd", "libqf.so")

QF_OK, QF_EINVAL, QF_ESHAPE, QF_EALIGN, QF_ENOTSUP = 0, 1, 2, 3, 4


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"QF_API\s+[\w\s\*]*?\b(qf_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(LIB):
        pytest.skip("libqf.so not built (run __graft_entry__.build())")
    import torch  # noqa: F401  (same HIP runtime as the GPU path)
    lib = ctypes.CDLL(LIB)
    lib.qf_last_error.restype = ctypes.c_char_p
    return lib


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for s in ["qf_fakequant_nvfp4", "qf_fakequant_mxfp4", "qf_fakequant_q4k", "qf_amax",
              "qf_qlinear_fwd", "qf_qlinear_bwd_ste", "qf_qlinear_grouped_fwd",
              "qf_qlinear_grouped_bwd_ste", "qf_workspace_size", "qf_last_error", "qf_version"]:
        assert s in syms


def test_library_exports_every_declared_symbol(L):
    for s in declared_symbols():
        assert hasattr(L, s), s
    assert L.qf_version() >= 100


I64 = ctypes.c_int64
P = ctypes.c_void_p


def test_quantizer_validation(L):
    f = L.qf_fakequant_mxfp4
    assert f(P(256), I64(4), I64(40), I64(40), None, None, None, None) == QF_ESHAPE
    assert b"multiple" in L.qf_last_error()
    assert f(None, I64(4), I64(64), I64(64), None, None, None, None) == QF_EINVAL
    assert f(P(258), I64(4), I64(64), I64(64), None, None, None, None) == QF_EALIGN
    assert f(P(256), I64(4), I64(64), I64(60), None, None, None, None) == QF_ESHAPE
    assert f(P(256), I64(4), I64(64), I64(68), None, None, None, None) == QF_EALIGN
    assert f(P(256), I64(-1), I64(64), I64(64), None, None, None, None) == QF_ESHAPE
    g = L.qf_fakequant_nvfp4
    assert g(P(256), I64(4), I64(24), I64(24), P(512), 0, None, None, None, None, None) == QF_ESHAPE
    assert g(P(256), I64(4), I64(32), I64(32), None, 0, None, None, None, None, None) == QF_EINVAL
    assert g(P(256), I64(4), I64(32), I64(32), P(512), 7, None, None, None, None, None) == QF_EINVAL
    assert g(P(256), I64(4), I64(32), I64(32), P(512), 0, P(512), None, None, None, None) == QF_EINVAL
    h = L.qf_fakequant_q4k
    assert h(P(256), I64(4), I64(128), I64(128), None, None, None) == QF_ESHAPE
    assert h(P(256), I64(4), I64(256), I64(256), P(7), None, None) == QF_EALIGN
    t = L.qf_fakequant_transposed
    t.argtypes = [ctypes.c_int, P, I64, I64, I64, P, P, I64, P]
    assert t(0, P(256), 8, 64, 64, None, P(256), 8, None) == QF_EINVAL         # format NONE
    assert t(2, P(256), 12, 64, 64, None, P(256), 16, None) == QF_ESHAPE       # R % 8
    assert t(2, P(256), 8, 48, 48, None, P(256), 8, None) == QF_ESHAPE         # K % 32
    assert t(1, P(256), 8, 64, 64, None, P(256), 8, None) == QF_EINVAL         # NVFP4 amax
    assert t(2, P(256), 8, 64, 64, None, None, 8, None) == QF_EINVAL           # no output
    assert t(2, P(256), 8, 64, 64, None, P(256), 4, None) == QF_ESHAPE         # ldo < R
    assert t(3, P(256), 8, 256, 256, None, P(264), 8, None) == QF_EALIGN       # out alignment


class Desc(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("ldx", ctypes.c_int64), ("ldw", ctypes.c_int64), ("ldy", ctypes.c_int64),
                ("wfmt", ctypes.c_int32), ("afmt", ctypes.c_int32),
                ("w_amax", ctypes.c_void_p), ("a_amax", ctypes.c_void_p),
                ("flags", ctypes.c_uint32)]


def test_workspace_size_and_desc_validation(L):
    n = ctypes.c_size_t()
    d = Desc(256, 512, 512, 0, 0, 0, 1, 0, None, None, 0)
    assert L.qf_workspace_size(ctypes.byref(d), ctypes.byref(n)) == QF_OK
    assert n.value >= 512 * 512 * 2
    d2 = Desc(256, 512, 512, 0, 0, 0, 2, 2, None, None, 0)
    assert L.qf_workspace_size(ctypes.byref(d2), ctypes.byref(n)) == QF_OK
    assert n.value >= (512 + 256) * 512 * 2
    bad = [Desc(256, 512, 500, 0, 0, 0, 1, 0, None, None, 0),   # K % 16
           Desc(256, 512, 512, 0, 0, 0, 3, 3, None, None, 0),   # Q4_K activations
           Desc(256, 512, 512, 0, 0, 0, 1, 1, None, None, 0),   # NVFP4 act without a_amax
           Desc(256, 512, 512, 0, 0, 0, 9, 0, None, None, 0),   # bad enum
           Desc(-1, 512, 512, 0, 0, 0, 1, 0, None, None, 0)]
    want = [QF_ESHAPE, QF_ENOTSUP, QF_EINVAL, QF_EINVAL, QF_ESHAPE]
    for dd, w in zip(bad, want):
        assert L.qf_workspace_size(ctypes.byref(dd), ctypes.byref(n)) == w
    # too-small workspace is rejected before any launch
    assert L.qf_qlinear_fwd(ctypes.byref(d), P(256), P(256), P(256), None, P(256),
                            ctypes.c_size_t(16), None) == QF_EINVAL
    assert b"workspace" in L.qf_last_error()
    # a misaligned saved buffer too
    assert L.qf_qlinear_fwd(ctypes.byref(d), P(256), P(256), P(256), P(272), P(256),
                            ctypes.c_size_t(1 << 40), None) == QF_EALIGN
    assert b"saved" in L.qf_last_error()


def test_saved_size_is_the_packed_operands(L):
    """qf_saved_size: packed W (and A when quantized), each region 256-byte aligned:
    NVFP4 256 B (S) + codes K/2 + E4M3 scales K/16 per row; MXFP4 codes + K/32 scales;
    Q4_K 144 bytes per 256 elements (Sec. 3.2.1's transient operands in deployment form)."""
    def up(v):
        return (v + 255) // 256 * 256
    n = ctypes.c_size_t()
    M, N, K = 264, 520, 512
    cases = [(1, 0, 256 + up(N * K // 2) + up(N * K // 16)),
             (2, 2, up(N * K // 2) + up(N * K // 32) + up(M * K // 2) + up(M * K // 32)),
             (3, 0, up(N * (K // 256) * 144)),
             (1, 1, 256 + up(N * K // 2) + up(N * K // 16) + 256 + up(M * K // 2) + up(M * K // 16)),
             (0, 0, 0)]
    for wf, af, want in cases:
        d = Desc(M, N, K, 0, 0, 0, wf, af, None, P(256) if af == 1 else None, 0)
        assert L.qf_saved_size(ctypes.byref(d), ctypes.byref(n)) == QF_OK
        assert n.value == want, (wf, af)
        assert n.value <= 0.5625 * (N + (M if af else 0)) * K + 3 * 256 + 2 * 256


class GDesc(ctypes.Structure):
    _fields_ = [("E", ctypes.c_int64), ("T", ctypes.c_int64), ("N", ctypes.c_int64),
                ("K", ctypes.c_int64), ("wfmt", ctypes.c_int32), ("afmt", ctypes.c_int32),
                ("w_amax", ctypes.c_void_p), ("flags", ctypes.c_uint32)]


def test_grouped_saved_size_and_validation(L):
    """qf_grouped_saved_size: the experts' packed W_hat back to back (NVFP4: one FP32 decode
    scale per expert in a 256-byte aligned region, then codes and E4M3 scales of all E N rows);
    qf_validate_grouped checks the saved buffer's alignment as the calls do."""
    def up(v):
        return (v + 255) // 256 * 256
    n = ctypes.c_size_t()
    E, T, N, K = 128, 1000, 3072, 1536
    for wf, want in [(1, up(4 * E) + up(E * N * K // 2) + up(E * N * K // 16)),
                     (2, up(E * N * K // 2) + up(E * N * K // 32)),
                     (3, up(E * N * (K // 256) * 144)), (0, 0)]:
        d = GDesc(E, T, N, K, wf, 0, None, 0)
        assert L.qf_grouped_saved_size(ctypes.byref(d), ctypes.byref(n)) == QF_OK
        assert n.value == want, wf
    d = GDesc(E, T, N, K, 1, 0, None, 0)
    assert L.qf_grouped_workspace_size(ctypes.byref(d), ctypes.byref(n)) == QF_OK
    vg = L.qf_validate_grouped
    vg.argtypes = [ctypes.POINTER(GDesc), P, P, P, P, P, ctypes.c_size_t]
    assert vg(ctypes.byref(d), P(256), P(512), P(768), P(1024), P(4096), n.value) == QF_OK
    assert vg(ctypes.byref(d), P(256), P(512), P(768), None, P(4096), n.value) == QF_OK
    assert vg(ctypes.byref(d), P(256), P(512), P(768), P(1040), P(4096), n.value) == QF_EALIGN
    assert b"saved" in L.qf_last_error()
    assert vg(ctypes.byref(d), P(256), P(512), P(768), P(1024), P(4096), n.value - 1) == QF_EINVAL


def test_validate_calls_mirror_the_entry_points(L):
    """qf_validate_*: host-only checks that return what the call itself would, without a
    launch (every case here would fail before one)."""
    v = L.qf_validate_fakequant
    assert v(1, P(256), I64(4), I64(64), I64(64)) == QF_OK
    assert v(2, P(256), I64(4), I64(48), I64(48)) == QF_ESHAPE        # K % 32
    assert b"multiple" in L.qf_last_error()
    assert v(3, P(256), I64(4), I64(512), I64(512)) == QF_OK
    assert v(3, P(256), I64(4), I64(384), I64(384)) == QF_ESHAPE      # K % 256
    assert v(9, P(256), I64(4), I64(64), I64(64)) == QF_EINVAL        # format
    assert v(1, P(264), I64(4), I64(64), I64(64)) == QF_EALIGN
    assert v(1, None, I64(4), I64(64), I64(64)) == QF_EINVAL
    n = ctypes.c_size_t()
    d = Desc(256, 512, 512, 0, 0, 0, 2, 2, None, None, 0)
    assert L.qf_workspace_size(ctypes.byref(d), ctypes.byref(n)) == QF_OK
    vq = L.qf_validate_qlinear
    vq.argtypes = [ctypes.POINTER(Desc), P, P, P, P, P, ctypes.c_size_t]
    assert vq(ctypes.byref(d), P(256), P(512), P(768), P(1024), P(4096), n.value) == QF_OK
    assert vq(ctypes.byref(d), P(256), P(512), P(768), P(1024), P(4096), n.value - 1) == QF_EINVAL
    assert vq(ctypes.byref(d), P(256), P(512), P(768), P(1040), P(4096), n.value) == QF_EALIGN
    assert vq(ctypes.byref(d), P(256), None, P(768), None, P(4096), n.value) == QF_EINVAL
    bad = Desc(256, 512, 500, 0, 0, 0, 1, 0, None, None, 0)
    assert vq(ctypes.byref(bad), P(256), P(512), P(768), None, P(4096), 1 << 40) == QF_ESHAPE
    nv_act = Desc(256, 512, 512, 0, 0, 0, 1, 1, None, None, 0)        # NVFP4 A needs a_amax
    assert vq(ctypes.byref(nv_act), P(256), P(512), P(768), None, P(4096), 1 << 40) == QF_EINVAL


def test_gemm_validation(L):
    f = L.qf_gemm_bf16
    args = lambda M, N, K, lda, ak, ldb, bk: f(I64(M), I64(N), I64(K), P(256), I64(lda), ak, P(256),
                                               I64(ldb), bk, P(256), I64(N), 0, None)
    assert args(64, 64, 60, 60, 1, 60, 1) == QF_ESHAPE      # K % 8 for k-major operands
    assert args(60, 64, 64, 64, 0, 64, 1) == QF_ESHAPE      # M % 8 for [K][M] A
    assert args(64, 64, 64, 32, 1, 64, 1) == QF_ESHAPE      # lda < K


def test_library_has_no_undefined_kernel_stubs():
    import shutil
    import subprocess
    if not os.path.exists(LIB) or shutil.which("nm") is None:
        pytest.skip("needs the built library and nm")
    out = subprocess.run(["nm", "--undefined-only", LIB], capture_output=True, text=True).stdout
    assert "__device_stub" not in out


class LoRA(ctypes.Structure):
    _fields_ = [("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("r", ctypes.c_int64),
                ("scale", ctypes.c_float), ("a_shared", ctypes.c_int32),
                ("b_shared", ctypes.c_int32)]


def test_lora_validation(L):
    f = L.qf_lora_fakequant
    lo = LoRA(256, 512, 16, 1.0, 0, 0)
    args = lambda fmt, lo_, codes=None, scales=None, packed=None, s_out=None, K=64: f(
        fmt, P(256), I64(8), I64(K), I64(K), ctypes.byref(lo_) if lo_ is not None else None,
        P(1024), 0, s_out, codes, scales, packed, None, None)
    assert args(2, None) == QF_EINVAL                                   # null descriptor
    assert args(2, LoRA(256, 512, 0, 1.0, 0, 0)) == QF_ESHAPE           # rank 0
    assert args(2, LoRA(256, 512, 5000, 1.0, 0, 0)) == QF_ESHAPE        # rank too large
    assert args(2, LoRA(None, 512, 4, 1.0, 0, 0)) == QF_EINVAL          # null factor
    assert args(2, LoRA(260, 512, 4, 1.0, 0, 0)) == QF_EALIGN           # misaligned factor
    assert args(3, lo, codes=P(256), K=256) == QF_EINVAL                # codes with Q4_K
    assert args(2, lo, packed=P(256)) == QF_EINVAL                      # packed with MXFP4
    assert args(2, lo, s_out=P(256)) == QF_EINVAL                       # s_out with MXFP4
    assert args(2, lo, K=48) == QF_ESHAPE                               # K % 32
    assert args(9, lo) == QF_EINVAL                                     # bad format
    t = L.qf_lora_fakequant_transposed
    assert t(2, P(256), I64(12), I64(64), I64(64), ctypes.byref(lo), None, P(256), I64(16),
             None) == QF_ESHAPE                                         # N % 8
    assert t(1, P(256), I64(8), I64(64), I64(64), ctypes.byref(lo), None, P(256), I64(8),
             None) == QF_EINVAL                                         # NVFP4 without amax
    n = ctypes.c_size_t()
    d = Desc(256, 512, 512, 0, 0, 0, 2, 2, None, None, 0)
    assert L.qf_lora_workspace_size(ctypes.byref(d), ctypes.byref(lo), ctypes.byref(n)) == QF_OK
    assert n.value >= (2 * 512 * 512 + 256 * 512) * 2                   # W_hat, W_hat^T, A_hat
    assert L.qf_qlinear_lora_fwd(ctypes.byref(d), ctypes.byref(lo), P(256), P(256), P(256),
                                 P(256), ctypes.c_size_t(16), None) == QF_EINVAL
    assert b"workspace" in L.qf_last_error()


class Member(ctypes.Structure):
    _fields_ = [("W", ctypes.c_void_p), ("rows", ctypes.c_int64), ("ldw", ctypes.c_int64)]


def test_export_validation(L):
    m = (Member * 9)(*[Member(256, 8, 64) for _ in range(9)])
    f = L.qf_export_fused
    args = lambda fmt, n, w_amax=None, ws2=None, K=64: f(fmt, m, n, I64(K), P(256), P(512), w_amax,
                                                         ws2, None, None, None)
    assert args(2, 0) == QF_EINVAL                         # no members
    assert args(2, 9) == QF_EINVAL                         # more than 8
    assert args(3, 2) == QF_EINVAL                         # Q4_K is not an FP4 export format
    assert args(2, 2, w_amax=P(1024)) == QF_EINVAL         # MXFP4 has no tensor scale
    assert args(1, 2) == QF_EINVAL                         # NVFP4 needs w_amax
    assert args(2, 2, K=48) == QF_ESHAPE                   # K % 32
    class Lay(ctypes.Structure):
        _fields_ = [("codes", ctypes.c_uint64), ("scales", ctypes.c_uint64),
                    ("scalars", ctypes.c_uint64), ("total", ctypes.c_uint64)]
    lay = Lay()
    assert L.qf_payload_layout_of(1, I64(160), I64(512), ctypes.byref(lay)) == QF_OK
    assert (lay.codes, lay.scales, lay.scalars) == (256, 256 + 40960, 256 + 40960 + 5120)
    assert L.qf_payload_layout_of(3, I64(160), I64(512), ctypes.byref(lay)) == QF_EINVAL
    assert L.qf_payload_write_header(1, I64(160), I64(512), P(128), None) == QF_EALIGN
