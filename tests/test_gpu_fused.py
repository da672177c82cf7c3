"""GPU parity of the forward that decodes the packed weight inside the GEMM (Eq. fakequant with
Q^-1 in the GEMM's prologue), of the layer's saved operands (the packed W_hat / A_hat kept for
the backward, Sec. 3.2.1) and of the backward that dequantizes them straight into the
transposed GEMM operands.

- The fused forward (QF_FLAG_DECODE_IN_GEMM) against the forward that writes W_hat in bf16:
  bit-identical Y, and within the Q26 tolerance of the FP64 oracle.
- The saved buffer against the oracle's codes, scales, tensor scale and Q4_K blocks, bit for bit.
- The backward from the saved buffer against the backward that quantizes again and the one that
  reuses the workspace: bit-identical dX and dW, and within tolerance of the oracle.
"""
import numpy as np
import pytest

import oracle
import workloads
from tests.helpers import assert_close, bf16_to_f64, empty_bf16, from_dev, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def qf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_39223_amd as qf
    qf.lib()
    return qf


def _inputs(seed, M, N, K, ld_pad=0):
    rng = np.random.default_rng(seed)
    tau = np.abs(rng.standard_t(3.0, size=K)).astype(np.float32)
    return {"X": workloads.normal_bf16(rng, (M, K), 1.0, col_scale=tau),
            "W": workloads.normal_bf16(rng, (N, K), 0.02),
            "dY": workloads.normal_bf16(rng, (M, N), 1.0)}


def _strided_dev(a, pad):
    if not pad:
        return to_dev(a)
    R, C = a.shape
    buf = np.full((R, C + pad), 0x7FC0, np.uint16)     # NaN padding: never read
    buf[:, :C] = a
    return to_dev(buf)[:, :C]


def _a_amax(w, afmt):
    if afmt != "nvfp4":
        return None, None
    g = float(np.float32(1.25 * oracle.amax(w["X"])))   # a running amax above this batch's
    return torch.tensor([g], dtype=torch.float32, device="cuda"), g


def _ref_operands(w, wfmt, afmt, a_amax):
    what = oracle.fakequant(w["W"], wfmt) if wfmt != "none" else w["W"]
    ahat = oracle.fakequant(w["X"], afmt, a_amax) if afmt != "none" else w["X"]
    return what, ahat


CASES = [("nvfp4", "none", 264, 520, 512, 0),       # ragged M and N, 8 stages
         ("mxfp4", "mxfp4", 300, 1000, 1024, 8),     # 16 stages: rotated k start per XCD
         ("q4k", "none", 256, 264, 768, 0),          # 3 super-blocks per row
         ("nvfp4", "nvfp4", 520, 256, 4096, 0),      # NVFP4 activations, running amax
         ("mxfp4", "none", 8, 2056, 64, 0),          # one stage, 9 tile columns
         ("nvfp4", "none", 1, 8, 128, 16),           # one row, one ragged tile
         ("q4k", "none", 600, 2048, 4096, 0)]        # 16 super-blocks, 8 x 3 tiles


@pytest.mark.parametrize("wfmt,afmt,M,N,K,pad", CASES)
def test_fused_forward_equals_materialized_and_oracle(qf, wfmt, afmt, M, N, K, pad):
    w = _inputs(M + N + K, M, N, K)
    X, W = _strided_dev(w["X"], pad), _strided_dev(w["W"], pad)
    a_amax, g = _a_amax(w, afmt)
    Ys = []
    for flags in (qf.FLAG_DECODE_IN_GEMM, 0):
        d = qf.qlinear_desc(M, N, K, wfmt, afmt, a_amax=a_amax, flags=flags,
                            ldx=X.stride(0), ldw=W.stride(0))
        ws = qf.workspace(d)
        Y = torch.full((M, N), 0x7FC0, dtype=torch.int16, device="cuda")
        qf.qlinear_fwd(d, X, W, Y, ws)
        torch.cuda.synchronize()
        Ys.append(from_dev(Y).view(np.uint16))
    assert np.array_equal(Ys[0], Ys[1]), "fused and materialized forwards differ"
    what, ahat = _ref_operands(w, wfmt, afmt, g)
    assert_close(bf16_to_f64(Ys[0]), oracle.linear_fwd(ahat, what), "Y")


def test_fused_forward_nonfinite_tensor_scale(qf):
    """A caller-given infinite amax: every decoded weight is +-inf or NaN; the fused and the
    materialized forwards give NaN / inf at the same places (NaN payloads unspecified)."""
    M, N, K = 264, 264, 256
    w = _inputs(5, M, N, K)
    g = torch.tensor([float("inf")], dtype=torch.float32, device="cuda")
    out = []
    for flags in (qf.FLAG_DECODE_IN_GEMM, 0):
        d = qf.qlinear_desc(M, N, K, "nvfp4", "none", w_amax=g, flags=flags)
        Y = empty_bf16((M, N))
        qf.qlinear_fwd(d, to_dev(w["X"]), to_dev(w["W"]), Y, qf.workspace(d))
        torch.cuda.synchronize()
        out.append(bf16_to_f64(from_dev(Y)))
    assert np.array_equal(np.isnan(out[0]), np.isnan(out[1]))
    fin = ~np.isnan(out[0])
    assert np.array_equal(out[0][fin], out[1][fin])


def _parse_packed(buf, fmt, R, K, off):
    def up(v):
        return (v + 255) // 256 * 256
    out = {}
    if fmt == "nvfp4":
        out["S"] = float(buf[off:off + 4].view(np.float32)[0])
        off += 256
    if fmt in ("nvfp4", "mxfp4"):
        out["codes"] = buf[off:off + R * K // 2].reshape(R, K // 2)
        off += up(R * K // 2)
        B = 16 if fmt == "nvfp4" else 32
        out["scales"] = buf[off:off + R * K // B].reshape(R, K // B)
        off += up(R * K // B)
    elif fmt == "q4k":
        out["packed"] = buf[off:off + R * (K // 256) * 144].reshape(R, K // 256, 144)
        off += up(R * (K // 256) * 144)
    return out, off


@pytest.mark.parametrize("wfmt,afmt", [("nvfp4", "none"), ("mxfp4", "mxfp4"), ("q4k", "none"),
                                       ("nvfp4", "nvfp4"), ("nvfp4", "mxfp4")])
def test_saved_operands_are_the_quantizers_packed_outputs(qf, wfmt, afmt):
    M, N, K = 136, 264, 512
    w = _inputs(17, M, N, K)
    a_amax, g = _a_amax(w, afmt)
    d = qf.qlinear_desc(M, N, K, wfmt, afmt, a_amax=a_amax)
    saved = torch.full((qf.saved_size(d),), 0xA5, dtype=torch.uint8, device="cuda")
    Y = empty_bf16((M, N))
    qf.qlinear_fwd(d, to_dev(w["X"]), to_dev(w["W"]), Y, qf.workspace(d), saved=saved)
    torch.cuda.synchronize()
    buf = from_dev(saved)
    pw, off = _parse_packed(buf, wfmt, N, K, 0)
    ref = {"nvfp4": oracle.nvfp4, "mxfp4": oracle.mxfp4, "q4k": oracle.q4k}[wfmt](w["W"])
    for k in ("codes", "scales", "packed"):
        if k in pw:
            np.testing.assert_array_equal(pw[k], ref[k], err_msg=f"W {k}")
    if wfmt == "nvfp4":
        assert pw["S"] == ref["S"]
    if afmt != "none":
        pa, off2 = _parse_packed(buf, afmt, M, K, off)
        assert off2 == qf.saved_size(d)
        refa = oracle.nvfp4(w["X"], g) if afmt == "nvfp4" else oracle.mxfp4(w["X"])
        np.testing.assert_array_equal(pa["codes"], refa["codes"], err_msg="X codes")
        np.testing.assert_array_equal(pa["scales"], refa["scales"], err_msg="X scales")
        if afmt == "nvfp4":
            assert pa["S"] == refa["S"]
    else:
        assert off == qf.saved_size(d)


@pytest.mark.parametrize("wfmt,afmt,M,N,K", [("nvfp4", "none", 264, 520, 512),
                                             ("mxfp4", "mxfp4", 392, 264, 544),
                                             ("q4k", "none", 264, 264, 768),
                                             ("nvfp4", "nvfp4", 200, 256, 512),
                                             ("mxfp4", "mxfp4", 16384, 136, 1280),
                                             ("nvfp4", "none", 13, 264, 256)])
def test_backward_from_saved_equals_requantized(qf, wfmt, afmt, M, N, K):
    """dX and dW from the saved packed operands (transposing dequantizer), from re-quantization
    and from the reused workspace: bit for bit the same (padded 16384-token strides, a token
    count that is not a multiple of 8), and within tolerance of the oracle."""
    w = _inputs(M * 3 + N + K, M, N, K)
    X, W, dY = to_dev(w["X"]), to_dev(w["W"]), to_dev(w["dY"])
    a_amax, g = _a_amax(w, afmt)
    outs = []
    for mode in ("saved", "requantize", "reuse"):
        d = qf.qlinear_desc(M, N, K, wfmt, afmt, a_amax=a_amax,
                            flags=qf.FLAG_REUSE_WS if mode == "reuse" else 0)
        ws = qf.workspace(d)
        saved = qf.saved_buffer(d) if mode == "saved" else None
        Y = empty_bf16((M, N))
        qf.qlinear_fwd(d, X, W, Y, ws, saved=saved)
        dX = empty_bf16((M, K))
        dW = torch.full((N, K), 7.0, dtype=torch.float32, device="cuda")
        qf.qlinear_bwd_ste(d, dY, X, W, dX, dW, ws, saved=saved)
        torch.cuda.synchronize()
        outs.append((from_dev(dX).view(np.uint16), from_dev(dW).view(np.uint32)))
    for name, (a, b) in zip(("requantize", "reuse"), outs[1:]):
        assert np.array_equal(outs[0][0], a), f"dX saved vs {name}"
        assert np.array_equal(outs[0][1], b), f"dW saved vs {name}"
    what, ahat = _ref_operands(w, wfmt, afmt, g)
    assert_close(bf16_to_f64(outs[0][0]), oracle.linear_dx(w["dY"], what), "dX")
    assert_close(outs[0][1].view(np.float32).astype(np.float64), oracle.linear_dw(w["dY"], ahat), "dW")
