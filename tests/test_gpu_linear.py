"""GPU parity of the MFMA GEMMs and the quantization-aware linear layer (forward +
straight-through backward) against the FP64 oracle on the same fake-quantized operands.

Tolerance (FP32 accumulation, bf16 outputs): per entry |y - r| / max(|r|, 1e-3 rms(r)),
max <= 2e-2 and mean <= 2e-3 (bf16 output rounding alone gives max 2^-9 ~ 1.95e-3).
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


def _rand_bf16(rng, shape, std=1.0):
    return workloads.normal_bf16(rng, shape, std)


# ---------------------------------------------------------------------------- plain GEMMs
@pytest.mark.parametrize("a_km,b_km,c32", [(1, 1, 0), (1, 0, 0), (0, 0, 1), (1, 1, 1),
                                           (0, 1, 0), (0, 0, 0), (1, 0, 1), (0, 1, 1)])
@pytest.mark.parametrize("M,N,K", [(256, 256, 64), (300, 264, 136), (8, 520, 1000),
                                   (513, 8, 72), (1, 16, 8)])
def test_gemm_layouts_ragged(qf, a_km, b_km, c32, M, N, K):
    if (not a_km and M % 8) or (not b_km and N % 8):
        pytest.skip("mn-major operands need a multiple of 8 along the contiguous axis")
    rng = np.random.default_rng(M * 7 + N * 3 + K)
    A = _rand_bf16(rng, (M, K))              # logical A(m, k)
    B = _rand_bf16(rng, (N, K))              # logical B(n, k)
    As = A if a_km else np.ascontiguousarray(A.T)
    Bs = B if b_km else np.ascontiguousarray(B.T)
    C = torch.empty(M, N, dtype=torch.float32 if c32 else torch.int16, device="cuda")
    qf.gemm_bf16(M, N, K, to_dev(As), As.shape[1], a_km, to_dev(Bs), Bs.shape[1], b_km, C, N, c32)
    torch.cuda.synchronize()
    got = from_dev(C).astype(np.float64) if c32 else bf16_to_f64(from_dev(C))
    assert_close(got, oracle.linear_fwd(A, B), f"gemm a_km={a_km} b_km={b_km}")


@pytest.mark.parametrize("M,N,K", [(264, 2056, 200), (512, 64, 136), (1032, 2304, 4104),
                                   (8, 2048, 8), (64, 0, 72), (2048, 4096, 1024),
                                   (520, 3840, 2056)])
def test_gemm_with_transposed_a_output(qf, M, N, K):
    """qf_gemm_bf16_at: C bit-identical to qf_gemm_bf16 and at = A^T exactly, padding columns
    untouched (8, 9 or 15 tile columns: A^T from the GEMM's staged tiles, up to two pieces per
    tile and stage; 16: at most one; ragged last stage and rows; 1 tile column or N = 0: from
    the transpose kernel)."""
    rng = np.random.default_rng(M * 5 + N + K)
    A, B = _rand_bf16(rng, (M, K)), _rand_bf16(rng, (N, K))
    Ad, Bd = to_dev(A), to_dev(B)
    ldat = M + 12
    at = torch.full((K, ldat), 0x1234, dtype=torch.int16, device="cuda")
    C = empty_bf16((M, N))
    qf.gemm_bf16_at(M, N, K, Ad, K, Bd, K, C, N, at, ldat)
    C2 = empty_bf16((M, N))
    qf.gemm_bf16(M, N, K, Ad, K, 1, Bd, K, 1, C2, N, 0)
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(C).view(np.uint16), from_dev(C2).view(np.uint16))
    a_t = from_dev(at).view(np.uint16)
    assert np.array_equal(a_t[:, :M], A.T)
    assert np.all(a_t[:, M:] == 0x1234)


def test_gemm_zero_depth_writes_zeros(qf):
    C = torch.full((64, 64), 7.0, dtype=torch.float32, device="cuda")
    A = torch.zeros(64, 8, dtype=torch.int16, device="cuda")
    qf.gemm_bf16(64, 64, 0, A, 8, 1, A, 8, 1, C, 64, 1)
    torch.cuda.synchronize()
    assert float(C.abs().max().item()) == 0.0


def test_gemm_strided_output_leaves_padding(qf):
    rng = np.random.default_rng(11)
    M, N, K, ldc = 200, 136, 96, 152
    A, B = _rand_bf16(rng, (M, K)), _rand_bf16(rng, (N, K))
    C = torch.full((M, ldc), -3.0, dtype=torch.float32, device="cuda")
    qf.gemm_bf16(M, N, K, to_dev(A), K, 1, to_dev(B), K, 1, C, ldc, 1)
    torch.cuda.synchronize()
    c = from_dev(C)
    assert np.all(c[:, N:] == -3.0)
    assert_close(c[:, :N], oracle.linear_fwd(A, B), "strided C")


# --------------------------------------------------------------------------- linear layer
def _layer(qf, w, wfmt, afmt, flags=0, w_amax=None, a_amax=None, reuse=False):
    M, N, K = w["X"].shape[0], w["W"].shape[0], w["W"].shape[1]
    X, W, dY = to_dev(w["X"]), to_dev(w["W"]), to_dev(w["dY"])
    # reuse: the workspace is kept from the forward to the backward (both calls carry the flag)
    d = qf.qlinear_desc(M, N, K, wfmt, afmt, w_amax=w_amax, a_amax=a_amax,
                        flags=qf.FLAG_REUSE_WS if reuse else 0)
    ws = qf.workspace(d)
    Y, dX = empty_bf16((M, N)), empty_bf16((M, K))
    dW = torch.empty(N, K, dtype=torch.float32, device="cuda")
    qf.qlinear_fwd(d, X, W, Y, ws)
    qf.qlinear_bwd_ste(d, dY, X, W, dX, dW, ws)
    torch.cuda.synchronize()
    return from_dev(Y), from_dev(dX), from_dev(dW)


def test_single_linear_nvfp4_full(qf):
    w = workloads.single_linear(seed=0)
    Y, dX, dW = _layer(qf, w, "nvfp4", "none")
    what = oracle.nvfp4(w["W"])["xhat"]
    assert_close(bf16_to_f64(Y), oracle.linear_fwd(w["X"], what), "Y")
    assert_close(bf16_to_f64(dX), oracle.linear_dx(w["dY"], what), "dX")
    assert_close(dW.astype(np.float64), oracle.linear_dw(w["dY"], w["X"]), "dW")
    # saving the quantized operands for the backward gives the same bits as re-quantizing
    Y2, dX2, dW2 = _layer(qf, w, "nvfp4", "none", reuse=True)
    assert np.array_equal(Y, Y2) and np.array_equal(dX, dX2) and np.array_equal(dW, dW2)


@pytest.mark.parametrize("wfmt,afmt", [("mxfp4", "mxfp4"), ("q4k", "none"), ("none", "none"),
                                       ("nvfp4", "mxfp4"), ("mxfp4", "none")])
def test_linear_formats_small(qf, wfmt, afmt):
    rng = np.random.default_rng(5)
    M, N, K = 384, 264, 512
    w = {"X": _rand_bf16(rng, (M, K)), "W": _rand_bf16(rng, (N, K), 0.02),
         "dY": _rand_bf16(rng, (M, N))}
    Y, dX, dW = _layer(qf, w, wfmt, afmt)
    what = oracle.fakequant(w["W"], wfmt)
    ahat = oracle.fakequant(w["X"], afmt)
    assert_close(bf16_to_f64(Y), oracle.linear_fwd(ahat, what), "Y")
    assert_close(bf16_to_f64(dX), oracle.linear_dx(w["dY"], what), "dX")
    assert_close(dW.astype(np.float64), oracle.linear_dw(w["dY"], ahat), "dW")


def test_nvfp4_activations_with_running_amax(qf):
    rng = np.random.default_rng(6)
    M, N, K = 256, 256, 256
    w = {"X": _rand_bf16(rng, (M, K)), "W": _rand_bf16(rng, (N, K), 0.02),
         "dY": _rand_bf16(rng, (M, N))}
    run = float(np.float32(1.25 * oracle.amax(w["X"])))      # running amax above this batch
    a_amax = torch.tensor([run], dtype=torch.float32, device="cuda")
    Y, dX, dW = _layer(qf, w, "nvfp4", "nvfp4", a_amax=a_amax)
    what = oracle.nvfp4(w["W"])["xhat"]
    ahat = oracle.nvfp4(w["X"], amax_in=run)["xhat"]
    assert_close(bf16_to_f64(Y), oracle.linear_fwd(ahat, what), "Y")
    assert_close(dW.astype(np.float64), oracle.linear_dw(w["dY"], ahat), "dW")


def test_tied_qkv_scale(qf):
    # Engine-specific scale sharing: one tensor scale for the fused Q, K, V weights, built
    # with qf_amax(accumulate) over the members and passed as w_amax.
    rng = np.random.default_rng(7)
    K = 512
    parts = [_rand_bf16(rng, (n, K), s) for n, s in ((512, 0.02), (128, 0.05), (128, 0.01))]
    Wqkv = np.concatenate(parts)
    g = torch.zeros(1, dtype=torch.float32, device="cuda")
    for i, p in enumerate(parts):
        qf.amax(to_dev(p), g, accumulate=i > 0)
    torch.cuda.synchronize()
    gval = float(g.item())
    assert gval == max(oracle.amax(p) for p in parts)
    w = {"X": _rand_bf16(rng, (256, K)), "W": Wqkv, "dY": _rand_bf16(rng, (256, Wqkv.shape[0]))}
    Y, dX, dW = _layer(qf, w, "nvfp4", "none", w_amax=g)
    what = oracle.nvfp4(Wqkv, amax_in=gval)["xhat"]
    assert_close(bf16_to_f64(Y), oracle.linear_fwd(w["X"], what), "Y")


def test_activation_gradient_decomposition_on_gpu(qf):
    # dW(W4A4) - dW(W4A16) = dO eps_A^T (Eq. activation-gradient-error), to FP32 accuracy
    rng = np.random.default_rng(8)
    M, N, K = 512, 256, 256
    w = {"X": _rand_bf16(rng, (M, K)), "W": _rand_bf16(rng, (N, K), 0.02),
         "dY": _rand_bf16(rng, (M, N))}
    _, _, dW44 = _layer(qf, w, "mxfp4", "mxfp4")
    _, _, dW416 = _layer(qf, w, "mxfp4", "none")
    eps = bf16_to_f64(oracle.mxfp4(w["X"])["xhat"]) - bf16_to_f64(w["X"])
    want = bf16_to_f64(w["dY"]).T @ eps
    scale = np.abs(bf16_to_f64(w["dY"])).T @ np.abs(bf16_to_f64(w["X"]))
    assert np.all(np.abs((dW44.astype(np.float64) - dW416) - want) <= 1e-5 * scale + 1e-6)


def test_mlp_up_mxfp4_full_size_sampled(qf):
    """The benchmarked workload (8192 x 14336 x 4096, MXFP4 weights and activations) in the
    launch configuration the benchmark times, checked on sampled entries + whole rows."""
    w = workloads.mlp_up(seed=0)
    M, N, K = w["M"], w["N"], w["K"]
    Y, dX, dW = _layer(qf, w, "mxfp4", "mxfp4")
    xq = oracle.mxfp4(w["X"])["xhat"]
    wq = oracle.mxfp4(w["W"])["xhat"]
    rng = np.random.default_rng(9)
    n = 1 << 14
    # Y[i, j] = sum_k xq[i, k] wq[j, k]
    i, j = rng.integers(0, M, n), rng.integers(0, N, n)
    assert_close(bf16_to_f64(Y[i, j]), oracle.dot_rows(xq, i, wq, j), "Y sampled")
    r = rng.integers(0, M, 2)
    assert_close(bf16_to_f64(Y[r]), oracle.linear_fwd(xq[r], wq), "Y rows")
    # dX[i, k] = sum_n dY[i, n] wq[n, k]
    wqT = np.ascontiguousarray(wq.T)
    i, k = rng.integers(0, M, n), rng.integers(0, K, n)
    assert_close(bf16_to_f64(dX[i, k]), oracle.dot_rows(w["dY"], i, wqT, k), "dX sampled")
    # dW[j, k] = sum_m dY[m, j] xq[m, k]
    dYT = np.ascontiguousarray(w["dY"].T)
    xqT = np.ascontiguousarray(xq.T)
    j, k = rng.integers(0, N, n // 4), rng.integers(0, K, n // 4)
    assert_close(dW[j, k].astype(np.float64), oracle.dot_rows(dYT, j, xqT, k), "dW sampled")
    # two whole rows of each gradient
    r = rng.integers(0, M, 2)
    assert_close(bf16_to_f64(dX[r]), oracle.linear_dx(w["dY"][r], wq), "dX rows")
    j = rng.integers(0, N, 2)
    assert_close(dW[j].astype(np.float64), oracle.linear_fwd(dYT[j], xqT), "dW rows")


def _nvfp4_xhat_threaded(W, g):
    """The oracle's NVFP4 x_hat of W with the tensor amax g, over row chunks in threads (each
    chunk one oracle call; the block scales depend on g and the block only)."""
    from concurrent.futures import ThreadPoolExecutor
    chunks = range(0, W.shape[0], 512)
    with ThreadPoolExecutor(max_workers=16) as ex:
        parts = ex.map(lambda r0: oracle.nvfp4(np.ascontiguousarray(W[r0:r0 + 512]), amax_in=g)["xhat"],
                       chunks)
        return np.concatenate(list(parts))


@pytest.mark.parametrize("name,members", [("qkv", (4096, 1024, 1024)), ("o", (4096,)),
                                          ("gate_up", (12288, 12288))])
def test_dense_layer_32k_tokens_sampled(qf, name, members):
    """The 9B-class layer's QKV, O and gate/up projections at 32768 tokens (NVFP4 weights,
    heavy-tailed activations) in the launch configuration the benchmark times.  A fused
    projection's tensor scale is tied over its members (Sec. 3.2.3 "Engine-specific scale
    sharing"): g is built with qf_amax over the member weights (overwrite, then accumulate) and
    handed to the layer, which must give what the oracle gives for the same g.  Sampled
    entries of Y, dX and dW plus two whole rows of each."""
    T, K = 32768, 4096
    N = sum(members)
    rng = np.random.default_rng(40 + N)
    tau = np.abs(rng.standard_t(3.0, size=K)).astype(np.float32)
    w = {"X": workloads.normal_bf16(rng, (T, K), 1.0, col_scale=tau),
         "W": workloads.normal_bf16(rng, (N, K), 0.02),
         "dY": workloads.normal_bf16(rng, (T, N), 1.0)}
    Wd = to_dev(w["W"])
    g = torch.zeros(1, dtype=torch.float32, device="cuda")
    r0 = 0
    for i, m in enumerate(members):
        qf.amax(Wd[r0:r0 + m], g, accumulate=i > 0)
        r0 += m
    torch.cuda.synchronize()
    g_ref = max(oracle.amax(np.ascontiguousarray(w["W"][a:a + m]))
                for a, m in zip(np.cumsum((0,) + members[:-1]), members))
    assert float(g.item()) == g_ref == oracle.amax(w["W"])
    Y, dX, dW = _layer(qf, w, "nvfp4", "none", w_amax=g)
    del Wd
    wq = _nvfp4_xhat_threaded(w["W"], g_ref)
    n = 1 << 12

    def sampled(a, ai, b, bi):
        return np.concatenate([oracle.dot_rows(a, ai[c:c + 256], b, bi[c:c + 256])
                               for c in range(0, len(ai), 256)])

    i, j = rng.integers(0, T, n), rng.integers(0, N, n)
    assert_close(bf16_to_f64(Y[i, j]), sampled(w["X"], i, wq, j), f"{name} Y sampled")
    r = rng.integers(0, T, 2)
    assert_close(bf16_to_f64(Y[r]), oracle.linear_fwd(w["X"][r], wq), f"{name} Y rows")
    wqT = np.ascontiguousarray(wq.T)
    i, k = rng.integers(0, T, n), rng.integers(0, K, n)
    assert_close(bf16_to_f64(dX[i, k]), sampled(w["dY"], i, wqT, k), f"{name} dX sampled")
    assert_close(bf16_to_f64(dX[r]), oracle.linear_dx(w["dY"][r], wq), f"{name} dX rows")
    del wqT, Y, dX
    dYT = np.ascontiguousarray(w["dY"].T)
    xT = np.ascontiguousarray(w["X"].T)
    j, k = rng.integers(0, N, n), rng.integers(0, K, n)
    assert_close(dW[j, k].astype(np.float64), sampled(dYT, j, xT, k), f"{name} dW sampled")
    j = rng.integers(0, N, 2)
    assert_close(dW[j].astype(np.float64), oracle.linear_fwd(dYT[j], xT), f"{name} dW rows")


def test_q4k_export_weight_forward_full_size_sampled(qf):
    """The Q4_K export weight (14336 x 4096, per-row log-normal scales) and its forward GEMM at
    X 4096 x 4096, in the launch configuration the benchmark times, on sampled entries + rows."""
    w = workloads.q4k_weight(seed=0)
    M, N, K = w["M"], w["N"], w["K"]
    X, W = to_dev(w["X"]), to_dev(w["W"])
    d = qf.qlinear_desc(M, N, K, "q4k", "none")
    ws = qf.workspace(d)
    Yd = empty_bf16((M, N))
    qf.qlinear_fwd(d, X, W, Yd, ws)
    torch.cuda.synchronize()
    Y = from_dev(Yd)
    wq = oracle.q4k(w["W"])["xhat"]
    rng = np.random.default_rng(25)
    i, j = rng.integers(0, M, 1 << 14), rng.integers(0, N, 1 << 14)
    assert_close(bf16_to_f64(Y[i, j]), oracle.dot_rows(w["X"], i, wq, j), "Y sampled")
    r = rng.integers(0, M, 2)
    assert_close(bf16_to_f64(Y[r]), oracle.linear_fwd(w["X"][r], wq), "Y rows")


def test_linear_determinism(qf):
    rng = np.random.default_rng(10)
    w = {"X": _rand_bf16(rng, (512, 1024)), "W": _rand_bf16(rng, (768, 1024), 0.02),
         "dY": _rand_bf16(rng, (512, 768))}
    a = _layer(qf, w, "nvfp4", "none")
    b = _layer(qf, w, "nvfp4", "none")
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("R,C,ldi", [(64, 256, 256), (8, 8, 8), (136, 520, 528), (8192, 72, 72)])
def test_transpose_exact(qf, R, C, ldi):
    rng = np.random.default_rng(R + C)
    x = rng.integers(0, 65536, size=(R, ldi), dtype=np.uint32).astype(np.uint16)
    xd = to_dev(x)[:, :C]
    out = torch.full((C, R + 8), 1234, dtype=torch.int16, device="cuda")[:, :R]
    qf.transpose_bf16(xd, out)
    torch.cuda.synchronize()
    got = from_dev(out.contiguous())
    np.testing.assert_array_equal(got, x[:, :C].T)


def test_layer_backward_with_m_not_multiple_of_8(qf):
    # M % 8 != 0 takes the kernel that reads the [M, *] operands directly (no transposes)
    rng = np.random.default_rng(12)
    M, N, K = 300, 136, 256
    w = {"X": _rand_bf16(rng, (M, K)), "W": _rand_bf16(rng, (N, K), 0.02),
         "dY": _rand_bf16(rng, (M, N))}
    Y, dX, dW = _layer(qf, w, "mxfp4", "mxfp4")
    what = oracle.mxfp4(w["W"])["xhat"]
    ahat = oracle.mxfp4(w["X"])["xhat"]
    assert_close(bf16_to_f64(Y), oracle.linear_fwd(ahat, what), "Y")
    assert_close(bf16_to_f64(dX), oracle.linear_dx(w["dY"], what), "dX")
    assert_close(dW.astype(np.float64), oracle.linear_dw(w["dY"], ahat), "dW")


@pytest.mark.parametrize("wfmt,afmt,reuse", [("mxfp4", "mxfp4", False), ("nvfp4", "none", False),
                                             ("mxfp4", "mxfp4", True)])
def test_layer_token_count_multiple_of_16384(qf, wfmt, afmt, reuse):
    """16384 tokens: the dW operands dY^T and A_hat^T sit in the workspace with a row stride of
    16384 + 128 elements (byte strides that are multiples of 32 KB get padded)."""
    rng = np.random.default_rng(21)
    M, N, K = 16384, 264, 512
    w = {"X": _rand_bf16(rng, (M, K)), "W": _rand_bf16(rng, (N, K), 0.02),
         "dY": _rand_bf16(rng, (M, N))}
    Y, dX, dW = _layer(qf, w, wfmt, afmt, reuse=reuse)
    what = oracle.fakequant(w["W"], wfmt)
    ahat = oracle.fakequant(w["X"], afmt)
    assert_close(bf16_to_f64(Y), oracle.linear_fwd(ahat, what), "Y")
    assert_close(bf16_to_f64(dX), oracle.linear_dx(w["dY"], what), "dX")
    assert_close(dW.astype(np.float64), oracle.linear_dw(w["dY"], ahat), "dW")


@pytest.mark.parametrize("M,N,K", [(512, 264, 768), (1032, 1000, 544), (16384, 136, 1280),
                                   (8, 72, 32), (2048, 64, 2304)])
def test_dw_alone_equals_dw_with_dx(qf, M, N, K):
    """dY^T for dW comes from the dX GEMM (which writes it from the dY tiles it stages) when
    both gradients are asked for, from the transpose kernel when dW alone is: bit-identical
    dW (tile columns that own 0 to several stages, a ragged last stage, padded strides)."""
    rng = np.random.default_rng(M + N + K)
    w = {"X": _rand_bf16(rng, (M, K)), "W": _rand_bf16(rng, (N, K), 0.02),
         "dY": _rand_bf16(rng, (M, N))}
    X, W, dY = to_dev(w["X"]), to_dev(w["W"]), to_dev(w["dY"])
    d = qf.qlinear_desc(M, N, K, "mxfp4", "mxfp4")
    outs = []
    for want_dx in (True, False):
        ws = qf.workspace(d)
        dX = empty_bf16((M, K)) if want_dx else None
        dW = torch.full((N, K), 7.0, dtype=torch.float32, device="cuda")
        qf.qlinear_bwd_ste(d, dY, X, W, dX, dW, ws)
        torch.cuda.synchronize()
        outs.append(from_dev(dW))
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    ahat = oracle.mxfp4(w["X"])["xhat"]
    assert_close(outs[0].astype(np.float64), oracle.linear_dw(w["dY"], ahat), "dW")


def test_dense_down_projection_32k_tokens_sampled(qf):
    """The 9B-class layer's down projection at 32K tokens (32768 x 4096 x 12288, NVFP4 weights,
    bf16 activations with heavy-tailed column scales) in the launch configuration the benchmark
    times (row stride 32768 + 128 for the dW operands), checked on sampled entries."""
    rng = np.random.default_rng(22)
    M, N, K = 32768, 4096, 12288
    tau = np.abs(rng.standard_t(3.0, size=K)).astype(np.float32)
    w = {"X": workloads.normal_bf16(rng, (M, K), 1.0, col_scale=tau),
         "W": workloads.normal_bf16(rng, (N, K), 0.02),
         "dY": workloads.normal_bf16(rng, (M, N), 1.0)}
    Y, dX, dW = _layer(qf, w, "nvfp4", "none")
    wq = oracle.nvfp4(w["W"])["xhat"]
    n = 2048

    def sampled(a, ai, b, bi):                    # chunked: rows are up to 32768 long
        return np.concatenate([oracle.dot_rows(a, ai[c:c + 256], b, bi[c:c + 256])
                               for c in range(0, len(ai), 256)])

    i, j = rng.integers(0, M, n), rng.integers(0, N, n)
    assert_close(bf16_to_f64(Y[i, j]), sampled(w["X"], i, wq, j), "Y sampled")
    wqT = np.ascontiguousarray(wq.T)
    i, k = rng.integers(0, M, n), rng.integers(0, K, n)
    assert_close(bf16_to_f64(dX[i, k]), sampled(w["dY"], i, wqT, k), "dX sampled")
    del wqT, Y, dX
    dYT = np.ascontiguousarray(w["dY"].T)
    xT = np.ascontiguousarray(w["X"].T)
    j, k = rng.integers(0, N, n), rng.integers(0, K, n)
    assert_close(dW[j, k].astype(np.float64), sampled(dYT, j, xT, k), "dW sampled")


def test_nt_gemm_pipeline_depths(qf):
    # K from below one stage to many stages, with and without a partial last stage
    rng = np.random.default_rng(13)
    M, N = 264, 520
    A = _rand_bf16(rng, (M, 4096))
    B = _rand_bf16(rng, (N, 4096))
    for K in [8, 32, 40, 64, 96, 128, 160, 200, 512, 1016, 4096]:
        C = torch.empty(M, N, dtype=torch.float32, device="cuda")
        qf.gemm_bf16(M, N, K, to_dev(A), 4096, 1, to_dev(B), 4096, 1, C, N, 1)
        torch.cuda.synchronize()
        assert_close(from_dev(C).astype(np.float64),
                     oracle.linear_fwd(np.ascontiguousarray(A[:, :K]), np.ascontiguousarray(B[:, :K])),
                     f"K={K}")


@pytest.mark.parametrize("wfmt,afmt,M,K", [("nvfp4", "none", 392, 544), ("mxfp4", "mxfp4", 392, 544),
                                           ("q4k", "none", 264, 768), ("nvfp4", "nvfp4", 200, 512),
                                           ("mxfp4", "none", 8, 256)])
def test_transposing_quantizer_matches_saved_operands(qf, wfmt, afmt, M, K):
    """The backward quantizes W (and X) straight into the transposed NT operands; with
    QF_FLAG_REUSE_WS it takes W_hat^T from the workspace's packed W_hat and A_hat^T from the
    forward GEMM, which wrote it from its staged A tiles (M = 8: from the transpose kernel).
    Both routes feed the same GEMMs, so dX and dW must agree bit for bit (ragged tiles in every
    direction)."""
    rng = np.random.default_rng(12)
    N = 264
    w = {"X": _rand_bf16(rng, (M, K)), "W": _rand_bf16(rng, (N, K), 0.02),
         "dY": _rand_bf16(rng, (M, N))}
    a_amax = None
    if afmt == "nvfp4":
        a_amax = torch.tensor([float(np.float32(1.1 * oracle.amax(w["X"])))],
                              dtype=torch.float32, device="cuda")
    Y, dX, dW = _layer(qf, w, wfmt, afmt, a_amax=a_amax)
    Y2, dX2, dW2 = _layer(qf, w, wfmt, afmt, a_amax=a_amax, reuse=True)
    assert np.array_equal(Y, Y2)
    assert np.array_equal(dX.view(np.uint16), dX2.view(np.uint16))
    assert np.array_equal(dW.view(np.uint32), dW2.view(np.uint32))


@pytest.mark.parametrize("M,N,K,ldc", [(264, 1000, 136, 1004), (8, 2048, 1000, 2048),
                                       (2048, 12, 200, 16), (512, 1024, 128, 1024),
                                       (300, 264, 136, 264)])
def test_gemm_split_last_round(qf, M, N, K, ldc):
    """FP32 NT GEMM with a workspace: grids of 8 tiles (one per XCD, all in the last, partial
    round) run as two K-halves plus a fixed-order sum; ragged edges, K tails, a strided C, and
    one shape (4 tiles) that does not split."""
    rng = np.random.default_rng(M + N + K)
    A, B = _rand_bf16(rng, (M, K)), _rand_bf16(rng, (N, K))
    C = torch.full((M, ldc), -3.0, dtype=torch.float32, device="cuda")
    ws = qf.gemm_workspace(M, N, 1)
    qf.gemm_bf16(M, N, K, to_dev(A), K, 1, to_dev(B), K, 1, C, ldc, 1, ws=ws)
    torch.cuda.synchronize()
    c = from_dev(C)
    assert np.all(c[:, N:] == -3.0)
    want = oracle.linear_fwd(A, B)
    assert_close(c[:, :N].astype(np.float64), want, "split gemm")
    # the same call again gives the same bits
    C2 = torch.full((M, ldc), -3.0, dtype=torch.float32, device="cuda")
    qf.gemm_bf16(M, N, K, to_dev(A), K, 1, to_dev(B), K, 1, C2, ldc, 1, ws=ws)
    torch.cuda.synchronize()
    assert np.array_equal(c.view(np.uint32), from_dev(C2).view(np.uint32))
