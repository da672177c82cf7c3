"""GPU parity of the grouped (mixture-of-experts) layer: per-expert fake quantization and
grouped GEMMs over device-resident row offsets equal looping the dense layer per expert."""
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


def run_grouped(qf, offsets, X, W, dY, wfmt, afmt, reuse=False, saved=False):
    """Forward + backward; the backward re-quantizes W (default), reuses the forward's
    workspace (reuse) or dequantizes the forward's saved packed experts (saved)."""
    E, N, K = W.shape
    T = X.shape[0]
    d = qf.grouped_desc(E, T, N, K, wfmt, afmt)
    ws = qf.grouped_workspace(d)
    sv = qf.grouped_saved_buffer(d) if saved else None
    off = torch.from_numpy(offsets.astype(np.int64)).cuda()
    Xd, Wd, dYd = to_dev(X), to_dev(W.reshape(E * N, K)), to_dev(dY)
    Y, dX = empty_bf16((T, N)), empty_bf16((T, K))
    dW = torch.full((E, N, K), 7.0, dtype=torch.float32, device="cuda")
    qf.qlinear_grouped_fwd(d, off, Xd, Wd, Y, ws, saved=sv)
    if reuse:
        d = qf.grouped_desc(E, T, N, K, wfmt, afmt, flags=qf.FLAG_REUSE_WS)
    qf.qlinear_grouped_bwd_ste(d, off, dYd, Xd, Wd, dX, dW, ws, saved=sv)
    torch.cuda.synchronize()
    return from_dev(Y), from_dev(dX), from_dev(dW)


@pytest.mark.parametrize("wfmt,afmt", [("nvfp4", "none"), ("mxfp4", "mxfp4"), ("q4k", "none")])
def test_grouped_matches_per_expert_loop(qf, wfmt, afmt):
    rng = np.random.default_rng(0)
    E, N, K = 6, 264, 512
    counts = np.array([0, 300, 1, 513, 0, 77])          # empty, ragged, single-row experts
    offsets = np.concatenate([[0], np.cumsum(counts)])
    T = int(offsets[-1])
    X = workloads.normal_bf16(rng, (T, K))
    W = np.stack([workloads.normal_bf16(rng, (N, K), 0.02 * (e + 1)) for e in range(E)])
    dY = workloads.normal_bf16(rng, (T, N))
    Y, dX, dW = run_grouped(qf, offsets, X, W, dY, wfmt, afmt)
    ahat = oracle.fakequant(X, afmt)
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        what = oracle.fakequant(W[e], wfmt)              # one tensor scale per expert
        if r1 > r0:
            assert_close(bf16_to_f64(Y[r0:r1]), oracle.linear_fwd(ahat[r0:r1], what), f"Y e={e}")
            assert_close(bf16_to_f64(dX[r0:r1]), oracle.linear_dx(dY[r0:r1], what), f"dX e={e}")
            assert_close(dW[e].astype(np.float64), oracle.linear_dw(dY[r0:r1], ahat[r0:r1]),
                         f"dW e={e}")
        else:
            assert np.all(dW[e] == 0.0)


def test_grouped_dw_tile_grid_split_over_xcds(qf):
    """Per-expert dW grids of 5 x 3 tiles (ragged in both dimensions) are dealt to the 8 XCDs
    in shares of 1 or 2 tiles; every expert's gradient is complete, empty experts are zero."""
    rng = np.random.default_rng(7)
    E, N, K = 5, 1032, 544
    counts = np.array([0, 700, 65, 1, 2000])
    offsets = np.concatenate([[0], np.cumsum(counts)])
    T = int(offsets[-1])
    X = workloads.normal_bf16(rng, (T, K))
    W = np.stack([workloads.normal_bf16(rng, (N, K), 0.02) for _ in range(E)])
    dY = workloads.normal_bf16(rng, (T, N))
    Y, dX, dW = run_grouped(qf, offsets, X, W, dY, "nvfp4", "mxfp4")
    ahat = oracle.fakequant(X, "mxfp4")
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            assert_close(dW[e].astype(np.float64), oracle.linear_dw(dY[r0:r1], ahat[r0:r1]),
                         f"dW e={e}")
        else:
            assert np.all(dW[e] == 0.0)


@pytest.mark.parametrize("K", [2048, 4096])
def test_grouped_dw_alone_equals_dw_with_dx(qf, K):
    """With 8 or more tile columns in dX the grouped dX launch writes the padded dY^T for dW
    (zeros past each expert's last token, written by the tile holding its last rows; 8 tile
    columns: up to two pieces per tile and stage, 16: one); asked for alone, dW takes it from
    the grouped transposer: bit-identical dW, equal to the oracle, and dX equal to the oracle."""
    rng = np.random.default_rng(26)
    E, N = 5, 136
    counts = np.array([0, 300, 1, 513, 77])
    offsets = np.concatenate([[0], np.cumsum(counts)])
    T = int(offsets[-1])
    X = workloads.normal_bf16(rng, (T, K))
    W = np.stack([workloads.normal_bf16(rng, (N, K), 0.02 * (e + 1)) for e in range(E)])
    dY = workloads.normal_bf16(rng, (T, N))
    d = qf.grouped_desc(E, T, N, K, "nvfp4", "none")
    off = torch.from_numpy(offsets.astype(np.int64)).cuda()
    Xd, Wd, dYd = to_dev(X), to_dev(W.reshape(E * N, K)), to_dev(dY)
    outs = []
    dx_got = None
    for want_dx in (True, False):
        ws = qf.grouped_workspace(d)
        ws.fill_(0x5A)                              # stale workspace bytes must not leak in
        dX = empty_bf16((T, K)) if want_dx else None
        dW = torch.full((E, N, K), 7.0, dtype=torch.float32, device="cuda")
        qf.qlinear_grouped_bwd_ste(d, off, dYd, Xd, Wd, dX, dW, ws)
        torch.cuda.synchronize()
        outs.append(from_dev(dW))
        if want_dx:
            dx_got = bf16_to_f64(from_dev(dX))
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            assert_close(outs[0][e].astype(np.float64), oracle.linear_dw(dY[r0:r1], X[r0:r1]),
                         f"dW e={e}")
            what = oracle.fakequant(W[e], "nvfp4")       # one tensor scale per expert
            assert_close(dx_got[r0:r1], oracle.linear_dx(dY[r0:r1], what), f"dX e={e}")
        else:
            assert np.all(outs[0][e] == 0.0)


def test_grouped_padded_token_count_multiple_of_16384(qf):
    """Two experts whose 64-aligned padded token count is exactly 16384: the dW operands sit
    in the workspace with a row stride of 16384 + 128 elements."""
    rng = np.random.default_rng(23)
    E, N, K = 2, 136, 256
    counts = np.array([8000, 8195])                # (16195 + 63 * 2 + 63) // 64 * 64 == 16384
    offsets = np.concatenate([[0], np.cumsum(counts)])
    T = int(offsets[-1])
    X = workloads.normal_bf16(rng, (T, K))
    W = np.stack([workloads.normal_bf16(rng, (N, K), 0.02 * (e + 1)) for e in range(E)])
    dY = workloads.normal_bf16(rng, (T, N))
    Y, dX, dW = run_grouped(qf, offsets, X, W, dY, "mxfp4", "mxfp4")
    ahat = oracle.fakequant(X, "mxfp4")
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        what = oracle.fakequant(W[e], "mxfp4")
        assert_close(bf16_to_f64(Y[r0:r1]), oracle.linear_fwd(ahat[r0:r1], what), f"Y e={e}")
        assert_close(bf16_to_f64(dX[r0:r1]), oracle.linear_dx(dY[r0:r1], what), f"dX e={e}")
        assert_close(dW[e].astype(np.float64), oracle.linear_dw(dY[r0:r1], ahat[r0:r1]),
                     f"dW e={e}")


def test_grouped_zipf_routing_sampled(qf):
    """128 experts, top-8 Zipf(1.1) routing (reduced token count and width), sampled."""
    tok, offsets = workloads.moe_routing(seed=0, tokens=2048, experts=128, topk=8)
    rng = np.random.default_rng(1)
    E, N, K = 128, 384, 256
    T = int(offsets[-1])
    Xtok = workloads.normal_bf16(rng, (2048, K))
    X = Xtok[tok]
    W = workloads.normal_bf16(rng, (E * N, K), 0.02).reshape(E, N, K)
    dY = workloads.normal_bf16(rng, (T, N))
    Y, dX, dW = run_grouped(qf, offsets, X, W, dY, "nvfp4", "none")
    for e in [0, 1, 5, 64, 127]:
        r0, r1 = offsets[e], offsets[e + 1]
        what = oracle.nvfp4(W[e])["xhat"]
        assert_close(bf16_to_f64(Y[r0:r1]), oracle.linear_fwd(X[r0:r1], what), f"Y e={e}")
        assert_close(bf16_to_f64(dX[r0:r1]), oracle.linear_dx(dY[r0:r1], what), f"dX e={e}")
        assert_close(dW[e].astype(np.float64), oracle.linear_dw(dY[r0:r1], X[r0:r1]), f"dW e={e}")


@pytest.mark.parametrize("N,K", [(3072, 1536), (3072, 3072)])
def test_moe_projection_full_size_sampled(qf, N, K):
    """The MoE layer's projections at full size (128 experts, Zipf(1.1) top-8 routing of
    32768 tokens = 262144 rows; down 1536 -> 3072 and gate/up 3072 -> 3072, whose dX launch
    also writes the padded dY^T; NVFP4 weights) in the launch configuration the benchmark
    times; entries sampled in the largest, smallest and three other experts."""
    _, offsets = workloads.moe_routing(seed=0, tokens=32768, experts=128, topk=8)
    E = 128
    T = int(offsets[-1])
    rng = np.random.default_rng(24)
    X = workloads.normal_bf16(rng, (T, K))
    W = workloads.normal_bf16(rng, (E * N, K), 0.02).reshape(E, N, K)
    dY = workloads.normal_bf16(rng, (T, N))
    d = qf.grouped_desc(E, T, N, K, "nvfp4", "none")
    ws = qf.grouped_workspace(d)
    sv = qf.grouped_saved_buffer(d)                 # as the benchmark: backward from saved
    off = torch.from_numpy(offsets.astype(np.int64)).cuda()
    Xd, Wd, dYd = to_dev(X), to_dev(W.reshape(E * N, K)), to_dev(dY)
    Yd, dXd = empty_bf16((T, N)), empty_bf16((T, K))
    dWd = torch.empty((E, N, K), dtype=torch.float32, device="cuda")
    qf.qlinear_grouped_fwd(d, off, Xd, Wd, Yd, ws, saved=sv)
    qf.qlinear_grouped_bwd_ste(d, off, dYd, Xd, Wd, dXd, dWd, ws, saved=sv)
    torch.cuda.synchronize()
    Y, dX = from_dev(Yd), from_dev(dXd)
    cnt = np.diff(offsets)
    experts = [int(np.argmax(cnt)), int(np.argmin(cnt))] + [int(e) for e in rng.choice(E, 3)]
    n = 1024
    for e in experts:
        r0, r1 = int(offsets[e]), int(offsets[e + 1])
        what = oracle.nvfp4(W[e])["xhat"]
        i, j, k = rng.integers(r0, r1, n), rng.integers(0, N, n), rng.integers(0, K, n)
        assert_close(bf16_to_f64(Y[i, j]), oracle.dot_rows(X, i, what, j), f"Y e={e}")
        assert_close(bf16_to_f64(dX[i, k]), oracle.dot_rows(dY, i, np.ascontiguousarray(what.T), k),
                     f"dX e={e}")
        dW = from_dev(dWd[e])
        j, k = rng.integers(0, N, n), rng.integers(0, K, n)
        dYT = np.ascontiguousarray(dY[r0:r1].T)
        XT = np.ascontiguousarray(X[r0:r1].T)
        assert_close(dW[j, k].astype(np.float64), oracle.dot_rows(dYT, j, XT, k), f"dW e={e}")


@pytest.mark.parametrize("wfmt", ["nvfp4", "mxfp4", "q4k"])
def test_grouped_transposing_quantizer_matches_saved_operands(qf, wfmt):
    """Expert W_hat^T straight from the transposing quantizer (per-expert NVFP4 scales) equals
    transposing the forward's saved W_hat: bit-identical dX."""
    rng = np.random.default_rng(13)
    E, N, K = 4, 136, 768
    counts = np.array([70, 0, 258, 9])
    offsets = np.concatenate([[0], np.cumsum(counts)])
    T = int(offsets[-1])
    X = workloads.normal_bf16(rng, (T, K))
    W = np.stack([workloads.normal_bf16(rng, (N, K), 0.02 * (e + 1)) for e in range(E)])
    dY = workloads.normal_bf16(rng, (T, N))
    _, dX, dW = run_grouped(qf, offsets, X, W, dY, wfmt, "none")
    _, dX2, dW2 = run_grouped(qf, offsets, X, W, dY, wfmt, "none", reuse=True)
    assert np.array_equal(dX.view(np.uint16), dX2.view(np.uint16))
    assert np.array_equal(dW.view(np.uint32), dW2.view(np.uint32))


@pytest.mark.parametrize("wfmt,afmt", [("nvfp4", "none"), ("mxfp4", "mxfp4"), ("q4k", "none")])
def test_grouped_saved_experts_and_backward_from_them(qf, wfmt, afmt):
    """The grouped forward's saved operand holds every expert's packed W_hat (NVFP4: codes, E4M3
    scales and the expert's own S; MXFP4; Q4_K blocks) bit for bit as the oracle packs it, and
    the backward that dequantizes it gives the same dX and dW bits as the backward that
    re-quantizes W and the one that reuses the workspace."""
    rng = np.random.default_rng(29)
    E, N, K = 5, 264, 768
    counts = np.array([70, 0, 258, 9, 300])
    offsets = np.concatenate([[0], np.cumsum(counts)])
    T = int(offsets[-1])
    X = workloads.normal_bf16(rng, (T, K))
    W = np.stack([workloads.normal_bf16(rng, (N, K), 0.02 * (e + 1)) for e in range(E)])
    dY = workloads.normal_bf16(rng, (T, N))
    d = qf.grouped_desc(E, T, N, K, wfmt, afmt)
    sv = torch.full((qf.grouped_saved_size(d),), 0xA5, dtype=torch.uint8, device="cuda")
    Y = empty_bf16((T, N))
    qf.qlinear_grouped_fwd(d, torch.from_numpy(offsets.astype(np.int64)).cuda(), to_dev(X),
                           to_dev(W.reshape(E * N, K)), Y, qf.grouped_workspace(d), saved=sv)
    torch.cuda.synchronize()
    buf = from_dev(sv)

    def up(v):
        return (v + 255) // 256 * 256
    o = 0
    if wfmt == "nvfp4":
        S = buf[:4 * E].view(np.float32)
        o = up(4 * E)
    refs = [{"nvfp4": oracle.nvfp4, "mxfp4": oracle.mxfp4, "q4k": oracle.q4k}[wfmt](W[e])
            for e in range(E)]
    if wfmt == "q4k":
        blk = buf[o:o + E * N * (K // 256) * 144].reshape(E, N, K // 256, 144)
        for e in range(E):
            np.testing.assert_array_equal(blk[e], refs[e]["packed"], err_msg=f"blocks e={e}")
    else:
        B = 16 if wfmt == "nvfp4" else 32
        codes = buf[o:o + E * N * K // 2].reshape(E, N, K // 2)
        o += up(E * N * K // 2)
        scales = buf[o:o + E * N * K // B].reshape(E, N, K // B)
        assert o + up(E * N * K // B) == qf.grouped_saved_size(d)
        for e in range(E):
            np.testing.assert_array_equal(codes[e], refs[e]["codes"], err_msg=f"codes e={e}")
            np.testing.assert_array_equal(scales[e], refs[e]["scales"], err_msg=f"scales e={e}")
            if wfmt == "nvfp4":
                assert S[e] == refs[e]["S"], e
    outs = [run_grouped(qf, offsets, X, W, dY, wfmt, afmt, saved=True),
            run_grouped(qf, offsets, X, W, dY, wfmt, afmt),
            run_grouped(qf, offsets, X, W, dY, wfmt, afmt, reuse=True)]
    for name, (_, dX, dW) in zip(("requantize", "reuse"), outs[1:]):
        assert np.array_equal(outs[0][1].view(np.uint16), dX.view(np.uint16)), f"dX vs {name}"
        assert np.array_equal(outs[0][2].view(np.uint32), dW.view(np.uint32)), f"dW vs {name}"
    ahat = oracle.fakequant(X, afmt)
    _, dX, dW = outs[0]
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            assert_close(bf16_to_f64(dX[r0:r1]), oracle.linear_dx(dY[r0:r1], refs[e]["xhat"]),
                         f"dX e={e}")
            assert_close(dW[e].astype(np.float64), oracle.linear_dw(dY[r0:r1], ahat[r0:r1]),
                         f"dW e={e}")
