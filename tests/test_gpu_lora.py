"""GPU parity of the LoRA-QAD path (Sec. 3.3, Eqs. qad-lora, export-lora) against the oracle.

* The merged quantizer (rank-r update fused into the quantizer's tile load): x_hat, codes,
  scales, Q4_K blocks, the merged amax and the NVFP4 decode scale are compared bit for bit
  with oracle.lora_quant (the merge is defined in binary32 with one fused multiply-add per
  rank term, so both sides take every quantization decision on the same bits).
* The layer (forward Y, straight-through dX, and the factor gradients dA, dB): FP32
  accumulation against the FP64 oracle on the same quantized operands, per entry
  |y - r| / max(|r|, 1e-3 rms(r)) with max <= 2e-2 and mean <= 2e-3.
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


def _factors(seed, N, K, r, scale=None):
    d = workloads.lora_factors(seed, N, K, r)
    if scale is not None:
        d["scale"] = scale
    return d


def _dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


# ------------------------------------------------------------------------- merged quantizer
QUANT_CASES = [  # fmt, N, K, r, scale
    ("mxfp4", 200, 768, 16, 2.0),     # ragged rows, three column tiles
    ("mxfp4", 64, 96, 1, 1.0),        # rank 1, ragged column tile
    ("nvfp4", 136, 560, 40, 0.5),     # rank not a multiple of the 16-term pass
    ("nvfp4", 8, 48, 3, 1.0),         # one ragged tile
    ("q4k", 72, 512, 16, 2.0),
    ("q4k", 130, 256, 33, 1.25),
    ("none", 104, 264, 7, 3.0),       # bf16 LoRA: the merged weight itself
]


@pytest.mark.parametrize("fmt,N,K,r,scale", QUANT_CASES)
def test_merged_quantizer_bit_exact(qf, fmt, N, K, r, scale):
    rng = np.random.default_rng(N + K + r)
    W = workloads.normal_bf16(rng, (N, K), 0.02)
    W[1, :8] = [0x8000, 0, 0x8000, 0, 0x0001, 0x8001, 0x3F80, 0xBF80]   # signed zeros, subnormals
    f = _factors(r, N, K, r, scale)
    f["B"][1] = 0.0                                    # row 1: no update (-0 merges to +0)
    A, B = _dev_f32(f["A"]), _dev_f32(f["B"])
    lo = qf.lora(A, B, f["scale"])
    Wd = to_dev(W)
    xhat = empty_bf16((N, K))
    outs = {}
    if fmt in ("nvfp4", "mxfp4"):
        outs["codes"] = torch.empty(N, K // 2, dtype=torch.uint8, device="cuda")
        outs["scales"] = torch.empty(N, K // (16 if fmt == "nvfp4" else 32), dtype=torch.uint8,
                                     device="cuda")
    if fmt == "q4k":
        outs["packed"] = torch.empty(N, K // 256, 144, dtype=torch.uint8, device="cuda")
    amax = torch.empty(1, dtype=torch.float32, device="cuda")
    s_out = torch.empty(1, dtype=torch.float32, device="cuda")
    nv = fmt == "nvfp4"
    qf.lora_fakequant(Wd, lo, fmt, amax=amax if nv else None, s_out=s_out if nv else None,
                      xhat=xhat, **outs)
    torch.cuda.synchronize()
    if fmt == "none":
        assert np.array_equal(from_dev(xhat), oracle.lora_merge(W, f["B"], f["A"], f["scale"]))
        return
    ref = oracle.lora_quant(W, f["B"], f["A"], f["scale"], fmt)
    assert np.array_equal(from_dev(xhat), ref["xhat"])
    for k, v in outs.items():
        assert np.array_equal(from_dev(v), ref[k]), k
    if nv:
        assert from_dev(amax)[0] == np.float32(ref["amax"])
        assert from_dev(s_out)[0] == np.float32(ref["S"])


@pytest.mark.parametrize("fmt,N,K,r", [("mxfp4", 200, 768, 16), ("nvfp4", 136, 560, 40),
                                       ("q4k", 72, 512, 5), ("none", 8, 64, 2)])
def test_merged_quantizer_transposed_bit_exact(qf, fmt, N, K, r):
    rng = np.random.default_rng(3 * N + K)
    W = workloads.normal_bf16(rng, (N, K), 0.02)
    f = _factors(r + 1, N, K, r)
    lo = qf.lora(_dev_f32(f["A"]), _dev_f32(f["B"]), f["scale"])
    m = oracle.lora_merge(W, f["B"], f["A"], f["scale"])
    g = None
    if fmt == "nvfp4":
        g = torch.tensor([oracle.amax(m)], dtype=torch.float32, device="cuda")
    ldo = N + 16
    out = torch.full((K, ldo), 0x1234, dtype=torch.int16, device="cuda")
    qf.lora_fakequant_transposed(to_dev(W), lo, fmt, out[:, :N], amax=g)
    torch.cuda.synchronize()
    got = from_dev(out)
    ref = m if fmt == "none" else oracle.fakequant(m, fmt)
    assert np.array_equal(got[:, :N], ref.T)
    assert np.all(got[:, N:] == 0x1234)


def test_merged_amax_tied_group(qf):
    # a tied group (Sec. 3.2.3 scale sharing) of two adapted members: running max of their
    # merged weights
    rng = np.random.default_rng(12)
    Ws = [workloads.normal_bf16(rng, (96, 256), s) for s in (0.02, 0.05)]
    fs = [_factors(20 + i, 96, 256, 8) for i in range(2)]
    amax = torch.full((1,), 123.0, dtype=torch.float32, device="cuda")
    keep = []
    for i, (W, f) in enumerate(zip(Ws, fs)):
        A, B = _dev_f32(f["A"]), _dev_f32(f["B"])
        keep += [A, B]
        qf.lora_amax(to_dev(W), qf.lora(A, B, f["scale"]), amax, accumulate=i > 0)
    torch.cuda.synchronize()
    want = max(oracle.amax(oracle.lora_merge(W, f["B"], f["A"], f["scale"]))
               for W, f in zip(Ws, fs))
    assert from_dev(amax)[0] == np.float32(want)


# ------------------------------------------------------------------------------- the layer
def _lora_layer(qf, X, W, dY, f, wfmt, afmt, reuse=False, a_amax=None, want=("dX", "dA", "dB")):
    M, K = X.shape
    N = W.shape[0]
    A, B = _dev_f32(f["A"]), _dev_f32(f["B"])
    lo = qf.lora(A, B, f["scale"])
    d = qf.qlinear_desc(M, N, K, wfmt, afmt, a_amax=a_amax)
    ws = qf.lora_workspace(d, lo)
    Y, dX = empty_bf16((M, N)), empty_bf16((M, K))
    dA = torch.full(f["A"].shape, 7.0, dtype=torch.float32, device="cuda")
    dB = torch.full(f["B"].shape, 7.0, dtype=torch.float32, device="cuda")
    Xd, Wd, dYd = to_dev(X), to_dev(W), to_dev(dY)
    qf.qlinear_lora_fwd(d, lo, Xd, Wd, Y, ws)
    if reuse:
        d = qf.qlinear_desc(M, N, K, wfmt, afmt, a_amax=a_amax, flags=qf.FLAG_REUSE_WS)
    qf.qlinear_lora_bwd_ste(d, lo, dYd, Xd, Wd, dX if "dX" in want else None,
                            dA if "dA" in want else None, dB if "dB" in want else None, ws)
    torch.cuda.synchronize()
    return from_dev(Y), from_dev(dX), from_dev(dA), from_dev(dB)


def _check_layer(X, W, dY, f, wfmt, afmt, got, tag=""):
    Y, dX, dA, dB = got
    m = oracle.lora_merge(W, f["B"], f["A"], f["scale"])
    what = m if wfmt == "none" else oracle.fakequant(m, wfmt)
    ahat = oracle.fakequant(X, afmt)
    assert_close(bf16_to_f64(Y), oracle.linear_fwd(ahat, what), f"{tag} Y")
    assert_close(bf16_to_f64(dX), oracle.linear_dx(dY, what), f"{tag} dX")
    rA, rB = oracle.lora_grads(dY, ahat, f["B"], f["A"], f["scale"])
    assert_close(dA.astype(np.float64), rA, f"{tag} dA")
    assert_close(dB.astype(np.float64), rB, f"{tag} dB")


@pytest.mark.parametrize("wfmt,afmt,M,N,K,r", [
    ("mxfp4", "mxfp4", 384, 264, 512, 16),
    ("nvfp4", "none", 203, 136, 256, 4),      # M not a multiple of 8
    ("q4k", "none", 129, 512, 768, 20),       # rank with a partial 16-term pass
    ("none", "none", 64, 64, 64, 1),
    ("nvfp4", "mxfp4", 520, 1000, 544, 64),
])
def test_lora_layer_small(qf, wfmt, afmt, M, N, K, r):
    rng = np.random.default_rng(M + N + K + r)
    X = workloads.normal_bf16(rng, (M, K))
    W = workloads.normal_bf16(rng, (N, K), 0.02)
    dY = workloads.normal_bf16(rng, (M, N))
    f = _factors(r, N, K, r)
    got = _lora_layer(qf, X, W, dY, f, wfmt, afmt)
    _check_layer(X, W, dY, f, wfmt, afmt, got, f"{wfmt}/{afmt}")
    # keeping the forward's quantized operands gives the same bits as re-quantizing
    again = _lora_layer(qf, X, W, dY, f, wfmt, afmt, reuse=True)
    for a, b in zip(got, again):
        assert np.array_equal(a, b)


def test_lora_layer_nvfp4_activations(qf):
    rng = np.random.default_rng(31)
    M, N, K, r = 256, 256, 256, 8
    X = workloads.normal_bf16(rng, (M, K))
    W = workloads.normal_bf16(rng, (N, K), 0.02)
    dY = workloads.normal_bf16(rng, (M, N))
    f = _factors(31, N, K, r)
    g = 3.0 * oracle.amax(X)                                   # a running amax above the batch's
    ga = torch.tensor([g], dtype=torch.float32, device="cuda")
    Y, dX, dA, dB = _lora_layer(qf, X, W, dY, f, "nvfp4", "nvfp4", a_amax=ga)
    m = oracle.lora_merge(W, f["B"], f["A"], f["scale"])
    what = oracle.fakequant(m, "nvfp4")
    ahat = oracle.nvfp4(X, g)["xhat"]
    assert_close(bf16_to_f64(Y), oracle.linear_fwd(ahat, what), "Y")
    rA, rB = oracle.lora_grads(dY, ahat, f["B"], f["A"], f["scale"])
    assert_close(dA.astype(np.float64), rA, "dA")
    assert_close(dB.astype(np.float64), rB, "dB")


def test_lora_layer_partial_outputs_and_zero_tokens(qf):
    rng = np.random.default_rng(41)
    M, N, K, r = 96, 128, 256, 16
    X = workloads.normal_bf16(rng, (M, K))
    W = workloads.normal_bf16(rng, (N, K), 0.02)
    dY = workloads.normal_bf16(rng, (M, N))
    f = _factors(41, N, K, r)
    full = _lora_layer(qf, X, W, dY, f, "mxfp4", "mxfp4")
    only_a = _lora_layer(qf, X, W, dY, f, "mxfp4", "mxfp4", want=("dA",))
    only_b = _lora_layer(qf, X, W, dY, f, "mxfp4", "mxfp4", want=("dB",))
    assert np.array_equal(only_a[2], full[2]) and np.all(only_a[3] == 7.0)
    assert np.array_equal(only_b[3], full[3]) and np.all(only_b[2] == 7.0)
    # no tokens: the factor gradients are zeros
    A, B = _dev_f32(f["A"]), _dev_f32(f["B"])
    lo = qf.lora(A, B, f["scale"])
    d = qf.qlinear_desc(0, N, K, "mxfp4", "mxfp4")
    ws = qf.lora_workspace(d, lo)
    dA = torch.full(f["A"].shape, 7.0, dtype=torch.float32, device="cuda")
    dB = torch.full(f["B"].shape, 7.0, dtype=torch.float32, device="cuda")
    Xe = torch.empty(0, K, dtype=torch.int16, device="cuda")
    dYe = torch.empty(0, N, dtype=torch.int16, device="cuda")
    qf.qlinear_lora_bwd_ste(d, lo, dYe, Xe, to_dev(W), None, dA, dB, ws)
    torch.cuda.synchronize()
    assert np.all(from_dev(dA) == 0.0) and np.all(from_dev(dB) == 0.0)


@pytest.mark.parametrize("wfmt", ["mxfp4", "nvfp4"])
def test_lora_layer_zero_adapter_matches_plain_layer(qf, wfmt):
    # B = 0 (the adapter's initialization): forward and dX equal the plain layer's bit for bit
    # (NVFP4: the merged tensor is stored once, then its amax and quantizer run over it)
    rng = np.random.default_rng(51)
    M, N, K, r = 256, 264, 512, 16
    X = workloads.normal_bf16(rng, (M, K))
    W = workloads.normal_bf16(rng, (N, K), 0.02)
    dY = workloads.normal_bf16(rng, (M, N))
    f = _factors(51, N, K, r)
    f["B"][:] = 0.0
    Y, dX, dA, dB = _lora_layer(qf, X, W, dY, f, wfmt, "mxfp4")
    d = qf.qlinear_desc(M, N, K, wfmt, "mxfp4")
    ws = qf.workspace(d)
    Y0, dX0 = empty_bf16((M, N)), empty_bf16((M, K))
    Xd, Wd = to_dev(X), to_dev(W)
    qf.qlinear_fwd(d, Xd, Wd, Y0, ws)
    qf.qlinear_bwd_ste(d, to_dev(dY), Xd, Wd, dX0, None, ws)
    torch.cuda.synchronize()
    assert np.array_equal(Y, from_dev(Y0)) and np.array_equal(dX, from_dev(dX0))
    assert np.all(dA == 0.0)


def test_lora_mlp_up_full_size_sampled(qf):
    """The MXFP4 W4A4 MLP up-projection (8192 x 14336 x 4096) with a rank-16 adapter, in the
    launch configuration the benchmark times: the merged W_hat bit for bit, Y and dX on
    sampled entries, dA and dB on sampled rows / columns."""
    w = workloads.mlp_up(seed=0)
    M, N, K = w["M"], w["N"], w["K"]
    f = workloads.lora_factors(1, N, K, r=16)
    Y, dX, dA, dB = _lora_layer(qf, w["X"], w["W"], w["dY"], f, "mxfp4", "mxfp4")
    wq = oracle.lora_quant(w["W"], f["B"], f["A"], f["scale"], "mxfp4")["xhat"]
    # W_hat of the merged weight, bit for bit, from the merged quantizer call
    lo = qf.lora(_dev_f32(f["A"]), _dev_f32(f["B"]), f["scale"])
    xh = empty_bf16((N, K))
    qf.lora_fakequant(to_dev(w["W"]), lo, "mxfp4", xhat=xh)
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(xh), wq)
    xq = oracle.mxfp4(w["X"])["xhat"]
    rng = np.random.default_rng(19)
    n = 1 << 14
    i, j = rng.integers(0, M, n), rng.integers(0, N, n)
    assert_close(bf16_to_f64(Y[i, j]), oracle.dot_rows(xq, i, wq, j), "Y sampled")
    wqT = np.ascontiguousarray(wq.T)
    i, k = rng.integers(0, M, n), rng.integers(0, K, n)
    assert_close(bf16_to_f64(dX[i, k]), oracle.dot_rows(w["dY"], i, wqT, k), "dX sampled")
    # dB[n, :] = s sum_m dY[m, n] (xq A^T)[m, :];  dA[:, k] = s sum_m (dY B)[m, :] xq[m, k]
    s = f["scale"]
    xf = bf16_to_f64(xq)
    U = xf @ f["A"].astype(np.float64).T
    cols = rng.integers(0, N, 64)
    dYc = bf16_to_f64(w["dY"][:, cols])
    assert_close(dB[cols].astype(np.float64), s * (dYc.T @ U), "dB sampled rows")
    V = np.zeros((M, f["r"]))
    B64 = f["B"].astype(np.float64)
    for m0 in range(0, M, 1024):
        V[m0:m0 + 1024] = bf16_to_f64(w["dY"][m0:m0 + 1024]) @ B64
    ks = rng.integers(0, K, 64)
    assert_close(dA[:, ks].astype(np.float64), s * (V.T @ xf[:, ks]), "dA sampled columns")


# ------------------------------------------------------------------------ grouped (MoE)
def _grouped_case(seed, E, N, K, counts):
    rng = np.random.default_rng(seed)
    off = np.zeros(E + 1, np.int64)
    off[1:] = np.cumsum(counts)
    T = int(off[-1])
    X = workloads.normal_bf16(rng, (max(T, 1), K))[:T]
    W = workloads.normal_bf16(rng, (E * N, K), 0.02).reshape(E, N, K)
    dY = workloads.normal_bf16(rng, (max(T, 1), N))[:T]
    return off, T, X, W, dY


@pytest.mark.parametrize("wfmt,afmt,shared,r", [
    ("mxfp4", "mxfp4", "none", 16),
    ("nvfp4", "none", "A", 8),          # gate/up layout: A shared, per-expert tensor amax
    ("nvfp4", "mxfp4", "B", 20),        # down layout: B shared
    ("q4k", "none", "none", 3),
])
def test_grouped_lora_layer(qf, wfmt, afmt, shared, r):
    E, N, K = 6, 264, 512
    counts = [37, 0, 300, 5, 1100, 64]     # an empty expert, chunks past 1024 rows, tiny ones
    off, T, X, W, dY = _grouped_case(r, E, N, K, counts)
    rng = np.random.default_rng(100 + r)
    A = (rng.standard_normal((r, K) if shared == "A" else (E, r, K)) / np.sqrt(K)).astype(np.float32)
    B = (rng.standard_normal((N, r) if shared == "B" else (E, N, r)) * 0.01).astype(np.float32)
    s = 2.0
    lo = qf.lora(_dev_f32(A), _dev_f32(B), s, a_shared=shared == "A", b_shared=shared == "B")
    offd = torch.from_numpy(off).cuda()
    Xd, Wd, dYd = to_dev(X), to_dev(W.reshape(E * N, K)), to_dev(dY)

    def run(reuse):
        d = qf.grouped_desc(E, T, N, K, wfmt, afmt)
        ws = qf.grouped_lora_workspace(d, lo)
        Y, dX = empty_bf16((T, N)), empty_bf16((T, K))
        dA = torch.full(A.shape, 7.0, dtype=torch.float32, device="cuda")
        dB = torch.full(B.shape, 7.0, dtype=torch.float32, device="cuda")
        qf.qlinear_grouped_lora_fwd(d, lo, offd, Xd, Wd, Y, ws)
        if reuse:
            d = qf.grouped_desc(E, T, N, K, wfmt, afmt, flags=qf.FLAG_REUSE_WS)
        qf.qlinear_grouped_lora_bwd_ste(d, lo, offd, dYd, Xd, Wd, dX, dA, dB, ws)
        torch.cuda.synchronize()
        return from_dev(Y), from_dev(dX), from_dev(dA), from_dev(dB)

    Y, dX, dA, dB = run(False)
    xh = oracle.lora_quant_grouped(W, B, A, s, wfmt) if wfmt != "none" else None
    ahat = oracle.fakequant(X, afmt)
    Yr = np.zeros((T, N))
    dXr = np.zeros((T, K))
    for e in range(E):
        rows = slice(off[e], off[e + 1])
        Yr[rows] = oracle.linear_fwd(ahat[rows], xh[e])
        dXr[rows] = oracle.linear_dx(dY[rows], xh[e])
    assert_close(bf16_to_f64(Y), Yr, "Y")
    assert_close(bf16_to_f64(dX), dXr, "dX")
    rA, rB = oracle.lora_grads_grouped(dY, ahat, off, B, A, s)
    assert_close(dA.astype(np.float64), rA, "dA")
    assert_close(dB.astype(np.float64), rB, "dB")
    if shared != "A":
        assert np.all(dA[1] == 0.0)        # expert 1 has no rows
    if shared != "B":
        assert np.all(dB[1] == 0.0)
    again = run(True)
    for a, b in zip((Y, dX, dA, dB), again):
        assert np.array_equal(a, b)


def test_grouped_lora_no_tokens(qf):
    E, N, K, r = 3, 64, 256, 4
    off = np.zeros(E + 1, np.int64)
    W = workloads.normal_bf16(np.random.default_rng(1), (E * N, K), 0.02)
    A = np.ones((E, r, K), np.float32)
    B = np.ones((E, N, r), np.float32)
    lo = qf.lora(_dev_f32(A), _dev_f32(B), 1.0)
    d = qf.grouped_desc(E, 0, N, K, "mxfp4", "none")
    ws = qf.grouped_lora_workspace(d, lo)
    dA = torch.full(A.shape, 7.0, dtype=torch.float32, device="cuda")
    dB = torch.full(B.shape, 7.0, dtype=torch.float32, device="cuda")
    e0 = torch.empty(0, K, dtype=torch.int16, device="cuda")
    e1 = torch.empty(0, N, dtype=torch.int16, device="cuda")
    qf.qlinear_grouped_lora_bwd_ste(d, lo, torch.from_numpy(off).cuda(), e1, e0, to_dev(W), None,
                                    dA, dB, ws)
    torch.cuda.synchronize()
    assert np.all(from_dev(dA) == 0.0) and np.all(from_dev(dB) == 0.0)
