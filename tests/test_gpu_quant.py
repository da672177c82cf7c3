"""GPU parity of the fake-quantization kernels against the CPU oracle: bit-exact codes,
scales, tensor scale and dequantized bf16 on seeded inputs (LLM-shaped tensors at full size,
wide-range and edge-case tensors, exhaustive bf16 inputs, ragged rows / strides)."""
import numpy as np
import pytest

import oracle
import workloads
from tests.helpers import empty_bf16, from_dev, to_dev, wide_range_bf16

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def qf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_39223_amd as qf
    qf.lib()
    return qf


def _strided(x, ld):
    """Embed [R, K] into an [R, ld] buffer (row stride ld) and return (buffer view, base)."""
    R, K = x.shape
    buf = np.full((R, ld), 0x7FC0, np.uint16)   # NaN padding: must never be read
    buf[:, :K] = x
    return buf


def run_mxfp4(qf, x, ld=None):
    R, K = x.shape
    if ld is None:
        xd = to_dev(x)
    else:
        xd = to_dev(_strided(x, ld))[:, :K]
    codes = torch.empty(R, K // 2, dtype=torch.uint8, device="cuda")
    scales = torch.empty(R, K // 32, dtype=torch.uint8, device="cuda")
    xhat = empty_bf16((R, K))
    qf.fakequant_mxfp4(xd, codes, scales, xhat)
    torch.cuda.synchronize()
    return {"codes": from_dev(codes), "scales": from_dev(scales), "xhat": from_dev(xhat)}


def run_nvfp4(qf, x, amax_in=None, ld=None):
    R, K = x.shape
    xd = to_dev(x) if ld is None else to_dev(_strided(x, ld))[:, :K]
    amax = torch.tensor([0.0 if amax_in is None else amax_in], dtype=torch.float32, device="cuda")
    s_out = torch.zeros(1, dtype=torch.float32, device="cuda")
    codes = torch.empty(R, K // 2, dtype=torch.uint8, device="cuda")
    scales = torch.empty(R, K // 16, dtype=torch.uint8, device="cuda")
    xhat = empty_bf16((R, K))
    mode = qf.AMAX_COMPUTE if amax_in is None else qf.AMAX_GIVEN
    qf.fakequant_nvfp4(xd, amax, mode, s_out, codes, scales, xhat)
    torch.cuda.synchronize()
    return {"codes": from_dev(codes), "scales": from_dev(scales), "xhat": from_dev(xhat),
            "S": float(s_out.item()), "amax": float(amax.item())}


def run_q4k(qf, x, ld=None):
    R, K = x.shape
    xd = to_dev(x) if ld is None else to_dev(_strided(x, ld))[:, :K]
    packed = torch.empty(R, K // 256, 144, dtype=torch.uint8, device="cuda")
    xhat = empty_bf16((R, K))
    qf.fakequant_q4k(xd, packed, xhat)
    torch.cuda.synchronize()
    return {"packed": from_dev(packed), "xhat": from_dev(xhat)}


def assert_same(got, want, keys, what=""):
    for k in keys:
        g, w = np.asarray(got[k]), np.asarray(want[k])
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)
            i = tuple(bad[0])
            raise AssertionError(f"{what} {k}: {len(bad)} mismatches, first at {i}: "
                                 f"got {g[i]} want {w[i]}")


def all_bf16_blocks(block, finite_only=False, seed=None):
    v = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    if finite_only:
        v = v[(v & 0x7F80) != 0x7F80]
    if seed is not None:
        v = np.random.default_rng(seed).permutation(v)
    n = len(v) // block * block
    return v[:n].reshape(-1, block)


# ------------------------------------------------------------------------------- MXFP4
def test_mxfp4_exhaustive_bf16_inputs(qf):
    for seed in (None, 1):
        x = all_bf16_blocks(32, seed=seed).reshape(-1, 256)
        assert_same(run_mxfp4(qf, x), oracle.mxfp4(x), ("codes", "scales", "xhat"), "mxfp4")


def test_mxfp4_wide_range_and_ragged(qf):
    rng = np.random.default_rng(0)
    for R, K, ld in [(1, 32, None), (3, 96, None), (37, 2080, None), (130, 4096, 4160),
                     (5, 8192, None)]:
        x = wide_range_bf16(rng, (R, K), lo_exp=-140, hi_exp=126)
        assert_same(run_mxfp4(qf, x, ld), oracle.mxfp4(x), ("codes", "scales", "xhat"),
                    f"mxfp4 {R}x{K}")


def test_mxfp4_full_size_mlp_up_operands(qf):
    w = workloads.mlp_up(seed=0)
    for name in ("W", "X"):
        assert_same(run_mxfp4(qf, w[name]), oracle.mxfp4(w[name]), ("codes", "scales", "xhat"),
                    "mxfp4 " + name)


# ------------------------------------------------------------------------------- NVFP4
def test_nvfp4_exhaustive_finite_bf16_inputs(qf):
    for seed in (None, 2):
        x = all_bf16_blocks(16, finite_only=True, seed=seed).reshape(-1, 64)
        want = oracle.nvfp4(x)
        got = run_nvfp4(qf, x)
        assert_same(got, want, ("codes", "scales", "xhat"), "nvfp4 computed g")
        assert got["S"] == want["S"]
        # the same inputs under several supplied (running / tied) amax values
        for g in [1.0, 3.0e-3, 2.5e5, 1.0e-30, 3.0e38]:
            g32 = float(np.float32(g))
            assert_same(run_nvfp4(qf, x[:64], amax_in=g32), oracle.nvfp4(x[:64], amax_in=g32),
                        ("codes", "scales", "xhat"), f"nvfp4 g={g}")


def test_nvfp4_wide_range_ragged_and_amax(qf):
    rng = np.random.default_rng(3)
    for R, K, ld in [(1, 16, None), (7, 48, None), (33, 4112, None), (64, 1024, 1040)]:
        for spread in (3, 30):
            x = wide_range_bf16(rng, (R, K), lo_exp=-spread, hi_exp=spread)
            want = oracle.nvfp4(x)
            got = run_nvfp4(qf, x, ld=ld)
            assert_same(got, want, ("codes", "scales", "xhat"), f"nvfp4 {R}x{K}")
            assert got["S"] == want["S"] and got["amax"] == oracle.amax(x)


def test_nvfp4_scales_whose_reciprocal_overflows(qf):
    """Block decode scales below 2^-128 (tensor amax among the float denormals, computed from a
    tensor of bf16 denormals or supplied by the caller): fl(1 / D) overflows, zeros scale to
    0 * Inf and encode as magnitude 0 as the oracle's nearest-value rule gives; every other
    element saturates at 6."""
    v = np.arange(0x80, dtype=np.uint16)                  # +0, the positive bf16 denormals
    x = np.concatenate([v, v | 0x8000]).reshape(-1, 64)   # and their negatives (-0 included)
    got, want = run_nvfp4(qf, x), oracle.nvfp4(x)
    assert_same(got, want, ("codes", "scales", "xhat"), "nvfp4 denormal tensor")
    assert got["S"] == want["S"] and got["amax"] == oracle.amax(x)
    xf = all_bf16_blocks(16, finite_only=True, seed=5).reshape(-1, 64)[:256]
    for g in [1.0e-39, 1.0e-41, 3.0e-44, 1.4e-45]:
        g32 = float(np.float32(g))
        assert_same(run_nvfp4(qf, xf, amax_in=g32), oracle.nvfp4(xf, amax_in=g32),
                    ("codes", "scales", "xhat"), f"nvfp4 g={g}")


def test_nvfp4_zero_tensor(qf):
    x = np.zeros((4, 64), np.uint16)
    x[2, 5] = 0x8000
    got = run_nvfp4(qf, x)
    assert_same(got, oracle.nvfp4(x), ("codes", "scales", "xhat"), "nvfp4 zeros")
    assert got["S"] == 0.0


def test_nvfp4_full_size_weights(qf):
    w = workloads.single_linear(seed=0)
    assert_same(run_nvfp4(qf, w["W"]), oracle.nvfp4(w["W"]), ("codes", "scales", "xhat", "S"),
                "nvfp4 512x512")
    rng = np.random.default_rng(4)
    W = workloads.normal_bf16(rng, (24576, 4096), 0.02)     # fused gate/up of the 9B layer
    assert_same(run_nvfp4(qf, W), oracle.nvfp4(W), ("codes", "scales", "xhat", "S"),
                "nvfp4 24576x4096")


# -------------------------------------------------------------------------------- Q4_K
def test_q4k_wide_range_edge_blocks_and_ragged(qf):
    rng = np.random.default_rng(5)
    # (K a multiple of 1024 takes the 16-element form: 7 x 2048 and 5 x 3072 leave whole
    # wavefronts of a workgroup past the row end, and odd row counts a half-used row pair)
    for R, K, ld in [(1, 256, None), (9, 768, None), (40, 4096, 4352), (3, 8448, None),
                     (7, 2048, None), (5, 3072, 3200)]:
        x = wide_range_bf16(rng, (R, K), lo_exp=-20, hi_exp=10, zero_frac=0.05)
        x[0, :32] = 0                                  # all-zero sub-block
        x[-1, 32:64] = 0x8000                          # all -0 sub-block
        x[-1, 64:96] = np.abs(x[-1, 64:96].astype(np.int32)).astype(np.uint16) | 0x8000
        assert_same(run_q4k(qf, x, ld), oracle.q4k(x), ("packed", "xhat"), f"q4k {R}x{K}")


@pytest.mark.parametrize("width", [256, 1024])
def test_q4k_exhaustive_bf16_inputs_below_limits(qf, width):
    # every bf16 pattern with magnitude below 2^100 (super-block ranges stay finite in FP32),
    # then every pattern below 2^14 (scales inside the FP16 range), in shuffled blocks; rows of
    # 256 and of 1024 elements (the row quantizer's two forms: 8 and 16 elements per lane)
    v = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    for lim, seed in ((2.0 ** 100, 7), (2.0 ** 14, 8)):
        mag = np.abs((v.astype(np.uint32) << 16).view(np.float32))
        sel = np.random.default_rng(seed).permutation(v[mag < lim])
        x = sel[: len(sel) // width * width].reshape(-1, width)
        assert_same(run_q4k(qf, x), oracle.q4k(x), ("packed", "xhat"), f"q4k below {lim}")


def q4k_tie_rows():
    """Super-blocks whose element quotients (x + t2) / t1 land exactly on half-integers: the
    first sub-block spans [-1/32, 29.5] (step 63/32, so d = 1/32), the other seven span
    [0, 15] (ls = 32, t1 = 1, t2 = 0) and hold k + 1/2 values (rounding ties)."""
    rng = np.random.default_rng(11)
    rows = []
    for r in range(6):
        subs = [np.concatenate([[29.5, -0.03125], rng.integers(0, 59, 30) * 0.5])]
        subs += [np.concatenate([[0.0, 15.0], rng.integers(0, 15, 30) + 0.5]) for _ in range(7)]
        row = np.concatenate([rng.permutation(s) for s in subs]).astype(np.float32)
        rows.append(-row[::-1].copy() if r % 2 else row)
    return (np.stack(rows).view(np.uint32) >> 16).astype(np.uint16)


def test_q4k_exact_rounding_ties(qf):
    x = q4k_tie_rows()
    ref = oracle.q4k(x)
    d, dmin, ls, lm, q = oracle.q4k_unpack_block(ref["packed"][0, 0])
    assert d == 0x2800 and ls[1:] == [32] * 7                 # t1 = 1 in sub-blocks 1-7
    assert_same(run_q4k(qf, x), ref, ("packed", "xhat"), "q4k ties")
    assert_same(run_q4k_mse(qf, x), oracle.q4k_mse(x), ("packed", "xhat"), "q4k-mse ties")


def test_q4k_exact_rounding_ties_1024_wide_rows(qf):
    # the tie rows laid end to end as rows of 1024 elements (the 16-elements-per-lane form)
    x = np.tile(q4k_tie_rows(), (2, 1))[:8].reshape(2, 1024)
    assert_same(run_q4k(qf, x), oracle.q4k(x), ("packed", "xhat"), "q4k ties, 1024-wide rows")


def test_q4k_full_size_export_weight(qf):
    w = workloads.q4k_weight(seed=0, scale=64)
    assert_same(run_q4k(qf, w["W"]), oracle.q4k(w["W"]), ("packed", "xhat"), "q4k 14336x4096")


# -------------------------------------------------------------- Q4_K with an MSE search
def run_q4k_mse(qf, x, ld=None):
    R, K = x.shape
    xd = to_dev(x) if ld is None else to_dev(_strided(x, ld))[:, :K]
    packed = torch.empty(R, K // 256, 144, dtype=torch.uint8, device="cuda")
    xhat = empty_bf16((R, K))
    qf.fakequant_q4k_mse(xd, packed, xhat)
    torch.cuda.synchronize()
    return {"packed": from_dev(packed), "xhat": from_dev(xhat)}


def test_q4k_mse_bit_exact(qf):
    rng = np.random.default_rng(15)
    cases = [
        ("normal", workloads.normal_bf16(rng, (37, 512), 0.02), None),
        ("heavy", workloads.to_bf16((rng.standard_t(3, size=(16, 1024)) * 0.02).astype(np.float32)), 1096),
        ("wide", wide_range_bf16(rng, (9, 768), lo_exp=-20, hi_exp=10, zero_frac=0.05), None),
        ("ints", workloads.to_bf16(rng.integers(-8, 9, size=(8, 256)).astype(np.float32)), None),
    ]
    x = cases[2][1]
    x[0, :32] = 0                                      # all-zero sub-block
    x[-1, 32:64] = 0x8000                              # all -0 sub-block
    x[-1, 64:96] = 0x3F80                              # constant sub-block
    for name, x, ld in cases:
        assert_same(run_q4k_mse(qf, x, ld), oracle.q4k_mse(x), ("packed", "xhat"), f"q4k-mse {name}")


def test_q4k_mse_exhaustive_bf16_inputs_below_limits(qf):
    v = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    mag = np.abs((v.astype(np.uint32) << 16).view(np.float32))
    sel = np.random.default_rng(9).permutation(v[mag < 2.0 ** 14])
    x = sel[: len(sel) // 256 * 256].reshape(-1, 256)
    assert_same(run_q4k_mse(qf, x), oracle.q4k_mse(x), ("packed", "xhat"), "q4k-mse exhaustive")


def test_q4k_mse_export_weight_rows(qf):
    w = workloads.q4k_weight(seed=0, n_scale=8)      # 1792 x 4096 rows of the export weight
    assert_same(run_q4k_mse(qf, w["W"]), oracle.q4k_mse(w["W"]), ("packed", "xhat"),
                "q4k-mse 1792x4096")


# ------------------------------------------------------------------------------- amax
def test_amax_and_running_accumulate(qf):
    rng = np.random.default_rng(6)
    a = wide_range_bf16(rng, (100, 1024), lo_exp=-5, hi_exp=5)
    b = wide_range_bf16(rng, (60, 1024), lo_exp=-5, hi_exp=9)
    out = torch.zeros(1, dtype=torch.float32, device="cuda")
    qf.amax(to_dev(a), out, accumulate=False)
    torch.cuda.synchronize()
    assert float(out.item()) == oracle.amax(a)
    qf.amax(to_dev(b), out, accumulate=True)
    torch.cuda.synchronize()
    assert float(out.item()) == max(oracle.amax(a), oracle.amax(b))
    qf.amax(to_dev(a), out, accumulate=True)
    torch.cuda.synchronize()
    assert float(out.item()) == max(oracle.amax(a), oracle.amax(b))


def test_amax_passes_do_not_see_each_other(qf):
    """Each amax pass folds into a reduction slot that its last workgroup clears: a pass over a
    small tensor right after one over a large tensor returns the small amax (no carry-over, no
    clearing dispatch), whatever the output held before; contiguous (flat) and strided (rows)
    tensors, a zero tensor, a NaN, and more passes than the slot ring holds."""
    rng = np.random.default_rng(11)
    big = wide_range_bf16(rng, (300, 1024), lo_exp=-3, hi_exp=12)
    small = wide_range_bf16(rng, (64, 4096), lo_exp=-8, hi_exp=-2)
    strided = wide_range_bf16(rng, (37, 520), lo_exp=-6, hi_exp=0)
    zero = np.zeros((16, 256), np.uint16)
    nan = small.copy()
    nan[5, 7] = 0x7FC1
    dev = {k: to_dev(v) for k, v in dict(big=big, small=small, zero=zero, nan=nan).items()}
    sd = to_dev(np.pad(strided, ((0, 0), (0, 8))))[:, :520]
    want = {"big": oracle.amax(big), "small": oracle.amax(small), "zero": 0.0,
            "strided": oracle.amax(strided)}
    out = torch.full((1,), 1e30, dtype=torch.float32, device="cuda")
    order = ["big", "small", "strided", "big", "zero", "strided", "small"] * 700   # 4900: round the ring
    got = torch.empty(len(order), dtype=torch.float32, device="cuda")
    for i, k in enumerate(order):
        qf.amax(sd if k == "strided" else dev[k], out, accumulate=False)
        got[i] = out[0]
    torch.cuda.synchronize()
    g = got.cpu().numpy()
    for i, k in enumerate(order):
        assert g[i] == want[k], (i, k, g[i], want[k])
    qf.amax(dev["nan"], out, accumulate=False)
    torch.cuda.synchronize()
    assert np.isnan(out.item())
    qf.amax(dev["small"], out, accumulate=False)      # the NaN pass left its slot clear too
    torch.cuda.synchronize()
    assert out.item() == want["small"]


def test_amax_empty_tensor(qf):
    out = torch.full((1,), 5.0, dtype=torch.float32, device="cuda")
    x = torch.empty((0, 64), dtype=torch.int16, device="cuda")
    qf.amax(x, out, accumulate=True)
    torch.cuda.synchronize()
    assert out.item() == 5.0
    qf.amax(x, out, accumulate=False)
    torch.cuda.synchronize()
    assert out.item() == 0.0


@pytest.mark.parametrize("K,col", [(12, 10), (5, 4), (1, 0), (1003, 1001)])
def test_amax_row_tail_not_multiple_of_8(qf, K, col):
    """K % 8 != 0 inside a wider row stride: the row's last K % 8 elements count (the maximum
    sits there) and the padding past K (larger still) is never read."""
    rng = np.random.default_rng(K)
    R, ld = 37, (K + 7) // 8 * 8 + 8
    x = (rng.standard_normal((R, ld)) * 0.5).astype(np.float32)
    x[:, K:] = 1e30                               # padding: must not be read
    x[17, col] = -7.25                            # the maximum |x| among the K columns
    u = x.view(np.uint32)
    buf = ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)
    out = torch.full((1,), 123.0, dtype=torch.float32, device="cuda")
    xd = to_dev(buf)[:, :K]
    qf.amax(xd, out, accumulate=False)
    torch.cuda.synchronize()
    assert float(out.item()) == oracle.amax(np.ascontiguousarray(buf[:, :K])) == 7.25


@pytest.mark.parametrize("R", [100, 600])
def test_amax_rows_two_dimensional_grid(qf, R):
    """Strided rows 2999 wide run the row kernel on a grid with two workgroup columns and 7 or 38
    workgroup rows; its workgroups fold in two levels by their linear index. The maximum is
    planted in one workgroup's region at a time (both columns, first / middle / last row band,
    the row's ragged tail) and must come out every time."""
    K, ld = 2999, 3008
    rng = np.random.default_rng(R)
    base = (rng.uniform(-0.9, 0.9, (R, ld))).astype(np.float32)
    base[:, K:] = 1e30                            # padding: must not be read
    bands = (R + 15) // 16
    spots = [(3, 7 * 8 + 2), (3, (256 + 7) * 8 + 2), (16 * (bands // 2) + 5, 11),
             (R - 1, 2100), (R - 1, K - 1), (16 * (bands - 1), K - 3)]
    out = torch.full((1,), 55.0, dtype=torch.float32, device="cuda")
    for r, c in spots:
        x = base.copy()
        x[r, c] = -9.5
        u = x.view(np.uint32)
        buf = ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)
        qf.amax(to_dev(buf)[:, :K], out, accumulate=False)
        torch.cuda.synchronize()
        assert float(out.item()) == oracle.amax(np.ascontiguousarray(buf[:, :K])) == 9.5, (r, c)


def test_q4k_handworked_block_bit_exact(qf):
    """The hand-worked super-block of the golden fixture: the kernel's 144 bytes equal the
    bytes worked out by hand (6-bit scale / min rounding, scale-bit and nibble layout)."""
    from tests.test_oracle_quant import _handworked_q4k_block
    x, _, _, _, _, blk = _handworked_q4k_block()
    xr = np.repeat(x, 3, axis=0)                  # a few rows, one super-block each
    packed = torch.empty(3, 1, 144, dtype=torch.uint8, device="cuda")
    xhat = empty_bf16((3, 256))
    qf.fakequant_q4k(to_dev(xr), packed, xhat)
    torch.cuda.synchronize()
    got = from_dev(packed)
    for r in range(3):
        assert bytes(got[r, 0]) == blk
    np.testing.assert_array_equal(from_dev(xhat), oracle.q4k(xr)["xhat"])


def test_determinism_two_runs(qf):
    w = workloads.mlp_up(seed=1, scale=8, n_scale=8)
    a = run_nvfp4(qf, w["X"])
    b = run_nvfp4(qf, w["X"])
    assert_same(a, b, ("codes", "scales", "xhat", "S"), "repeat")


def test_empty_inputs_are_no_ops(qf):
    x = torch.zeros(0, 64, dtype=torch.int16, device="cuda")
    xhat = torch.zeros(0, 64, dtype=torch.int16, device="cuda")
    qf.fakequant_mxfp4(x, None, None, xhat)
    amax = torch.full((1,), 5.0, device="cuda")
    s_out = torch.full((1,), 5.0, device="cuda")
    qf.fakequant_nvfp4(x, amax, qf.AMAX_COMPUTE, s_out, None, None, xhat)
    torch.cuda.synchronize()
    assert float(amax.item()) == 0.0 and float(s_out.item()) == 0.0


@pytest.mark.parametrize("fmt,R,K,ldo", [("mxfp4", 8, 32, None), ("mxfp4", 72, 2080, 80),
                                         ("nvfp4", 136, 528, None), ("nvfp4", 64, 256, 200),
                                         ("q4k", 200, 768, None), ("q4k", 8, 256, 16)])
def test_transposed_fakequant_bit_exact(qf, fmt, R, K, ldo):
    """out[k][r] = x_hat[r][k]: ragged 64 x 256 tiles both ways, padded output rows kept."""
    rng = np.random.default_rng(21)
    if fmt == "q4k":
        x = wide_range_bf16(rng, (R, K), lo_exp=-20, hi_exp=12)
    else:
        x = wide_range_bf16(rng, (R, K), lo_exp=-140, hi_exp=126)
    if fmt == "mxfp4":
        x[1, 5] = 0x7FC0                           # NaN block
        x[3, min(40, K - 1)] = 0xFF80              # -Inf block
    ldo = ldo or R
    amax_in = None
    amax = None
    if fmt == "nvfp4":
        amax_in = float(np.float32(oracle.amax(x)))
        amax = torch.tensor([amax_in], dtype=torch.float32, device="cuda")
    out = torch.full((K, ldo), 0x1234, dtype=torch.int16, device="cuda")
    qf.fakequant_transposed(to_dev(x), fmt, out, amax)
    torch.cuda.synchronize()
    got = from_dev(out)
    want = oracle.fakequant(x, fmt, amax_in)
    assert np.array_equal(got[:, :R], np.ascontiguousarray(want.T)), fmt
    assert np.all(got[:, R:] == 0x1234)
