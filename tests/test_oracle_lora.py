"""Pins of the LoRA-QAD oracle (Sec. 3.3, Eqs. qad-lora, export-lora; gradients by Eq. ste
and the chain rule through W + s B A).  Each test checks the oracle against something other
than itself: IEEE identities, exactly representable closed forms, cases where the merge
order or a missing fused multiply-add would change the result, an FP64 reference within one
bf16 step, torch autograd in float64, and the paper's statement that the exported checkpoint
comes from the same merged weights as training."""
import numpy as np
import pytest

import oracle
from tests.helpers import bf16_to_f64, f64_to_bf16_exact
import workloads

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _w(rng, N, K, std=0.02):
    return workloads.normal_bf16(rng, (N, K), std)


def test_zero_update_returns_the_base_weight():
    rng = np.random.default_rng(1)
    w = _w(rng, 24, 40)
    w[0, :4] = [0x8000, 0x0000, 0x7F80, 0xFF80]        # -0, +0, +inf, -inf
    w[1, 0] = 0x7FC0                                   # NaN
    A = rng.standard_normal((3, 40)).astype(np.float32)
    m = oracle.lora_merge(w, np.zeros((24, 3), np.float32), A, 2.0)
    exp = w.copy()
    exp[0, 0] = 0x0000                                 # IEEE: -0 + (+0) = +0
    assert np.array_equal(m, exp)


def test_integer_closed_form():
    # W, B integers; A = 1; s = 0.5: W + 0.5 * rowsum(B) is exact in bf16
    rng = np.random.default_rng(2)
    N, K, r = 16, 64, 5
    wv = rng.integers(-8, 9, size=(N, K)).astype(np.float64)
    B = rng.integers(-6, 7, size=(N, r)).astype(np.float32)
    A = np.ones((r, K), np.float32)
    m = oracle.lora_merge(f64_to_bf16_exact(wv), B, A, 0.5)
    assert np.array_equal(bf16_to_f64(m), wv + 0.5 * B.astype(np.float64).sum(1, keepdims=True))


def test_operands_are_not_transposed():
    # B A with powers of two per (n, j) and (j, k): every entry is an exact sum of two
    # powers of two that bf16 holds, and swapping the rank index or a factor changes it
    N, K, r = 3, 8, 2
    B = np.array([[1, 2], [4, 8], [16, 32]], np.float32)
    A = np.array([[2.0 ** -(k + 1) for k in range(K)], [2.0 ** -(k + 3) for k in range(K)]],
                 np.float32)
    m = oracle.lora_merge(np.zeros((N, K), np.uint16), B, A, 1.0)
    assert np.array_equal(bf16_to_f64(m), B.astype(np.float64) @ A.astype(np.float64))


def test_rank_terms_accumulate_in_increasing_order():
    # terms 2^24, 1, 1: in rank order each +1 ties back to 2^24; in reverse order 2^24 + 2
    B = np.array([[2.0 ** 24, 1.0, 1.0]], np.float32)
    A = np.ones((3, 8), np.float32)
    m = oracle.lora_merge(np.zeros((1, 8), np.uint16), B, A, 1.0)
    assert np.all(bf16_to_f64(m) == 2.0 ** 24)


def test_each_rank_term_is_one_fused_multiply_add():
    # acc = -(1 + 2^-11), then (1 + 2^-12)^2 = 1 + 2^-11 + 2^-24: the fused step leaves
    # exactly 2^-24, a separately rounded product (to 1 + 2^-11) would leave 0
    u = 1.0 + 2.0 ** -12
    B = np.array([[-(1.0 + 2.0 ** -11), u]], np.float32)
    A = np.array([[1.0] * 8, [u] * 8], np.float32)
    m = oracle.lora_merge(np.zeros((1, 8), np.uint16), B, A, 1.0)
    assert np.all(bf16_to_f64(m) == 2.0 ** -24)


def test_scale_applies_to_the_product_then_the_sum_rounds_once():
    # W = 1, s * acc = 2^-8 + 2^-17: 1 + t lies just above the half step 2^-8 of bf16 at 1
    # and rounds once, up to 1 + 2^-7; rounding t to bf16 first (2^-8) would leave a tie
    # that goes to the even 1.0
    w = np.full((1, 8), 0x3F80, np.uint16)
    B = np.array([[1.0]], np.float32)
    A = np.full((1, 8), 2.0 ** -9 + 2.0 ** -18, np.float32)
    m = oracle.lora_merge(w, B, A, 2.0)
    assert np.all(m == 0x3F81)


def test_matches_float64_merge_within_one_bf16_step():
    d = workloads.lora_factors(3, 96, 256, r=16)
    rng = np.random.default_rng(4)
    w = _w(rng, 96, 256)
    m = bf16_to_f64(oracle.lora_merge(w, d["B"], d["A"], d["scale"]))
    ref = bf16_to_f64(w) + d["scale"] * (d["B"].astype(np.float64) @ d["A"].astype(np.float64))
    step = np.exp2(np.floor(np.log2(np.abs(ref))) - 7)          # one bf16 step at |ref|
    assert np.all(np.abs(m - ref) <= step)
    assert np.mean(np.abs(m - ref) <= 0.5 * step) > 0.99       # round-to-nearest almost always
    assert np.mean(m != bf16_to_f64(w)) > 0.3                  # the update moves many elements


@pytest.mark.parametrize("fmt", ["nvfp4", "mxfp4", "q4k"])
def test_export_decodes_to_the_training_weight(fmt):
    # Eq. export-lora quantizes the same merged weight the forward pass used (Eq. qad-lora):
    # decoding the exported codes gives the training W_hat bit for bit
    d = workloads.lora_factors(5, 32, 512, r=4)
    w = _w(np.random.default_rng(6), 32, 512)
    q = oracle.lora_quant(w, d["B"], d["A"], d["scale"], fmt)
    if fmt == "nvfp4":
        dec = oracle.nvfp4_dequant(q["codes"], q["scales"], q["S"], 512)
        assert q["amax"] == oracle.amax(q["merged"])
        assert q["amax"] != oracle.amax(w)
    elif fmt == "mxfp4":
        dec = oracle.mxfp4_dequant(q["codes"], q["scales"], 512)
    else:
        dec = oracle.q4k_dequant(q["packed"], 512)
    assert np.array_equal(dec, q["xhat"])
    assert not np.array_equal(q["xhat"], oracle.fakequant(w, fmt))


def test_factor_gradients_match_torch_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    M, N, K, r = 12, 40, 24, 3
    dy = workloads.normal_bf16(rng, (M, N))
    ahat = workloads.normal_bf16(rng, (M, K))
    w = _w(rng, N, K)
    A = rng.standard_normal((r, K)).astype(np.float32)
    B = rng.standard_normal((N, r)).astype(np.float32)
    s = 0.75
    dA, dB = oracle.lora_grads(dy, ahat, B, A, s)
    tA = torch.tensor(A, dtype=torch.float64, requires_grad=True)
    tB = torch.tensor(B, dtype=torch.float64, requires_grad=True)
    # straight-through: the quantizer is the identity in the backward, so the loss seen by
    # the factors is <dO, A_hat (W + s B A)^T>
    Wm = torch.tensor(bf16_to_f64(w)) + s * (tB @ tA)
    loss = (torch.tensor(bf16_to_f64(dy)) * (torch.tensor(bf16_to_f64(ahat)) @ Wm.T)).sum()
    loss.backward()
    assert np.allclose(dA, tA.grad.numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(dB, tB.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_factor_gradient_finite_difference():
    rng = np.random.default_rng(8)
    M, N, K, r = 6, 10, 8, 2
    dy = bf16_to_f64(workloads.normal_bf16(rng, (M, N)))
    ah = bf16_to_f64(workloads.normal_bf16(rng, (M, K)))
    A = rng.standard_normal((r, K))
    B = rng.standard_normal((N, r))
    s = 1.5
    dA, dB = oracle.lora_grads(workloads.to_bf16(dy), workloads.to_bf16(ah), B, A, s)
    loss = lambda A_, B_: float((dy * (ah @ (s * B_ @ A_).T)).sum())   # W drops out (linear)
    h = 1e-6
    for (j, k) in [(0, 0), (1, 5)]:
        Ap = A.copy(); Ap[j, k] += h
        Am = A.copy(); Am[j, k] -= h
        assert abs((loss(Ap, B) - loss(Am, B)) / (2 * h) - dA[j, k]) < 1e-6 * max(1, abs(dA[j, k]))
    for (n, j) in [(0, 1), (9, 0)]:
        Bp = B.copy(); Bp[n, j] += h
        Bm = B.copy(); Bm[n, j] -= h
        assert abs((loss(A, Bp) - loss(A, Bm)) / (2 * h) - dB[n, j]) < 1e-6 * max(1, abs(dB[n, j]))


@pytest.mark.parametrize("shared", ["none", "A", "B"])
def test_grouped_factor_gradients_match_torch_autograd(shared):
    # the MoE layer's loss is the sum of the experts' losses; autograd on the whole layer
    # pins the per-expert terms and the sum over experts of a shared factor
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(9)
    E, N, K, r = 3, 16, 8, 2
    off = np.array([0, 5, 5, 12])                       # expert 1 receives no rows
    T = int(off[-1])
    dy = workloads.normal_bf16(rng, (T, N))
    ah = workloads.normal_bf16(rng, (T, K))
    A = rng.standard_normal((r, K) if shared == "A" else (E, r, K)).astype(np.float32)
    B = rng.standard_normal((N, r) if shared == "B" else (E, N, r)).astype(np.float32)
    s = 0.5
    dA, dB = oracle.lora_grads_grouped(dy, ah, off, B, A, s)
    tA = torch.tensor(A, dtype=torch.float64, requires_grad=True)
    tB = torch.tensor(B, dtype=torch.float64, requires_grad=True)
    loss = 0
    for e in range(E):
        Ae = tA if shared == "A" else tA[e]
        Be = tB if shared == "B" else tB[e]
        rows = slice(off[e], off[e + 1])
        loss = loss + (torch.tensor(bf16_to_f64(dy[rows])) *
                       (torch.tensor(bf16_to_f64(ah[rows])) @ (s * Be @ Ae).T)).sum()
    loss.backward()
    assert np.allclose(dA, tA.grad.numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(dB, tB.grad.numpy(), rtol=1e-12, atol=1e-12)
    if shared != "A":
        assert np.all(dA[1] == 0)                       # no rows, no gradient


def test_grouped_quant_is_per_expert():
    rng = np.random.default_rng(10)
    E, N, K, r = 2, 8, 64, 2
    w = workloads.normal_bf16(rng, (E * N, K), 0.02).reshape(E, N, K)
    w[1] *= 0                                           # expert 1: zero base weight
    A = rng.standard_normal((r, K)).astype(np.float32) * np.float32(0.01)
    B = rng.standard_normal((E, N, r)).astype(np.float32)
    xh = oracle.lora_quant_grouped(w, B, A, 1.0, "nvfp4")
    for e in range(E):   # each expert's tensor scale comes from its own merged weight
        assert np.array_equal(xh[e], oracle.lora_quant(w[e], B[e], A, 1.0, "nvfp4")["xhat"])
