"""Pins of the QAD distillation-loss oracle (Sec. 3.3, Eq. qad-objective): closed forms and
invariances of the forward KL, torch autograd for the gradient, brute force for top-1."""
import math

import numpy as np
import pytest

import oracle
import workloads
from tests.helpers import f64_to_bf16_exact


def _bf(a):
    return workloads.to_bf16(np.asarray(a, np.float32))


def test_identical_distributions_have_zero_loss_and_gradient():
    z = _bf(np.random.default_rng(0).standard_normal((4, 64)) * 3)
    loss, kl, grad, agree = oracle.qad_kl(z, z)
    assert abs(loss) < 1e-15 and np.all(np.abs(kl) < 1e-15) and np.all(grad == 0)
    assert np.all(agree == 1)


def test_two_token_vocabulary_closed_form():
    # softmax of (a, b) is a Bernoulli(sigma(a - b)): KL = p log(p/q) + (1-p) log((1-p)/(1-q))
    zt = f64_to_bf16_exact([[2.0, 0.0], [0.5, 1.5]])
    zs = f64_to_bf16_exact([[0.0, 1.0], [1.0, 1.0]])
    loss, kl, grad, _ = oracle.qad_kl(zt, zs)
    sig = lambda x: 1 / (1 + math.exp(-x))
    for i, (a, b, c, d) in enumerate([(2, 0, 0, 1), (0.5, 1.5, 1, 1)]):
        p, q = sig(a - b), sig(c - d)
        want = p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))
        assert abs(kl[i] - want) < 1e-14
        assert abs(grad[i, 0] - (q - p) / 2) < 1e-15
    assert abs(loss - kl.mean()) < 1e-15


def test_uniform_student_gives_log_v_minus_entropy():
    rng = np.random.default_rng(1)
    V = 100
    zt = _bf(rng.standard_normal((3, V)))
    zs = np.zeros((3, V), np.uint16)
    _, kl, _, _ = oracle.qad_kl(zt, zs)
    t = workloads.from_bf16(zt).astype(np.float64)
    p = np.exp(t - t.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    H = -(p * np.log(p)).sum(1)
    assert np.allclose(kl, math.log(V) - H, rtol=0, atol=1e-13)


def test_shift_invariance_and_nonnegativity():
    rng = np.random.default_rng(2)
    zt = rng.integers(-20, 20, size=(5, 48)).astype(np.float64) / 4
    zs = rng.integers(-20, 20, size=(5, 48)).astype(np.float64) / 4
    _, kl1, g1, _ = oracle.qad_kl(f64_to_bf16_exact(zt), f64_to_bf16_exact(zs))
    _, kl2, g2, _ = oracle.qad_kl(f64_to_bf16_exact(zt + 8), f64_to_bf16_exact(zs - 16))
    assert np.allclose(kl1, kl2, atol=1e-12) and np.allclose(g1, g2, atol=1e-15)
    assert np.all(kl1 > 0)
    assert np.allclose(g1.sum(axis=1), 0, atol=1e-15)      # gradient of a softmax sums to 0


def test_gradient_matches_torch_autograd():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    zt = _bf(rng.standard_normal((6, 40)) * 2)
    zs = _bf(rng.standard_normal((6, 40)) * 2)
    loss, kl, grad, _ = oracle.qad_kl(zt, zs)
    t = torch.tensor(workloads.from_bf16(zt), dtype=torch.float64)
    s = torch.tensor(workloads.from_bf16(zs), dtype=torch.float64, requires_grad=True)
    ref = torch.nn.functional.kl_div(torch.log_softmax(s, 1), torch.log_softmax(t, 1),
                                     log_target=True, reduction="batchmean")
    ref.backward()
    assert abs(loss - ref.item()) < 1e-13
    assert np.allclose(grad, s.grad.numpy(), atol=1e-15)


def test_top1_agreement_first_index_on_ties():
    zt = f64_to_bf16_exact([[1, 3, 3, 0], [5, 1, 1, 5], [0, 0, 0, 0]])
    zs = f64_to_bf16_exact([[1, 3, 2, 3], [1, 5, 1, 5], [0, 0, 0, 0]])
    _, _, _, agree = oracle.qad_kl(zt, zs)
    assert list(agree) == [1, 0, 1]        # argmax: (1,1), (0,1), (0,0)
