"""Pins of the Q4_K MSE-search oracle (the PTQ objective ||W - W_q||^2 of Sec. 4).  The search
is this library's own design, so the pins check what the objective fixes: never worse than the
min-max quantizer per super-block (FP64 errors of the decoded blocks), clearly better on
average, least-squares optimality of the refit, nearest codes for the chosen scales, exact
recovery of on-grid data, and that the packed blocks decode to x_hat."""
import numpy as np
import pytest

import oracle
import workloads
from tests.helpers import bf16_to_f64


def _err_per_block(x, packed):
    K = x.shape[1]
    dec = bf16_to_f64(oracle.q4k_dequant(packed, K))
    # the engine decodes t1 C - t2; x_hat rounds it to bf16, so use the exact decode: FP64 of
    # the bf16 x_hat differs from t1 C - t2 by < 2^-9 relative, far below the gaps compared
    e = (bf16_to_f64(x) - dec) ** 2
    return e.reshape(x.shape[0], K // 256, 256).sum(-1)


@pytest.mark.parametrize("kind", ["normal", "heavy", "wide", "skewed"])
def test_never_worse_than_min_max(kind):
    rng = np.random.default_rng({"normal": 1, "heavy": 2, "wide": 3, "skewed": 4}[kind])
    R, K = 24, 1024
    if kind == "normal":
        x = workloads.normal_bf16(rng, (R, K), 0.02)
    elif kind == "heavy":
        x = workloads.to_bf16((rng.standard_t(3, size=(R, K)) * 0.02).astype(np.float32))
    elif kind == "wide":
        x = workloads.normal_bf16(rng, (R, K), 1.0, row_scale=np.exp(rng.normal(0, 3, R)))
    else:
        x = workloads.to_bf16((np.abs(rng.standard_normal((R, K))) * 0.05 - 0.01).astype(np.float32))
    m = oracle.q4k_mse(x)
    b = oracle.q4k(x)
    em, eb = _err_per_block(x, m["packed"]), _err_per_block(x, b["packed"])
    assert np.all(em <= eb * (1 + 1e-5) + 1e-30)
    assert np.array_equal(oracle.q4k_dequant(m["packed"], K), m["xhat"])
    if kind in ("normal", "heavy"):
        assert em.sum() < 0.9 * eb.sum()          # the search pays off on bell-shaped weights


def test_refit_is_the_least_squares_optimum_for_its_codes():
    rng = np.random.default_rng(3)
    for _ in range(50):
        x = (rng.standard_normal(32) * 0.03).astype(np.float32)
        a, mu, q = oracle.q4k_mse_subblock(x)
        A = np.stack([q.astype(np.float64), -np.ones(32)], axis=1)
        sol, *_ = np.linalg.lstsq(A, x.astype(np.float64), rcond=None)
        if sol[1] >= 0 and sol[0] > 0:               # unconstrained optimum is feasible
            assert abs(a - sol[0]) <= 1e-4 * abs(sol[0])
            assert abs(mu - sol[1]) <= 1e-4 * max(abs(sol[1]), abs(sol[0]))
        # the chosen (a, mu) with its codes beats the min-max step with its own codes
        lo, hi = min(0.0, float(x.min())), float(x.max())
        a0, mu0 = (hi - lo) / 15, -lo
        q0 = np.clip(np.rint((x + mu0) / a0), 0, 15)
        e0 = ((x - (a0 * q0 - mu0)) ** 2).sum()
        e1 = ((x - (a * q - mu)) ** 2).sum()
        assert e1 <= e0 * (1 + 1e-5)


def test_codes_are_nearest_for_the_chosen_scales():
    rng = np.random.default_rng(4)
    x = workloads.normal_bf16(rng, (8, 512), 0.02)
    m = oracle.q4k_mse(x)
    for r in range(8):
        for sb in range(2):
            d, dmin, ls, lm, q = oracle.q4k_unpack_block(m["packed"][r, sb])
            d, dmin = oracle.f16_to_f32(d), oracle.f16_to_f32(dmin)
            xv = bf16_to_f64(x[r, 256 * sb:256 * (sb + 1)])
            for j in range(8):
                t1, t2 = d * ls[j], dmin * lm[j]
                grid = t1 * np.arange(16) - t2
                for i in range(32):
                    dist = np.abs(xv[32 * j + i] - grid)
                    assert dist[q[32 * j + i]] <= dist.min() * (1 + 1e-6) + 1e-12


def test_on_grid_data_is_recovered_exactly():
    # every sub-block holds the 16 levels t1 C - t2 of one grid twice: the searched blocks
    # decode to the input exactly (after the bf16 rounding of x_hat)
    d, dmin = 2.0 ** -6, 2.0 ** -8
    rng = np.random.default_rng(5)
    vals = []
    for j in range(8):
        t1, t2 = d * 1.0, dmin * 2.0
        levels = t1 * np.arange(16) - t2
        vals.append(rng.permutation(np.concatenate([levels, levels])))
    x = workloads.to_bf16(np.concatenate(vals).astype(np.float32))[None, :]
    m = oracle.q4k_mse(x)
    assert np.array_equal(m["xhat"], x)
