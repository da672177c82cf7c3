"""Pins for the oracle's quantizers (NVFP4, MXFP4, Q4_K) and Q4_K packing.

The checks come from what the formats fix, not from re-running the oracle's own steps:
exact representability of on-grid inputs, idempotence Q(Q^-1(Q(x))) = Q(x) (NVFP4 with
normal block scales, MXFP4 always), brute-force nearest-code and nearest-scale searches,
error bounds, the paper's effective bits per weight (Tab. formats), a hand-worked Q4_K
scale field, and the decode equations (Eqs. nvfp4-dequant, mxfp4-dequant, q4k-dequant)
applied to the stored codes and scales.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from tests.helpers import (E2M1_MAGS, bf16_to_f64, block_view, f64_to_bf16_exact,
                           unpack_nibbles, wide_range_bf16)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
E4M3_TAB = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(
    torch.float64).numpy()
E8M0_TAB = torch.arange(256, dtype=torch.uint8).view(torch.float8_e8m0fnu).to(
    torch.float64).numpy()


def _nearest_e2m1(v):
    """Brute-force nearest E2M1 magnitude code, ties to even, saturating above 6."""
    d = np.abs(E2M1_MAGS[None, :] - np.asarray(v, np.float64)[..., None])
    out = np.argmin(d, axis=-1)
    dmin = d.min(axis=-1)
    tie = (d == dmin[..., None]).sum(-1) > 1
    out = np.where(tie & (out % 2 == 1), out + 1, out)
    return np.where(np.asarray(v) > 6.0, 7, out)


def _signs(x):
    return (np.asarray(x) >> 15).astype(np.uint8)


# ============================================================================= MXFP4
def _mx_inputs(seed=0, R=64, K=256):
    rng = np.random.default_rng(seed)
    return wide_range_bf16(rng, (R, K), lo_exp=-135, hi_exp=124)


def test_mxfp4_scale_places_block_max_in_top_binade():
    x = _mx_inputs()
    q = oracle.mxfp4(x)
    a = np.abs(block_view(bf16_to_f64(x), 32)).max(-1)
    p = q["scales"].astype(np.int64) - 127
    ratio = a / np.exp2(p.astype(np.float64))
    nz = a > 0
    unclamped = nz & (p > -127)
    assert np.all((ratio[unclamped] >= 4) & (ratio[unclamped] < 8))
    # clamped at the smallest scale: the block max is below 4 * 2^-127
    assert np.all(ratio[nz & (p == -127)] < 8)
    assert np.all(q["scales"][~nz] == 0)
    assert np.all(q["scales"] <= 252)


def test_mxfp4_scale_brute_force_over_all_e8m0():
    # The scale is the smallest power of two that keeps the block max below 8 (so the
    # largest E2M1 value 6 is reached without going past the top binade), searched over
    # all 255 finite E8M0 values.
    x = _mx_inputs(seed=1, R=32, K=128)
    q = oracle.mxfp4(x)
    a = np.abs(block_view(bf16_to_f64(x), 32)).max(-1)
    for r in range(a.shape[0]):
        for b in range(a.shape[1]):
            if a[r, b] == 0:
                continue
            ok = [c for c in range(255) if a[r, b] / E8M0_TAB[c] < 8]
            assert q["scales"][r, b] == min(ok)


def test_mxfp4_codes_are_nearest_and_decode_matches_equation():
    x = _mx_inputs(seed=2)
    q = oracle.mxfp4(x)
    K = x.shape[1]
    codes = unpack_nibbles(q["codes"], K)
    scale = np.repeat(E8M0_TAB[q["scales"]], 32, axis=1)
    ratio = np.abs(bf16_to_f64(x)) / scale
    np.testing.assert_array_equal(codes & 7, _nearest_e2m1(ratio))
    np.testing.assert_array_equal(codes >> 3, _signs(x))
    # Eq. mxfp4-dequant: W_hat = 2^p * C
    want = np.where(codes >> 3, -1.0, 1.0) * E2M1_MAGS[codes & 7] * scale
    np.testing.assert_array_equal(q["xhat"], f64_to_bf16_exact(want))
    np.testing.assert_array_equal(oracle.mxfp4_dequant(q["codes"], q["scales"], K), q["xhat"])


def test_mxfp4_idempotent():
    for seed in range(4):
        x = _mx_inputs(seed=10 + seed)
        q1 = oracle.mxfp4(x)
        q2 = oracle.mxfp4(q1["xhat"])
        np.testing.assert_array_equal(q2["scales"], q1["scales"])
        np.testing.assert_array_equal(q2["codes"], q1["codes"])
        np.testing.assert_array_equal(q2["xhat"], q1["xhat"])


def test_mxfp4_on_grid_inputs_exact():
    rng = np.random.default_rng(3)
    R, K = 40, 128
    p = rng.integers(-127, 121, size=(R, K // 32))
    m = rng.integers(0, 8, size=(R, K))
    m.reshape(R, K // 32, 32)[:, :, 0] = rng.choice([6, 7], size=(R, K // 32))  # max 4 or 6
    s = rng.choice([-1.0, 1.0], size=(R, K))
    v = s * E2M1_MAGS[m] * np.exp2(np.repeat(p, 32, axis=1).astype(np.float64))
    x = f64_to_bf16_exact(v)
    q = oracle.mxfp4(x)
    np.testing.assert_array_equal(q["xhat"], x)
    np.testing.assert_array_equal(q["scales"], p + 127)


def test_mxfp4_clipping_region():
    # a / 2^p in [7, 8) rounds to the largest value 6 (code 7).
    base = np.full((1, 32), 0.5)
    for frac in [7.0, 7.5, 7.96875]:
        for p in [-100, -3, 0, 5, 100]:
            v = base.copy() * 2.0 ** p
            v[0, 5] = frac * 2.0 ** p
            x = f64_to_bf16_exact(v)
            q = oracle.mxfp4(x)
            assert q["scales"][0, 0] == p + 127
            c = unpack_nibbles(q["codes"], 32)[0, 5]
            assert c == 7 and bf16_to_f64(q["xhat"][0, 5]) == 6.0 * 2.0 ** p


def test_mxfp4_zero_and_nonfinite_blocks():
    x = np.zeros((2, 64), np.uint16)
    x[0, 3] = 0x8000                      # -0
    x[1, 40] = 0x7F80                     # +inf in block 1 of row 1
    x[1, 0] = 0x3F80
    q = oracle.mxfp4(x)
    assert q["scales"][0, 0] == 0 and q["scales"][0, 1] == 0
    assert unpack_nibbles(q["codes"], 64)[0, 3] == 8 and q["xhat"][0, 3] == 0x8000
    assert q["scales"][1, 1] == 0xFF and np.all(q["xhat"][1, 32:] == 0x7FC0)
    assert np.all(unpack_nibbles(q["codes"], 64)[1, 32:] == 0)
    assert q["scales"][1, 0] == 127 - 2 and q["xhat"][1, 0] == 0x3F80


def test_mxfp4_error_bound():
    x = _mx_inputs(seed=5)
    q = oracle.mxfp4(x)
    scale = np.repeat(E8M0_TAB[q["scales"]], 32, axis=1)
    r = np.abs(bf16_to_f64(x)) / scale
    err = np.abs(bf16_to_f64(q["xhat"]) - bf16_to_f64(x)) / scale
    half_gap = np.where(r <= 2, 0.25, np.where(r <= 4, 0.5, 1.0))
    clipped = r > 6
    assert np.all(err[~clipped] <= half_gap[~clipped])
    assert np.all(err[clipped] < 2.0)


# ============================================================================= NVFP4
def _nv_inputs(seed=0, R=48, K=256, spread=6):
    rng = np.random.default_rng(seed)
    return wide_range_bf16(rng, (R, K), lo_exp=-spread, hi_exp=spread)


def test_nvfp4_tensor_scale_and_block_scale_nearest():
    x = _nv_inputs()
    q = oracle.nvfp4(x)
    g = np.float32(np.abs(bf16_to_f64(x)).max())
    S = np.float32(g / np.float32(2688.0))
    assert q["S"] == S
    ab = np.abs(block_view(bf16_to_f64(x), 16)).max(-1).astype(np.float32)
    t = ab / np.float32(np.float32(6.0) * S)                 # float32 ops
    tab = E4M3_TAB[:0x7F]
    for (r, b), tv in np.ndenumerate(t):
        d = np.abs(tab - float(tv))
        best = np.flatnonzero(d == d.min())
        want = best[0] if len(best) == 1 else [c for c in best if c % 2 == 0][0]
        if tv >= 448:
            want = 0x7E
        assert q["scales"][r, b] == want


def test_nvfp4_amax_block_hits_top_of_both_grids():
    for seed in range(5):
        x = _nv_inputs(seed=seed)
        q = oracle.nvfp4(x)
        xf = np.abs(bf16_to_f64(x))
        r, k = np.unravel_index(np.argmax(xf), xf.shape)
        assert q["scales"][r, k // 16] == 0x7E
        assert unpack_nibbles(q["codes"], x.shape[1])[r, k] & 7 == 7
        assert q["xhat"][r, k] == x[r, k]


def test_nvfp4_codes_nearest_and_decode_equation():
    x = _nv_inputs(seed=7)
    K = x.shape[1]
    q = oracle.nvfp4(x)
    codes = unpack_nibbles(q["codes"], K)
    S = np.float32(q["S"])
    D = (S * np.repeat(E4M3_TAB[q["scales"]], 16, axis=1).astype(np.float32)).astype(np.float32)
    # Eq. nvfp4-dequant: W_hat = s_FP32 * s_E4M3 * C, rounded once in FP32 then to bf16
    prod = (E2M1_MAGS[codes & 7].astype(np.float32) * D).astype(np.float32)
    prod = np.where(codes >> 3, -prod, prod).astype(np.float32)
    u = prod.view(np.uint32)
    want = ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)
    np.testing.assert_array_equal(q["xhat"], want)
    np.testing.assert_array_equal(oracle.nvfp4_dequant(q["codes"], q["scales"], q["S"], K), q["xhat"])
    # nearest code to the exact ratio, except within FP32 rounding of a midpoint
    ratio = np.abs(bf16_to_f64(x)) / D.astype(np.float64)
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    near_mid = np.min(np.abs(ratio[..., None] - mids) / mids, axis=-1) < 1e-6
    ok = (codes & 7) == _nearest_e2m1(ratio)
    assert np.all(ok | near_mid)
    np.testing.assert_array_equal(codes >> 3, _signs(x))


def _normal_scale_blocks(scales):
    return ((scales >> 3) & 15) >= 1


def test_nvfp4_idempotent_on_normal_scale_blocks():
    # Re-quantizing x_hat with g recomputed from x_hat reproduces codes and scales for
    # every block whose E4M3 scale is normal; subnormal block scales are the documented
    # exception (the ratio max/6 can land on a neighbouring subnormal).
    n_checked = 0
    for seed in range(6):
        x = _nv_inputs(seed=20 + seed, spread=4)
        q1 = oracle.nvfp4(x)
        q2 = oracle.nvfp4(q1["xhat"])
        assert q2["S"] == q1["S"]
        keep = _normal_scale_blocks(q1["scales"])
        np.testing.assert_array_equal(q2["scales"][keep], q1["scales"][keep])
        c1 = block_view(unpack_nibbles(q1["codes"], x.shape[1]), 16)[keep]
        c2 = block_view(unpack_nibbles(q2["codes"], x.shape[1]), 16)[keep]
        np.testing.assert_array_equal(c2, c1)
        n_checked += keep.sum()
    assert n_checked > 1000


def test_nvfp4_on_grid_inputs_exact():
    rng = np.random.default_rng(8)
    R, K = 16, 128
    for k2 in [-20, -3, 0, 7]:
        S = 2.0 ** k2
        normal_codes = np.array([c for c in range(0x08, 0x7F)])
        sc = rng.choice(normal_codes, size=(R, K // 16))
        sc[0, 0] = 0x7E                                   # the block that carries g
        m = rng.integers(0, 8, size=(R, K))
        m.reshape(R, K // 16, 16)[:, :, 0] = 7            # block max is 6
        s = rng.choice([-1.0, 1.0], size=(R, K))
        v = s * E2M1_MAGS[m] * np.repeat(E4M3_TAB[sc], 16, axis=1) * S
        x = f64_to_bf16_exact(v)
        q = oracle.nvfp4(x)
        assert q["S"] == S
        np.testing.assert_array_equal(q["scales"], sc)
        np.testing.assert_array_equal(q["xhat"], x)


def test_nvfp4_supplied_amax_and_zero_tensor():
    x = _nv_inputs(seed=9)
    g = float(np.float32(np.abs(bf16_to_f64(x)).max()))
    a = oracle.nvfp4(x)
    b = oracle.nvfp4(x, amax_in=g)
    for key in ("codes", "scales", "xhat"):
        np.testing.assert_array_equal(a[key], b[key])
    # a larger running amax lowers every block scale and never saturates
    c = oracle.nvfp4(x, amax_in=4 * g)
    assert c["S"] == np.float32(np.float32(4 * g) / np.float32(2688))
    assert np.all(c["scales"] <= 0x7E)
    z = np.zeros((4, 32), np.uint16)
    z[1, 1] = 0x8000
    q = oracle.nvfp4(z)
    assert q["S"] == 0.0 and np.all(q["scales"] == 0)
    assert q["xhat"][1, 1] == 0x8000 and np.all(q["xhat"][0] == 0)


def test_nvfp4_error_bound():
    x = _nv_inputs(seed=11)
    q = oracle.nvfp4(x)
    S = np.float32(q["S"])
    D = (S * np.repeat(E4M3_TAB[q["scales"]], 16, axis=1).astype(np.float32)).astype(np.float64)
    r = np.abs(bf16_to_f64(x)) / D
    err = np.abs(bf16_to_f64(q["xhat"]) - bf16_to_f64(x)) / D
    half_gap = np.where(r <= 2, 0.25, np.where(r <= 4, 0.5, 1.0))
    ok = r <= 6
    # one FP32 and one bf16 rounding of the dequantized value on top of the grid error
    slack = 2.0 ** -8 * (E2M1_MAGS[unpack_nibbles(q["codes"], x.shape[1]) & 7] + 1e-30)
    assert np.all(err[ok] <= half_gap[ok] + slack[ok] + 1e-6)


# ============================================================================== Q4_K
def _q4k_inputs(seed=0, R=24, K=512):
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((R, K)) * 0.02 * np.exp(rng.normal(0, 0.5, (R, 1)))
    v[:, :32] += 0.05                        # an all-positive-ish sub-block
    v[0, 256:288] = -np.abs(v[0, 256:288])   # an all-negative sub-block
    v[1, 0:32] = 0.0                         # an all-zero sub-block
    f = v.astype(np.float32)
    u = f.view(np.uint32)
    return ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)


def test_q4k_pack_unpack_identity_exhaustive_fields():
    rng = np.random.default_rng(0)
    for t in range(64):
        ls = [(t + 7 * j) % 64 for j in range(8)]
        lm = [(63 - t + 5 * j) % 64 for j in range(8)]
        q = list(rng.integers(0, 16, 256))
        q[t] = t % 16
        d, m = int(rng.integers(0, 0x7C00)), int(rng.integers(0, 0x7C00))
        blk = oracle.q4k_pack_block(d, m, ls, lm, q)
        assert blk.shape == (144,)
        d2, m2, ls2, lm2, q2 = oracle.q4k_unpack_block(blk)
        assert (d2, m2, ls2, lm2, q2) == (d, m, ls, lm, [int(v) for v in q])


def test_q4k_scale_field_matches_hand_worked_layout():
    lines = [l.split() for l in open(os.path.join(GOLDEN, "q4k_scale_bytes.txt"))
             if l.strip() and not l.startswith("#")]
    ls = [int(v) for v in lines[0]]
    lm = [int(v) for v in lines[1]]
    want = bytes(int(v, 16) for v in lines[2])
    q = [(i * 7) % 16 for i in range(256)]
    blk = oracle.q4k_pack_block(0x1234, 0xABCD, ls, lm, q)
    assert bytes(blk[0:4]) == bytes([0x34, 0x12, 0xCD, 0xAB])
    assert bytes(blk[4:16]) == want
    # code bytes: byte 32c+l holds q[64c+l] (low nibble) and q[64c+32+l] (high nibble)
    for c in range(4):
        for l in range(32):
            assert blk[16 + 32 * c + l] == q[64 * c + l] | (q[64 * c + 32 + l] << 4)


def _handworked_q4k_block():
    """The hand-worked super-block of tests/golden/q4k_block_handworked.txt: input bf16 bits,
    listed FP16 d / dmin, 6-bit scales and mins, and the expected 144 bytes."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "q4k_block_handworked.txt"))
            if l.strip() and not l.startswith("#")]
    vals = rows[:8]
    x = np.zeros((1, 256), np.uint16)
    for j, line in enumerate(vals):
        assert len(line) == 32
        for i, t in enumerate(line):
            v = np.float32(int(t) * 2.0 ** -13)
            u = int(np.array([v]).view(np.uint32)[0])
            assert u & 0xFFFF == 0, "fixture value not exact in bf16"
            x[0, 32 * j + i] = (u >> 16) | (0x8000 if t.startswith("-") else 0)
    dh, mh = (int(v, 16) for v in rows[8])
    ls = [int(v) for v in rows[9]]
    lm = [int(v) for v in rows[10]]
    blk = bytes(int(v, 16) for r in rows[11:] for v in r)
    assert len(blk) == 144
    return x, dh, mh, ls, lm, blk


def test_q4k_handworked_block_bytes():
    # Every field and byte of this block was worked out by hand from the reading (nearest 6-bit
    # scale and min, ties to even) and the public block layout; a truncated or half-up 6-bit
    # rounding, a swapped nibble or sub-block, or a misplaced scale bit changes the bytes.
    x, dh, mh, ls, lm, blk = _handworked_q4k_block()
    q = oracle.q4k(x)
    got = bytes(q["packed"].reshape(-1))
    assert got[0:4] == blk[0:4], "d / dmin"
    assert got[4:16] == blk[4:16], "scale bytes"
    assert got[16:] == blk[16:], "code bytes"
    d2, m2, ls2, lm2, q2 = oracle.q4k_unpack_block(q["packed"][0, 0])
    assert (d2, m2, ls2, lm2) == (dh, mh, ls, lm)
    assert q2 == [(i % 32 + i // 32) % 16 for i in range(256)]
    # x_hat follows Eq. q4k-dequant from the listed fields (d = dmin = 2^-10 here, so every
    # t1 q - t2 is a multiple of 2^-10 below 1024 of them: exact in FP32, rounded once to bf16)
    xh = bf16_to_f64(q["xhat"][0])
    for i in range(256):
        j = i // 32
        want = np.float32((ls[j] * q2[i] - lm[j]) * 2.0 ** -10)
        u = int(np.array([want]).view(np.uint32)[0])
        u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
        assert q["xhat"][0, i] == u, (i, xh[i], float(want))


def test_q4k_dequant_of_packed_bytes_reproduces_xhat():
    x = _q4k_inputs(seed=1)
    q = oracle.q4k(x)
    np.testing.assert_array_equal(oracle.q4k_dequant(q["packed"], x.shape[1]), q["xhat"])


def _q4k_fields(packed):
    R, NB, _ = packed.shape
    d = np.zeros((R, NB)); m = np.zeros((R, NB))
    ls = np.zeros((R, NB, 8), int); lm = np.zeros((R, NB, 8), int); qq = np.zeros((R, NB, 256), int)
    for r in range(R):
        for b in range(NB):
            dh, mh, a, bb, c = oracle.q4k_unpack_block(packed[r, b])
            d[r, b] = float(np.array([dh], np.uint16).view(np.float16)[0])
            m[r, b] = float(np.array([mh], np.uint16).view(np.float16)[0])
            ls[r, b] = a; lm[r, b] = bb; qq[r, b] = c
    return d, m, ls, lm, qq


def test_q4k_superblock_scales_match_numpy_float16():
    x = _q4k_inputs(seed=2)
    q = oracle.q4k(x)
    d, m, ls, lm, qq = _q4k_fields(q["packed"])
    xs = bf16_to_f64(x).astype(np.float32).reshape(x.shape[0], -1, 8, 32)
    lo = np.minimum(xs.min(-1), np.float32(0))
    hi = xs.max(-1)
    a = ((hi - lo).astype(np.float32) / np.float32(15)).astype(np.float32)
    mu = (-lo).astype(np.float32)
    want_d = (a.max(-1) / np.float32(63)).astype(np.float32).astype(np.float16).astype(np.float64)
    want_m = (mu.max(-1) / np.float32(63)).astype(np.float32).astype(np.float16).astype(np.float64)
    np.testing.assert_array_equal(d, want_d)
    np.testing.assert_array_equal(m, want_m)
    # the 6-bit scale reproduces each sub-block's step to within half a step of d
    unclamped = ls < 63
    assert np.all(np.abs(d[..., None] * ls - a)[unclamped] <= d[..., None].repeat(8, -1)[unclamped] / 2 * (1 + 1e-6))
    # and the 6-bit min reproduces each offset to within half a step of dmin (nearest, not
    # truncated: about half of these offsets sit more than half a step above a multiple)
    unclamped = (lm < 63) & (m[..., None] > 0)
    mm = m[..., None].repeat(8, -1)
    assert np.all(np.abs(mm * lm - mu)[unclamped] <= mm[unclamped] / 2 * (1 + 1e-6))
    frac = (mu / np.where(mm > 0, mm, 1))[unclamped] % 1.0
    assert np.count_nonzero(frac > 0.55) > 10    # the check above covers round-up cases


def test_q4k_codes_are_nearest_grid_points():
    x = _q4k_inputs(seed=3)
    q = oracle.q4k(x)
    d, m, ls, lm, qq = _q4k_fields(q["packed"])
    R, NB = d.shape
    t1 = (d[..., None] * ls).astype(np.float32).astype(np.float64)
    t2 = (m[..., None] * lm).astype(np.float32).astype(np.float64)
    xv = bf16_to_f64(x).reshape(R, NB, 8, 32)
    grid = t1[..., None, None] * np.arange(16) - t2[..., None, None]        # [R,NB,8,1,16]
    dist = np.abs(xv[..., None] - grid)
    best = dist.min(-1)
    chosen = np.take_along_axis(dist, qq.reshape(R, NB, 8, 32)[..., None], -1)[..., 0]
    ok = (chosen <= best * (1 + 1e-5) + 1e-12) | (t1[..., None] == 0)
    assert np.all(ok)
    # Eq. q4k-dequant applied to the stored fields gives x_hat (up to the final rounding)
    deq = t1[..., None] * qq.reshape(R, NB, 8, 32) - t2[..., None]
    np.testing.assert_allclose(bf16_to_f64(q["xhat"]).reshape(deq.shape), deq, rtol=2 ** -8, atol=1e-30)


def test_q4k_is_not_always_idempotent_but_stays_on_its_grid():
    # Documented: Q4_K min-max re-quantization may pick a different grid, so only a weaker
    # property is pinned -- x_hat re-quantizes to values within one step of itself.
    x = _q4k_inputs(seed=4)
    q1 = oracle.q4k(x)
    q2 = oracle.q4k(q1["xhat"])
    d, m, ls, lm, qq = _q4k_fields(q1["packed"])
    step = np.repeat((d[..., None] * ls).reshape(x.shape[0], -1), 32, axis=1)
    diff = np.abs(bf16_to_f64(q2["xhat"]) - bf16_to_f64(q1["xhat"]))
    assert np.all(diff <= step * 1.01 + 1e-30)


# ====================================================================== Tab. formats
def test_effective_bits_per_weight_match_paper_table():
    rows = {}
    for line in open(os.path.join(GOLDEN, "format_table.txt")):
        if line.strip() and not line.startswith("#"):
            f, blk, sb, sym, bits = line.split()
            rows[f] = (int(blk), int(sb), int(sym), float(bits))
    R, K = 4, 512
    x = _q4k_inputs(seed=0, R=R, K=K)
    nv = oracle.nvfp4(x)
    mx = oracle.mxfp4(x)
    qk = oracle.q4k(x)
    n = R * K
    assert 8 * (nv["codes"].nbytes + nv["scales"].nbytes) / n == rows["nvfp4"][3]
    assert 8 * (mx["codes"].nbytes + mx["scales"].nbytes) / n == rows["mxfp4"][3]
    assert 8 * qk["packed"].nbytes / n == rows["q4k"][3]
    assert K // nv["scales"].shape[1] == rows["nvfp4"][0]
    assert K // mx["scales"].shape[1] == rows["mxfp4"][0]


def test_q4k_signed_zeros_count_as_positive_zero():
    # Reading of Eq. q4k: codes are unsigned, so the sign of a zero input carries no
    # information; -0 and +0 inputs give the same packed block and x_hat.
    x = _q4k_inputs(seed=6, R=4, K=256)
    x[:, :32] = 0x0000
    x[:, 40:60] = 0x0000
    y = x.copy()
    y[:, :32] = 0x8000
    y[:, 40:60:2] = 0x8000
    a, b = oracle.q4k(x), oracle.q4k(y)
    np.testing.assert_array_equal(a["packed"], b["packed"])
    np.testing.assert_array_equal(a["xhat"], b["xhat"])
    d, m, ls, lm, qq = _q4k_fields(a["packed"])
    assert np.all(np.signbit(m) == False)
