"""Pins for the oracle's scalar codecs (E2M1, E4M3, E8M0, bfloat16, float16).

Each test checks the oracle against something other than itself: the value set the
paper prints (Eq. e2m1-values), the rounding intervals of round-to-nearest-even written
out as thresholds, PyTorch's own float8 / bfloat16 casts and numpy's float16 cast.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load_values(name):
    vals = []
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if line and not line.startswith("#"):
            vals.append(float(line))
    return vals


# ----------------------------------------------------------------------------- E2M1
def test_e2m1_value_set_matches_paper():
    paper = sorted(set(_load_values("e2m1_values.txt")))
    got = sorted(set(oracle.e2m1_value(c) for c in range(16)))
    assert got == paper
    assert len(paper) == 15
    # 16 codes: +0 and -0 are distinct codes with the sign in bit 3
    assert math.copysign(1.0, oracle.e2m1_value(8)) == -1.0
    assert oracle.e2m1_value(0) == 0.0 and math.copysign(1.0, oracle.e2m1_value(0)) == 1.0


def test_e2m1_roundtrip_all_codes():
    for m in range(8):
        assert oracle.e2m1_encode(abs(oracle.e2m1_value(m))) == m


# Round-to-nearest-even intervals for the E2M1 magnitudes, written as thresholds: each
# midpoint between neighbours goes to the neighbour whose code is even.
_INTERVALS = [  # (lo, lo_inclusive, hi, hi_inclusive, code)
    (0.0, True, 0.25, True, 0),
    (0.25, False, 0.75, False, 1),
    (0.75, True, 1.25, True, 2),
    (1.25, False, 1.75, False, 3),
    (1.75, True, 2.5, True, 4),
    (2.5, False, 3.5, False, 5),
    (3.5, True, 5.0, True, 6),
    (5.0, False, math.inf, True, 7),
]


def _interval_code(v):
    for lo, loi, hi, hii, c in _INTERVALS:
        if (v > lo or (loi and v == lo)) and (v < hi or (hii and v == hi)):
            return c
    raise AssertionError(v)


def test_e2m1_encode_thresholds():
    probes = [0.0, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.0, 6.0001, 1e30, math.inf]
    for mid in [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]:
        probes += [np.nextafter(mid, 0.0), np.nextafter(mid, 10.0)]
    rng = np.random.default_rng(1)
    probes += list(rng.uniform(0, 8, 2000)) + list(np.float32(rng.uniform(0, 1, 500)))
    for v in probes:
        assert oracle.e2m1_encode(float(v)) == _interval_code(float(v)), v
    assert oracle.e2m1_encode(6.0001) == 7 and oracle.e2m1_encode(1e30) == 7


# ----------------------------------------------------------------------------- E4M3
def _torch_e4m3_table():
    return torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_e4m3_decode_matches_torch_all_codes():
    tab = _torch_e4m3_table()
    for c in range(256):
        ours = oracle.e4m3_decode(c)
        if c in (0x7F, 0xFF):
            assert math.isnan(ours) and math.isnan(tab[c])
        else:
            assert ours == tab[c], hex(c)
    assert oracle.e4m3_decode(0x7E) == 448.0


def test_e4m3_roundtrip_all_finite_codes():
    for c in range(0x7F):
        assert oracle.e4m3_encode(oracle.e4m3_decode(c)) == c


def test_e4m3_encode_matches_torch_cast_below_464():
    tab = _torch_e4m3_table()[:0x7F]
    mids = (tab[:-1] + tab[1:]) / 2
    rng = np.random.default_rng(2)
    vals = np.concatenate([tab, mids, np.nextafter(mids, 0), np.nextafter(mids, 1e9),
                           rng.uniform(0, 464, 4000), np.exp(rng.uniform(-12, 6, 4000)),
                           [464.0, 460.0, 448.5]]).astype(np.float32)
    vals = vals[(vals >= 0) & (vals <= 464)]
    ref = torch.from_numpy(vals).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    ours = np.array([oracle.e4m3_encode(float(v)) for v in vals])
    np.testing.assert_array_equal(ours, ref)


def test_e4m3_encode_saturates_instead_of_nan():
    # Documented divergence: PyTorch's cast gives NaN above 464, the E4M3 block scale of
    # NVFP4 saturates at the largest finite value 448.
    for t in [464.0001, 480.0, 1000.0, 1e30, math.inf]:
        assert oracle.e4m3_encode(t) == 0x7E


def test_e4m3_encode_is_nearest_by_brute_force():
    tab = _torch_e4m3_table()[:0x7F]
    rng = np.random.default_rng(3)
    for t in np.exp(rng.uniform(-10, 6.2, 3000)):
        t = float(np.float32(t))
        d = np.abs(tab - t)
        best = np.flatnonzero(d == d.min())
        want = best[0] if len(best) == 1 else [b for b in best if b % 2 == 0][0]
        if t >= 448:
            want = 0x7E
        assert oracle.e4m3_encode(t) == want, t


# ----------------------------------------------------------------------------- E8M0
def test_e8m0_all_codes_match_torch():
    tab = torch.arange(256, dtype=torch.uint8).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
    for c in range(256):
        ours = oracle.e8m0_decode(c)
        if c == 0xFF:
            assert math.isnan(ours) and math.isnan(tab[c])
        else:
            assert ours == tab[c], c
            m, e = math.frexp(ours)
            assert m == 0.5  # an exact power of two (Eq. mxfp4-dequant)


# ------------------------------------------------------------------------ bf16 / fp16
def _special_f32():
    rng = np.random.default_rng(4)
    bits = np.concatenate([
        rng.integers(0, 2**32, 20000, dtype=np.uint64),
        # exact ties: low 16 bits = 0x8000 with even and odd kept parts
        (rng.integers(0, 2**16, 4000, dtype=np.uint64) << 16) | 0x8000,
        np.arange(0, 70000, dtype=np.uint64),  # subnormals near zero
        np.array([0x7F7F7FFF, 0x7F7F8000, 0x7F7FFFFF, 0x7F800000, 0xFF800000, 0x80000000,
                  0x00008000, 0x00018000, 0x3F808000, 0x3F818000], np.uint64),
    ]).astype(np.uint32)
    f = bits.view(np.float32)
    return f[~np.isnan(f)]


def test_bf16_rounding_matches_torch():
    f = _special_f32()
    ref = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    ours = np.array([oracle.bf16_from_f32(float(v)) for v in f], np.uint16)
    np.testing.assert_array_equal(ours, ref)
    assert oracle.bf16_from_f32(float("nan")) == 0x7FC0


def test_bf16_decode_is_upper_half():
    rng = np.random.default_rng(5)
    for h in rng.integers(0, 2**16, 3000):
        h = int(h)
        want = np.array([h << 16], np.uint32).view(np.float32)[0]
        got = oracle.bf16_to_f32(h)
        assert (math.isnan(got) and math.isnan(want)) or got == want


def test_fp16_rounding_matches_numpy_below_overflow():
    f = _special_f32()
    f = f[np.abs(f) < 65520.0]
    ref = f.astype(np.float16).view(np.uint16)
    ours = np.array([oracle.f16_from_f32(float(v)) for v in f], np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_fp16_saturates_and_decodes():
    assert oracle.f16_from_f32(65520.0) == 0x7BFF
    assert oracle.f16_from_f32(1e30) == 0x7BFF
    for h in range(0, 0x7C00, 7):
        assert oracle.f16_to_f32(h) == float(np.array([h], np.uint16).view(np.float16)[0])
