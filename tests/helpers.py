"""Test-side utilities: tolerance metric, bf16 decoding, edge-case tensor builders.

Nothing here implements the method: it builds inputs and measures errors.
"""
import math

import numpy as np

E2M1_MAGS = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def bf16_to_f64(h):
    return (np.asarray(h).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_exact(v):
    """bf16 bits of values that bfloat16 represents exactly (asserts exactness)."""
    f = np.asarray(v, np.float64).astype(np.float32)
    assert np.all(f.astype(np.float64) == np.asarray(v, np.float64))
    u = f.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0)
    return (u >> 16).astype(np.uint16)


def rel_err(y, ref):
    """Per-entry error |y - r| / max(|r|, 1e-3 * rms(r)); returns (max, mean)."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    rms = math.sqrt(float(np.mean(ref * ref))) if ref.size else 0.0
    floor = max(1e-3 * rms, 1e-30)
    e = np.abs(y - ref) / np.maximum(np.abs(ref), floor)
    return float(e.max()) if e.size else 0.0, float(e.mean()) if e.size else 0.0


MAX_REL = 2e-2
MEAN_REL = 2e-3


def assert_close(y, ref, what=""):
    mx, mean = rel_err(y, ref)
    assert mx <= MAX_REL and mean <= MEAN_REL, f"{what}: max rel {mx:.3e}, mean rel {mean:.3e}"
    return mx, mean


def wide_range_bf16(rng, shape, lo_exp=-130, hi_exp=120, zero_frac=0.02, neg_zero_frac=0.01):
    """bf16 tensor whose rows are blocks of very different magnitudes, with +-0 sprinkled in."""
    R, K = shape
    mant = rng.standard_normal((R, K))
    row_exp = rng.integers(lo_exp, hi_exp, size=(R, 1))
    v = mant * np.exp2(row_exp.astype(np.float64))
    v = np.where(rng.random((R, K)) < zero_frac, 0.0, v)
    v = np.where(rng.random((R, K)) < neg_zero_frac, -0.0, v)
    f = v.astype(np.float32)
    u = f.view(np.uint32)
    return ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)


def block_view(a, block):
    R, K = a.shape
    return a.reshape(R, K // block, block)


def unpack_nibbles(codes, K):
    codes = np.asarray(codes)
    out = np.empty((codes.shape[0], K), np.uint8)
    out[:, 0::2] = codes & 15
    out[:, 1::2] = codes >> 4
    return out


# ------------------------------------------------------------------ GPU marshalling helpers
def to_dev(a, dev="cuda"):
    """Upload a numpy array (raw bits for bf16) to the GPU without changing its bytes."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(dev)


def from_dev(t, dtype=None):
    arr = t.detach().cpu().numpy()
    if arr.dtype == np.int16:
        arr = arr.view(np.uint16)
    return arr if dtype is None else arr.astype(dtype)


def empty_bf16(shape, dev="cuda"):
    import torch
    return torch.empty(shape, dtype=torch.int16, device=dev)
