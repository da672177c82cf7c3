"""Seeded synthetic inputs shaped like the LLM linear layers that simulated quantization runs in.

This module holds input generation only: random draws, scaling of the draws into the
distributions below, and the float32 -> bfloat16 (round to nearest even) storage
conversion.  It contains none of the quantization or GEMM arithmetic, so it can serve
both the GPU path and the CPU oracle.

The paper trains on real checkpoints and datasets; these stand in for them with the
tensor shapes and value distributions of the layers it quantizes (Sec. 3.2, Sec. 4.1):

* ``single_linear``     NVFP4 weight-only single layer: W [512,512] ~ N(0, 0.02),
                        X [256,512] ~ N(0,1) with 4 distinct columns scaled x50, dY ~ N(0,1).
* ``mlp_up``            MXFP4 W4A4 8B-class MLP up-projection: X [8192,4096] ~ N(0,1) with
                        round(1% of 4096) = 41 distinct channels x20, W [14336,4096] ~ N(0,0.02),
                        dY [8192,14336] ~ N(0,1).
* ``dense_layer``       9B-class transformer layer at 32K tokens, NVFP4 weight-only: inputs
                        x = z * |tau_c|, z ~ N(0,1), tau_c ~ Student-t(3) per channel; weights
                        ~ N(0,0.02): QKV [6144,4096] (4096+1024+1024, grouped-query), O [4096,4096],
                        gate/up [2*12288,4096], down [4096,12288]; dY ~ N(0,1).
* ``moe_experts``       128 experts, top-8 routing of 32768 tokens with Zipf(1.1) expert
                        popularity (Gumbel-top-8 sampling), hidden 3072, expert intermediate
                        1536: W_gu [128][3072][3072], W_d [128][3072][1536] ~ N(0,0.02).
* ``q4k_weight``        W [14336,4096] ~ N(0,0.02) x per-row log-normal(0,0.5), X [4096,4096] ~ N(0,1).
* ``qad_logits``        Teacher / student logits for the QAD loss (Sec. 3.3, Eq. qad-objective):
                        L tokens over a vocabulary V (the paper's Qwen3 models: 151936),
                        teacher z_T = 2 N(0,1) plus +6..+14 on 1..4 "preferred" tokens per row
                        (peaked next-token distributions), student z_S = z_T + N(0, 0.5^2)
                        (a quantization-perturbed copy: KL per token ~0.1, as in the paper's
                        evaluation KL), both rounded to bf16.
* ``lora_factors``      LoRA-QAD adapters of rank r on an [N, K] weight (Sec. 3.3; the paper's
                        ranks are 4, 16, 64, 256 and its memory table uses 16): FP32
                        A [r, K] ~ N(0, 1/K) and B [N, r] ~ N(0, (0.001 sqrt(K/r))^2), so a
                        trained-like update s B A with s = alpha / r = 2 has std 0.002, a tenth
                        of the N(0, 0.02) base weight (enough to move many quantization codes).

Draws use ``numpy.random.default_rng(seed)`` in float32, in the order listed.  Large
tensors are drawn in row chunks from the same generator, so the bytes depend only on the
seed and the shape.  ``scale`` divides the token count (rows) for test-sized variants.
"""
from __future__ import annotations

import numpy as np



def to_bf16(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bits, round to nearest even (inputs here are always finite)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def from_bf16(h: np.ndarray) -> np.ndarray:
    return (h.astype(np.uint32) << 16).view(np.float32)


def normal_bf16(rng: np.random.Generator, shape, std: float = 1.0,
                row_scale: np.ndarray | None = None,
                col_scale: np.ndarray | None = None) -> np.ndarray:
    """N(0, std^2) draws (optionally times per-row / per-column factors) stored as bf16."""
    R, C = shape
    out = np.empty((R, C), np.uint16)
    step = max(1, (1 << 24) // max(C, 1))
    for r0 in range(0, R, step):
        r1 = min(R, r0 + step)
        z = rng.standard_normal((r1 - r0, C), dtype=np.float32)
        if std != 1.0:
            z *= np.float32(std)
        if row_scale is not None:
            z *= row_scale[r0:r1, None].astype(np.float32)
        if col_scale is not None:
            z *= col_scale[None, :].astype(np.float32)
        out[r0:r1] = to_bf16(z)
    return out


def single_linear(seed: int = 0, scale: int = 1) -> dict:
    rng = np.random.default_rng(seed)
    M, N, K = 256 // scale, 512, 512
    W = normal_bf16(rng, (N, K), 0.02)
    cols = rng.choice(K, 4, replace=False)
    colscale = np.ones(K, np.float32)
    colscale[cols] = 50.0
    X = normal_bf16(rng, (M, K), 1.0, col_scale=colscale)
    dY = normal_bf16(rng, (M, N), 1.0)
    return {"X": X, "W": W, "dY": dY, "M": M, "N": N, "K": K, "wfmt": "nvfp4", "afmt": "none",
            "outlier_cols": np.sort(cols)}


def mlp_up(seed: int = 0, scale: int = 1, n_scale: int = 1, k_scale: int = 1) -> dict:
    rng = np.random.default_rng(seed)
    M, N, K = 8192 // scale, 14336 // n_scale, 4096 // k_scale
    nout = int(round(0.01 * K))
    cols = rng.choice(K, nout, replace=False)
    colscale = np.ones(K, np.float32)
    colscale[cols] = 20.0
    X = normal_bf16(rng, (M, K), 1.0, col_scale=colscale)
    W = normal_bf16(rng, (N, K), 0.02)
    dY = normal_bf16(rng, (M, N), 1.0)
    return {"X": X, "W": W, "dY": dY, "M": M, "N": N, "K": K, "wfmt": "mxfp4", "afmt": "mxfp4"}


def q4k_weight(seed: int = 0, scale: int = 1, n_scale: int = 1) -> dict:
    rng = np.random.default_rng(seed)
    N, K, M = 14336 // n_scale, 4096, 4096 // scale
    rows = np.exp(rng.normal(0.0, 0.5, size=N)).astype(np.float32)
    W = normal_bf16(rng, (N, K), 0.02, row_scale=rows)
    X = normal_bf16(rng, (M, K), 1.0)
    dY = normal_bf16(rng, (M, N), 1.0)
    return {"X": X, "W": W, "dY": dY, "M": M, "N": N, "K": K, "wfmt": "q4k", "afmt": "none"}


DENSE_LINEARS = (("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 24576, 4096),
                 ("down", 4096, 12288))


def dense_layer(seed: int = 0, scale: int = 1, width_scale: int = 1) -> dict:
    """One transformer layer's four fused linears (seven projections)."""
    rng = np.random.default_rng(seed)
    T = 32768 // scale
    out = {"T": T, "wfmt": "nvfp4", "afmt": "none", "linears": []}
    for name, N, K in DENSE_LINEARS:
        N //= width_scale
        K //= width_scale
        tau = np.abs(rng.standard_t(3.0, size=K)).astype(np.float32)
        X = normal_bf16(rng, (T, K), 1.0, col_scale=tau)
        W = normal_bf16(rng, (N, K), 0.02)
        dY = normal_bf16(rng, (T, N), 1.0)
        out["linears"].append({"name": name, "X": X, "W": W, "dY": dY, "M": T, "N": N, "K": K})
    return out


def moe_routing(seed: int = 0, tokens: int = 32768, experts: int = 128, topk: int = 8,
                zipf_s: float = 1.1):
    """Expert of every (token, slot) pair and the per-expert row counts.

    Expert popularity p_e is proportional to rank_e^-s over a seeded permutation of ranks;
    each token draws `topk` distinct experts by Gumbel-top-k on log p + Gumbel noise.
    Returns (token index per sorted row, group offsets [E+1])."""
    rng = np.random.default_rng(seed)
    ranks = rng.permutation(experts) + 1
    logp = -zipf_s * np.log(ranks.astype(np.float64))
    logp -= np.log(np.exp(logp).sum())
    g = rng.gumbel(size=(tokens, experts))
    choice = np.argsort(-(logp[None, :] + g), axis=1)[:, :topk]          # [T, topk]
    expert_of_row = choice.reshape(-1)
    token_of_row = np.repeat(np.arange(tokens), topk)
    order = np.argsort(expert_of_row, kind="stable")
    counts = np.bincount(expert_of_row, minlength=experts)
    offsets = np.zeros(experts + 1, np.int64)
    offsets[1:] = np.cumsum(counts)
    return token_of_row[order], offsets


def moe_experts(seed: int = 0, tokens: int = 32768, experts: int = 128, hidden: int = 3072,
                inter: int = 1536, topk: int = 8) -> dict:
    """Grouped expert workload (host arrays; intended for reduced sizes in tests)."""
    tok, offsets = moe_routing(seed, tokens, experts, topk)
    rng = np.random.default_rng(seed + 1)
    Xtok = normal_bf16(rng, (tokens, hidden), 1.0)
    X = Xtok[tok]
    Wgu = normal_bf16(rng, (experts * 2 * inter, hidden), 0.02).reshape(experts, 2 * inter, hidden)
    Wd = normal_bf16(rng, (experts * hidden, inter), 0.02).reshape(experts, hidden, inter)
    T = X.shape[0]
    Xd = normal_bf16(rng, (T, inter), 1.0)
    dYgu = normal_bf16(rng, (T, 2 * inter), 1.0)
    dYd = normal_bf16(rng, (T, hidden), 1.0)
    return {"offsets": offsets, "X": X, "Wgu": Wgu, "Wd": Wd, "Xd": Xd, "dYgu": dYgu,
            "dYd": dYd, "E": experts, "T": T, "hidden": hidden, "inter": inter}


def lora_factors(seed: int, N: int, K: int, r: int = 16, alpha: float | None = None) -> dict:
    """FP32 LoRA factors A [r, K], B [N, r] and the multiplier s = alpha / r (alpha = 2r)."""
    rng = np.random.default_rng(seed)
    A = (rng.standard_normal((r, K), dtype=np.float32) * np.float32(1.0 / np.sqrt(K)))
    B = (rng.standard_normal((N, r), dtype=np.float32) * np.float32(0.001 * np.sqrt(K / r)))
    a = 2.0 * r if alpha is None else float(alpha)
    return {"A": A.astype(np.float32), "B": B.astype(np.float32), "r": r, "scale": a / r}


def qad_logits(seed: int, L: int, V: int = 151936) -> dict:
    """bf16 teacher / student logits [L, V] (see the module docstring)."""
    rng = np.random.default_rng(seed)
    zt = np.empty((L, V), np.uint16)
    zs = np.empty((L, V), np.uint16)
    step = max(1, (1 << 22) // max(V, 1))
    for r0 in range(0, L, step):
        r1 = min(L, r0 + step)
        t = rng.standard_normal((r1 - r0, V), dtype=np.float32) * np.float32(2.0)
        for i in range(r1 - r0):
            k = int(rng.integers(1, 5))
            idx = rng.integers(0, V, size=k)
            t[i, idx] += rng.uniform(6.0, 14.0, size=k).astype(np.float32)
        s_ = t + rng.standard_normal((r1 - r0, V), dtype=np.float32) * np.float32(0.5)
        zt[r0:r1] = to_bf16(t)
        zs[r0:r1] = to_bf16(s_)
    return {"zt": zt, "zs": zs, "L": L, "V": V}
