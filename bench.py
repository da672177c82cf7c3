"""Benchmark: one quantization-aware linear layer step (fake quant + BF16 MFMA GEMMs,
forward + straight-through backward) on one MI355X.

Workload (default): the 8B-class MLP up-projection with MXFP4 weights and activations,
X [8192, 4096], W [14336, 4096], dY [8192, 14336] (seeded synthetic bf16, see workloads/).
One step is the layer's two C-ABI calls, qf_qlinear_fwd then qf_qlinear_bwd_ste, which run
the whole hot path:
    forward:  Q(W) -> W_hat, Q(X) -> X_hat (MXFP4 quantize-dequantize), Y = X_hat W_hat^T
    backward: Q(W) -> W_hat^T and Q(X) -> X_hat^T (transposing quantizer: the quantized
              tensors are transient, as in the paper), dY^T, dX = dY W_hat,
              dW = dY^T X_hat (FP32); all three products are NT GEMMs
`value` is the step's throughput in TFLOP/s over the three GEMMs' 3 * 2MNK flops, with the
quantization time inside the step.  A second pass issues the same kernels one C-ABI call at a
time, each bracketed by HIP events on the stream it runs on: that gives the per-kernel
durations of the roofline record.  The fake-quant kernel bandwidth is measured separately
over rotating input buffers (>1 GB) so the 256 MB MALL cannot serve repeated reads.

Prints ONE JSON line.  Only --gpus 1 is supported.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense BF16 MFMA
PEAK_HBM_GBPS = 8000.0        # MI355X HBM3E


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    # untimed: the GPU clock under back-to-back GEMMs settles over the first ~10 steps
    p.add_argument("--warmup", type=int, default=25)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-rows", type=int, default=256,
                   help="token rows in the CPU oracle's bounded sample of the step")
    p.add_argument("--main-only", action="store_true",
                   help="time only the MXFP4 MLP up-projection step (used for counter runs)")
    p.add_argument("--rows", default=None,
                   help="run only these secondary row groups (comma-separated: quant, dense, moe, "
                        "lora, moe_lora, kl, q4k) and print them as one JSON object; no step timing "
                        "(used for per-row kernel traces)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 1 GiB device-to-device copy (reference for the "
                        "HBM byte counters) and exit")
    return p.parse_args()


def measured_traffic(launch):
    """HBM bytes per launch of `launch` from the committed FETCH_SIZE/WRITE_SIZE counter summary
    (copy-calibrated), or None when no summary covers it or the kernel source has changed since
    the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "gemm_nt_mlp_up_step_traffic.json")
    try:
        rec = json.load(open(path))
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
        entry = rec["launches"].get(launch)
    except (OSError, ValueError, KeyError, AttributeError):
        return None
    if entry is None or hashlib.sha256(src).hexdigest() != rec["source_sha256"]:
        return None
    return entry["bytes"]


def copy_calibration():
    """A plain copy of known size: 2^30 bytes read and 2^30 bytes written, 5 times."""
    import torch
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": 1 << 30, "repeats": 5}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the layer has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    import torch
    import paper_2609_39223_amd as qf
    import workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    qf.lib()
    if args.rows:
        print(json.dumps({"rows": other_rows(qf, torch, dev, set(args.rows.split(",")))}),
              flush=True)
        return
    w = workloads.mlp_up(seed=0)
    M, N, K = w["M"], w["N"], w["K"]

    def up(a):
        return torch.from_numpy(a.view(np.int16)).to(dev)

    X, W, dY = up(w["X"]), up(w["W"]), up(w["dY"])
    Y = torch.empty(M, N, dtype=torch.int16, device=dev)
    dX = torch.empty(M, K, dtype=torch.int16, device=dev)
    dW = torch.empty(N, K, dtype=torch.float32, device=dev)

    # ---- the timed step: the layer's two C-ABI calls, forward then STE backward ------------
    desc = qf.qlinear_desc(M, N, K, "mxfp4", "mxfp4")
    ws = qf.workspace(desc)

    def layer_step():
        qf.qlinear_fwd(desc, X, W, Y, ws)
        qf.qlinear_bwd_ste(desc, dY, X, W, dX, dW, ws)

    for _ in range(args.warmup):
        layer_step()
    torch.cuda.synchronize()
    sev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    sev[0].record()
    for i in range(args.steps):
        layer_step()
        sev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = [sev[i].elapsed_time(sev[i + 1]) for i in range(args.steps)]
    ms_step = float(np.mean(step_ms))
    gemm_flops = 2.0 * M * N * K
    tflops = 3 * gemm_flops / (ms_step * 1e-3) / 1e12
    del ws

    # ---- per-launch breakdown: the same kernels the two calls issue, one C-ABI call each, so
    # every launch is bracketed by HIP events on the stream it runs on ------------------------
    what = torch.empty(N, K, dtype=torch.int16, device=dev)
    xhat = torch.empty(M, K, dtype=torch.int16, device=dev)
    whatt = torch.empty(K, N, dtype=torch.int16, device=dev)
    xhatt = torch.empty(K, M, dtype=torch.int16, device=dev)
    dYt = torch.empty(N, M, dtype=torch.int16, device=dev)
    gws = qf.gemm_workspace(N, K, 1)        # dW's split last round, as in the layer call
    # (the dX GEMM also writes dY^T, the left operand of dW, as the layer's backward does)
    phases = ["quant_W", "quant_X", "gemm_fwd", "quant_W_transposed", "gemm_dX_and_dY_transposed",
              "quant_X_transposed", "gemm_dW"]
    calls = [
        lambda: qf.fakequant_mxfp4(W, None, None, what),
        lambda: qf.fakequant_mxfp4(X, None, None, xhat),
        lambda: qf.gemm_bf16(M, N, K, xhat, K, 1, what, K, 1, Y, N, 0),
        lambda: qf.fakequant_transposed(W, "mxfp4", whatt),
        lambda: qf.gemm_bf16_at(M, K, N, dY, N, whatt, N, dX, K, dYt, M),
        lambda: qf.fakequant_transposed(X, "mxfp4", xhatt),
        lambda: qf.gemm_bf16(N, K, M, dYt, M, 1, xhatt, M, 1, dW, K, 1, ws=gws),
    ]

    def step(ev=None):
        for i, c in enumerate(calls):
            if ev is not None:
                ev[i].record()
            c()
        if ev is not None:
            ev[len(calls)].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(phases) + 1)]
              for _ in range(args.steps)]
    for s_ in range(args.steps):
        step(events[s_])
    torch.cuda.synchronize()
    per_phase = np.zeros(len(phases))
    for ev in events:
        per_phase += [ev[i].elapsed_time(ev[i + 1]) for i in range(len(phases))]
    per_phase /= args.steps
    gemm_ms = {p: float(per_phase[i]) for i, p in enumerate(phases) if p.startswith("gemm")}
    dom = max(gemm_ms, key=gemm_ms.get)
    achieved = gemm_flops / (gemm_ms[dom] * 1e-3) / 1e12

    # ---- fake-quant bandwidth over rotating buffers (W-shaped, > 1 GB in total) -----------
    nbuf = 10
    bufs = [torch.empty_like(W) for _ in range(nbuf)]
    for b in bufs:   # finite bf16 payloads of N(0, 0.02)-like magnitude
        b.copy_((torch.randn(N, K, device=dev) * 0.02).to(torch.bfloat16).view(torch.int16))
    codes = torch.empty(N, K // 2, dtype=torch.uint8, device=dev)
    scales = torch.empty(N, K // 32, dtype=torch.uint8, device=dev)
    outs = torch.empty(N, K, dtype=torch.int16, device=dev)
    for b in bufs[:2]:
        qf.fakequant_mxfp4(b, codes, scales, outs)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 3 * nbuf
    e0.record()
    for i in range(reps):
        qf.fakequant_mxfp4(bufs[i % nbuf], codes, scales, outs)
    e1.record()
    torch.cuda.synchronize()
    q_ms = e0.elapsed_time(e1) / reps
    q_bytes = N * K * (2 + 2 + 0.5 + 1.0 / 32)
    q_gbps = q_bytes / (q_ms * 1e-3) / 1e9
    del bufs

    del X, W, dY, what, xhat, whatt, xhatt, dYt, Y, dX, dW, gws
    torch.cuda.empty_cache()
    rows = None if args.main_only else other_rows(qf, torch, dev)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_rows)

    out = {
        "metric": "fake-quant GB/s and fused fake-quant+BF16 GEMM TFLOP/s (fwd+bwd), 1 MI355X",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations with 41 outlier channels x20, N(0,0.02) weights)",
        "config": {"workload": "mlp_up_mxfp4_w4a4: X 8192x4096, W 14336x4096, fwd + STE bwd",
                   "M": M, "N": N, "K": K, "wfmt": "mxfp4", "afmt": "mxfp4"},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(dom), "traffic_unit": "bytes per launch"},
        "phases_ms": {p: round(float(per_phase[i]), 4) for i, p in enumerate(phases)},
        "phases_sum_ms": round(float(per_phase.sum()), 4),
        "fakequant": {"kernel": "mxfp4 (codes+scales+x_hat)", "tensor": f"{N}x{K}",
                      "GBps": round(q_gbps, 1), "frac_hbm": round(q_gbps / PEAK_HBM_GBPS, 4),
                      "us": round(q_ms * 1e3, 2), "bytes_per_elem": 4.53125},
        "wall_s_timed": round(wall, 3),
        "rows": rows,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def _time(torch, fn, reps=10, warm=2):
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def _randn_bf16(torch, gen, shape, std=1.0, col_scale=None, row_scale=None):
    z = torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32)
    if std != 1.0:
        z.mul_(std)
    if col_scale is not None:
        z.mul_(col_scale[None, :])
    if row_scale is not None:
        z.mul_(row_scale[:, None])
    return z.to(torch.bfloat16)


def other_rows(qf, torch, dev, only=None):
    """Throughput of the remaining hot-path steps on their own workloads (seeded synthetic
    data drawn on the GPU): every quantizer and the amax pass over W-shaped tensors through
    rotating buffers, the transpose, the 9B-class dense layer at 32K tokens (NVFP4 weights,
    tied QKV and gate/up scales), the 128-expert grouped layer (NVFP4 weights, Zipf(1.1)
    top-8 routing), the LoRA-QAD layer (rank-16 adapter on the MLP up-projection) and the
    Q4_K export packing + forward GEMM."""
    def want(name):
        return only is None or name in only

    import workloads
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0)
    out = {}
    N, K = 14336, 4096
    if want("quant"):
        nbuf = 10
        bufs = [_randn_bf16(torch, gen, (N, K), 0.02) for _ in range(nbuf)]
        codes = torch.empty(N, K // 2, dtype=torch.uint8, device=dev)
        sc16 = torch.empty(N, K // 16, dtype=torch.uint8, device=dev)
        sc32 = torch.empty(N, K // 32, dtype=torch.uint8, device=dev)
        packed = torch.empty(N, K // 256, 144, dtype=torch.uint8, device=dev)
        xh = torch.empty(N, K, dtype=torch.int16, device=dev)
        amax = torch.zeros(1, dtype=torch.float32, device=dev)
        s_out = torch.zeros(1, dtype=torch.float32, device=dev)
        tr = torch.empty(K, N, dtype=torch.int16, device=dev)
        it = [0]

        def nxt():
            it[0] += 1
            return bufs[it[0] % nbuf]

        def gbps(fn, bpe):
            ms = _time(torch, fn, reps=3 * nbuf)
            g = N * K * bpe / (ms * 1e-3) / 1e9
            return {"us": round(ms * 1e3, 2), "GBps": round(g, 1), "frac_hbm": round(g / PEAK_HBM_GBPS, 4),
                    "bytes_per_elem": bpe}

        out["a1_amax"] = gbps(lambda: qf.amax(nxt(), amax), 2.0)
        out["nvfp4_amax_computed"] = gbps(
            lambda: qf.fakequant_nvfp4(nxt(), amax, qf.AMAX_COMPUTE, s_out, codes, sc16, xh), 4.5625)
        out["nvfp4_amax_given"] = gbps(
            lambda: qf.fakequant_nvfp4(nxt(), amax, qf.AMAX_GIVEN, s_out, codes, sc16, xh), 4.5625)
        out["mxfp4"] = gbps(lambda: qf.fakequant_mxfp4(nxt(), codes, sc32, xh), 4.53125)
        out["mxfp4_xhat_only"] = gbps(lambda: qf.fakequant_mxfp4(nxt(), None, None, xh), 4.0)
        out["q4k_pack"] = gbps(lambda: qf.fakequant_q4k(nxt(), packed, xh), 4.5625)
        out["transpose"] = gbps(lambda: qf.transpose_bf16(nxt(), tr), 4.0)
        for k in list(out):
            out[k]["tensor"] = f"{N}x{K}"
        del bufs, codes, sc16, sc32, packed, xh, tr

    if want("dense"):
        # ---- 9B-class dense layer at 32K tokens: QKV, O, gate/up, down (NVFP4 weights) ---------
        T = 32768
        layer = []
        flops = 0.0
        for name, n, k in workloads.DENSE_LINEARS:
            tau = torch.from_numpy(np.abs(np.random.default_rng(k).standard_t(3.0, size=k))
                                   .astype(np.float32)).to(dev)
            Xl = _randn_bf16(torch, gen, (T, k), col_scale=tau)
            Wl = _randn_bf16(torch, gen, (n, k), 0.02)
            dYl = _randn_bf16(torch, gen, (T, n))
            d = qf.qlinear_desc(T, n, k, "nvfp4", "none")
            layer.append((d, Xl, Wl, dYl, torch.empty(T, n, dtype=torch.bfloat16, device=dev),
                          torch.empty(T, k, dtype=torch.bfloat16, device=dev),
                          torch.empty(n, k, dtype=torch.float32, device=dev), qf.workspace(d)))
            flops += 3 * 2.0 * T * n * k

        def dense_step():
            for d, Xl, Wl, dYl, Yl, dXl, dWl, ws in layer:
                qf.qlinear_fwd(d, Xl, Wl, Yl, ws)
                qf.qlinear_bwd_ste(d, dYl, Xl, Wl, dXl, dWl, ws)

        ms = _time(torch, dense_step, reps=3, warm=1)
        out["dense_layer_32k_nvfp4"] = {"ms": round(ms, 3), "TFLOPs": round(flops / (ms * 1e-3) / 1e12, 1),
                                        "work": "T=32768, QKV 6144, O 4096, gate/up 24576, down 4096x12288, fwd + STE bwd"}
        del layer
        torch.cuda.empty_cache()

    if want("moe"):
        # ---- 128-expert grouped layer, Zipf(1.1) top-8 routing of 32768 tokens -------------------
        _, offsets = workloads.moe_routing(seed=0, tokens=32768, experts=128, topk=8)
        E, Tm, H, I = 128, int(offsets[-1]), 3072, 1536
        off = torch.from_numpy(offsets).to(dev)
        gflops = 0.0
        glayers = []
        for n, k in ((2 * I, H), (H, I)):
            Xg = _randn_bf16(torch, gen, (Tm, k))
            Wg = _randn_bf16(torch, gen, (E * n, k), 0.02)
            dYg = _randn_bf16(torch, gen, (Tm, n))
            d = qf.grouped_desc(E, Tm, n, k, "nvfp4", "none")
            glayers.append((d, Xg, Wg, dYg, torch.empty(Tm, n, dtype=torch.bfloat16, device=dev),
                            torch.empty(Tm, k, dtype=torch.bfloat16, device=dev),
                            torch.empty(E, n, k, dtype=torch.float32, device=dev), qf.grouped_workspace(d)))
            gflops += 3 * 2.0 * Tm * n * k

        def moe_step():
            for d, Xg, Wg, dYg, Yg, dXg, dWg, ws in glayers:
                qf.qlinear_grouped_fwd(d, off, Xg, Wg, Yg, ws)
                qf.qlinear_grouped_bwd_ste(d, off, dYg, Xg, Wg, dXg, dWg, ws)

        ms = _time(torch, moe_step, reps=3, warm=1)
        cnt = np.diff(offsets)
        out["moe_grouped_nvfp4"] = {"ms": round(ms, 3), "TFLOPs": round(gflops / (ms * 1e-3) / 1e12, 1),
                                    "work": f"128 experts, {Tm} routed rows (per expert {cnt.min()}..{cnt.max()}), "
                                            "gate/up 3072->3072 + down 1536->3072, fwd + STE bwd"}
        del glayers
        torch.cuda.empty_cache()

    if want("lora"):
        # ---- LoRA-QAD: the MXFP4 W4A4 MLP up-projection with a rank-16 adapter -------------------
        out["lora_mlp_up_r16"] = lora_row(qf, torch, dev, gen)

    if want("moe_lora"):
        # ---- MoE LoRA-QAD: the same 128 experts with rank-16 adapters in the hybrid layout ------
        _, offsets = workloads.moe_routing(seed=0, tokens=32768, experts=128, topk=8)
        E, Tm, H, I = 128, int(offsets[-1]), 3072, 1536
        off = torch.from_numpy(offsets).to(dev)
        r = 16
        glayers = []
        for n, k, shared in ((2 * I, H, "A"), (H, I, "B")):
            Xg = _randn_bf16(torch, gen, (Tm, k))
            Wg = _randn_bf16(torch, gen, (E * n, k), 0.02)
            dYg = _randn_bf16(torch, gen, (Tm, n))
            Ag = torch.randn((r, k) if shared == "A" else (E, r, k), generator=gen, device=dev) / np.sqrt(k)
            Bg = torch.randn((n, r) if shared == "B" else (E, n, r), generator=gen, device=dev) * (0.001 * np.sqrt(k / r))
            lo = qf.lora(Ag.contiguous(), Bg.contiguous(), 2.0, a_shared=shared == "A",
                         b_shared=shared == "B")
            d = qf.grouped_desc(E, Tm, n, k, "nvfp4", "none")
            glayers.append((d, lo, Xg, Wg, dYg, torch.empty(Tm, n, dtype=torch.bfloat16, device=dev),
                            torch.empty(Tm, k, dtype=torch.bfloat16, device=dev),
                            torch.empty_like(Ag), torch.empty_like(Bg), qf.grouped_lora_workspace(d, lo)))

        def moe_lora_step():
            for d, lo, Xg, Wg, dYg, Yg, dXg, dAg, dBg, ws in glayers:
                qf.qlinear_grouped_lora_fwd(d, lo, off, Xg, Wg, Yg, ws)
                qf.qlinear_grouped_lora_bwd_ste(d, lo, off, dYg, Xg, Wg, dXg, dAg, dBg, ws)

        ms = _time(torch, moe_lora_step, reps=3, warm=1)
        gf = 2 * 2.0 * Tm * (2 * I * H + H * I)
        out["moe_lora_nvfp4_r16"] = {"ms": round(ms, 3), "TFLOPs": round(gf / (ms * 1e-3) / 1e12, 1),
                                     "work": "the 128-expert layer above with frozen expert weights and "
                                             "rank-16 adapters (gate/up: A shared, down: B shared), fwd + "
                                             "STE bwd (dX, dA, dB); TFLOPs counts fwd + dX GEMMs"}
        del glayers
        torch.cuda.empty_cache()

    if want("kl"):
        # ---- QAD distillation loss: 8192 tokens over a 151936-token vocabulary ------------------
        out["qad_kl_8k_v152k"] = kl_row(qf, torch, dev, gen)

    if want("q4k"):
        # ---- Q4_K export: quantize + pack W [14336, 4096], then the forward GEMM at M = 4096 ----
        Wq = _randn_bf16(torch, gen, (N, K), 0.02, row_scale=torch.exp(0.5 * torch.randn(N, generator=gen, device=dev)))
        Xq = _randn_bf16(torch, gen, (4096, K))
        d = qf.qlinear_desc(4096, N, K, "q4k", "none")
        ws = qf.workspace(d)
        Yq = torch.empty(4096, N, dtype=torch.bfloat16, device=dev)
        packed = torch.empty(N, K // 256, 144, dtype=torch.uint8, device=dev)
        ms_pack = _time(torch, lambda: qf.fakequant_q4k(Wq, packed, None), reps=10)
        ms_fwd = _time(torch, lambda: qf.qlinear_fwd(d, Xq, Wq, Yq, ws), reps=10)
        xm = torch.empty(N, K, dtype=torch.bfloat16, device=dev)
        x0 = torch.empty(N, K, dtype=torch.bfloat16, device=dev)
        ms_mse = _time(torch, lambda: qf.fakequant_q4k_mse(Wq, packed, xm), reps=5)
        qf.fakequant_q4k(Wq, None, x0)
        torch.cuda.synchronize()
        wf = Wq.float()
        ratio = float(((wf - xm.float()) ** 2).sum() / ((wf - x0.float()) ** 2).sum())
        out["q4k_mse_search"] = {
            "us": round(ms_mse * 1e3, 1),
            "GBps": round(N * K * (2 + 2 + 144 / 256) / (ms_mse * 1e-3) / 1e9, 1),
            "sq_error_vs_min_max": round(ratio, 4),
            "work": "W 14336x4096 (per-row log-normal scale) -> 144-byte blocks + x_hat with the "
                    "searched sub-block steps (17 candidates, least-squares refit); ALU-bound"}
        del xm, x0, wf
        out["q4k_export_and_forward"] = {
            "pack_us": round(ms_pack * 1e3, 2),
            "pack_GBps": round(N * K * (2 + 144 / 256) / (ms_pack * 1e-3) / 1e9, 1),
            "forward_ms": round(ms_fwd, 4),
            "forward_TFLOPs": round(2.0 * 4096 * N * K / (ms_fwd * 1e-3) / 1e12, 1),
            "work": "W 14336x4096 (per-row log-normal scale) -> 144-byte blocks; Y = X Q(W)^T, X 4096x4096"}
    return out


def lora_row(qf, torch, dev, gen):
    """LoRA-QAD step on the MLP up-projection shape (X 8192x4096, frozen W 14336x4096, rank-16
    FP32 factors, scale 2): the layer's two C-ABI calls (merged quantize + forward GEMM; merged
    transposed quantize + dX GEMM + dA, dB), and each backward output on its own."""
    M, N, K, r = 8192, 14336, 4096, 16
    X = _randn_bf16(torch, gen, (M, K))
    W = _randn_bf16(torch, gen, (N, K), 0.02)
    dY = _randn_bf16(torch, gen, (M, N))
    A = torch.randn(r, K, generator=gen, device=dev) * (1.0 / np.sqrt(K))
    B = torch.randn(N, r, generator=gen, device=dev) * (0.001 * np.sqrt(K / r))
    lo = qf.lora(A.contiguous(), B.contiguous(), 2.0)
    d = qf.qlinear_desc(M, N, K, "mxfp4", "mxfp4")
    ws = qf.lora_workspace(d, lo)
    Y = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
    dX = torch.empty(M, K, dtype=torch.bfloat16, device=dev)
    dA = torch.empty(r, K, dtype=torch.float32, device=dev)
    dB = torch.empty(N, r, dtype=torch.float32, device=dev)
    xh = torch.empty(N, K, dtype=torch.bfloat16, device=dev)
    tr = torch.empty(K, N, dtype=torch.bfloat16, device=dev)

    def step():
        qf.qlinear_lora_fwd(d, lo, X, W, Y, ws)
        qf.qlinear_lora_bwd_ste(d, lo, dY, X, W, dX, dA, dB, ws)

    ms = _time(torch, step, reps=10, warm=2)
    ms_fwd = _time(torch, lambda: qf.qlinear_lora_fwd(d, lo, X, W, Y, ws), reps=10)
    ms_dx = _time(torch, lambda: qf.qlinear_lora_bwd_ste(d, lo, dY, X, W, dX, None, None, ws), reps=10)
    ms_da = _time(torch, lambda: qf.qlinear_lora_bwd_ste(d, lo, dY, X, W, None, dA, None, ws), reps=10)
    ms_db = _time(torch, lambda: qf.qlinear_lora_bwd_ste(d, lo, dY, X, W, None, None, dB, ws), reps=10)
    ms_q = _time(torch, lambda: qf.lora_fakequant(W, lo, "mxfp4", xhat=xh), reps=20)
    ms_qt = _time(torch, lambda: qf.lora_fakequant_transposed(W, lo, "mxfp4", tr), reps=20)
    gemm = 2.0 * M * N * K
    lora_flops = 2 * (2.0 * N * K * r) + 2 * (2.0 * M * K * r) + 2 * (2.0 * M * N * r)
    merge_gflop = 2.0 * N * K * r / 1e9
    return {
        "ms": round(ms, 4),
        "TFLOPs": round((2 * gemm + lora_flops) / (ms * 1e-3) / 1e12, 1),
        "fwd_ms": round(ms_fwd, 4), "bwd_dX_only_ms": round(ms_dx, 4),
        "bwd_dA_only_ms": round(ms_da, 4), "bwd_dB_only_ms": round(ms_db, 4),
        "merged_quant_us": round(ms_q * 1e3, 2),
        "merged_quant_GBps": round(N * K * 4.0 / (ms_q * 1e-3) / 1e9, 1),
        "merged_quant_TFLOPs": round(merge_gflop / (ms_q * 1e-3) / 1e3, 2),
        "merged_quant_transposed_us": round(ms_qt * 1e3, 2),
        "work": "X 8192x4096, W 14336x4096 frozen, A 16x4096 / B 14336x16 FP32, MXFP4 W4A4; "
                "fwd + STE bwd (dX, dA, dB); TFLOPs counts fwd + dX GEMMs and the rank-16 terms"}


def kl_row(qf, torch, dev, gen):
    """Forward KL of Eq. qad-objective with its student-logit gradient and top-1 agreement, for
    one 8K-token sequence over a 151936-token vocabulary (bf16 logits, teacher 2 N(0,1) with
    three boosted tokens per row, student = teacher + N(0, 0.25))."""
    L, V = 8192, 151936
    t = torch.randn(L, V, generator=gen, device=dev) * 2
    hot = torch.randint(0, V, (L, 3), generator=gen, device=dev)
    t.scatter_add_(1, hot, torch.rand(L, 3, generator=gen, device=dev) * 8 + 6)
    s = t + torch.randn(L, V, generator=gen, device=dev) * 0.5
    zt, zs = t.to(torch.bfloat16), s.to(torch.bfloat16)
    del t, s
    kl = torch.empty(L, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    agree = torch.empty(L, dtype=torch.int32, device=dev)
    grad = torch.empty(L, V, dtype=torch.bfloat16, device=dev)
    ms = _time(torch, lambda: qf.qad_kl(zt, zs, kl, loss=loss, grad=grad, agree=agree), reps=10)
    ms_loss = _time(torch, lambda: qf.qad_kl(zt, zs, kl, loss=loss, agree=agree), reps=10)
    n = L * V
    out = {"ms": round(ms, 4), "tokens_per_s": round(L / (ms * 1e-3), 1),
           "GBps_algorithmic": round(n * 6.0 / (ms * 1e-3) / 1e9, 1),
           "frac_hbm": round(n * 6.0 / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
           "loss_only_ms": round(ms_loss, 4),
           "loss_only_GBps": round(n * 4.0 / (ms_loss * 1e-3) / 1e9, 1),
           "loss": round(float(loss.item()), 6),
           "work": "L=8192 tokens, V=151936, bf16 logits; algorithmic bytes 6 per element "
                   "(two logits read, gradient written); the kernel reads the logits twice"}
    del zt, zs, grad
    torch.cuda.empty_cache()
    return out


def cpu_baseline(w, rows):
    """The CPU oracle on a bounded sample of the same step: `rows` token rows of X and dY
    (full W): MXFP4 fake quant of W and of the sampled X rows, then the three FP64 products
    restricted to those rows.  Throughput counts the sample's 3 * 2 * rows * N * K flops."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = 1
    M, N, K = w["M"], w["N"], w["K"]
    Xs, dYs = w["X"][:rows], w["dY"][:rows]
    t0 = time.perf_counter()
    wq = oracle.mxfp4(w["W"])["xhat"]
    xq = oracle.mxfp4(Xs)["xhat"]
    oracle.linear_fwd(xq, wq)
    oracle.linear_dx(dYs, wq)
    oracle.linear_dw(dYs, xq)
    dt = time.perf_counter() - t0
    flops = 3 * 2.0 * rows * N * K
    return {"value": round(flops / dt / 1e12, 5), "unit": "TFLOP/s", "cores": int(cores),
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"{rows} of {M} token rows (full {N}x{K} weight quantized), MXFP4 W4A4 "
                      "fwd + dX + dW in FP64"}


if __name__ == "__main__":
    main()
