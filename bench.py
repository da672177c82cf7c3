"""Benchmark: the 9B-class transformer layer at 32K tokens through the quantization-aware
linear layer (NVFP4 weight fake quant + BF16 MFMA GEMMs, forward + straight-through backward)
on one MI355X.

Workload (the headline): one 32768-token sequence through a 9B-class dense layer's four fused
linears -- QKV 4096 -> 6144 (4096 + 1024 + 1024, one tied tensor scale), O 4096 -> 4096,
gate/up 4096 -> 2 x 12288 (tied), down 12288 -> 4096 -- seven projections, NVFP4 weight-only;
activations x = z |tau_c| with z ~ N(0,1) and heavy-tailed per-channel tau_c ~ Student-t(3),
weights ~ N(0, 0.02), upstream gradients ~ N(0,1) (seeded, drawn on the GPU).  One step is
the eight C-ABI calls qf_qlinear_fwd + qf_qlinear_bwd_ste of the four linears, which run the
whole hot path per linear:
    forward:  amax(W) -> g, Q(W) -> W_hat (NVFP4 quantize-dequantize), Y = X W_hat^T
    backward: amax(W), Q(W) -> W_hat^T (transposing quantizer), dX = dY W_hat with dY^T as a
              by-product, X^T, dW = dY^T X (FP32); all three products are NT GEMMs
`value` is the step's throughput in TFLOP/s over the 21 GEMMs' 3 * 2MNK flops (37.93 TF),
quantization and transposes inside the step.  A second pass issues the same kernels one
C-ABI call at a time, each bracketed by HIP events on the stream it runs on: that gives the
per-kernel durations of the roofline record.  Rows time the other configurations (the MXFP4
MLP up-projection, the quantizers over rotating buffers, the MoE layer, Q4_K export, ...).

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
METRIC = "fake-quant GB/s and fused fake-quant+BF16 GEMM TFLOP/s (fwd+bwd), 1 MI355X"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    # untimed: the GPU clock under back-to-back GEMMs settles over the first steps
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-rows", type=int, default=32,
                   help="token rows in the CPU oracle's bounded sample of the step")
    p.add_argument("--main-only", action="store_true",
                   help="time only the headline step and its per-call pass (no rows, no CPU "
                        "baseline)")
    p.add_argument("--phases-once", action="store_true",
                   help="issue the headline's per-call pass once, with no warm-up or timing "
                        "(dispatch order = phase order; used for the HBM counter runs)")
    p.add_argument("--rows", default=None,
                   help="run only these secondary row groups (comma-separated: mlp_up, quant, "
                        "moe, lora, moe_lora, kl, q4k, single, blas) and print them as one JSON object; no "
                        "headline step (used for per-row kernel traces)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 1 GiB device-to-device copy (reference for the "
                        "HBM byte counters) and exit")
    return p.parse_args()


def measured_traffic(profile, launch):
    """HBM bytes per launch of `launch` from a committed FETCH_SIZE / WRITE_SIZE counter
    summary (copy-calibrated) under profiles/, or None when none covers it or a kernel source
    has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", profile)
    try:
        rec = json.load(open(path))
        for src, sha in rec["sources"].items():
            if hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest() != sha:
                return None
        entry = rec["launches"].get(launch)
    except (OSError, ValueError, KeyError, AttributeError):
        return None
    return None if entry is None else entry["bytes"]


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


def dense_layer_inputs(torch, dev, gen):
    """The 9B-class layer's four fused linears at T = 32768 (seeded draws on the GPU)."""
    import workloads
    T = 32768
    lins = []
    for name, n, k in workloads.DENSE_LINEARS:
        tau = torch.from_numpy(np.abs(np.random.default_rng(k).standard_t(3.0, size=k))
                               .astype(np.float32)).to(dev)
        X = _randn_bf16(torch, gen, (T, k), col_scale=tau)
        W = _randn_bf16(torch, gen, (n, k), 0.02)
        dY = _randn_bf16(torch, gen, (T, n))
        lins.append({"name": name, "T": T, "N": n, "K": k, "X": X, "W": W, "dY": dY})
    return lins


def dense_phase_calls(qf, torch, dev, lin):
    """The kernels one linear's qf_qlinear_fwd + qf_qlinear_bwd_ste launch with a saved buffer
    and the workspace kept (QF_FLAG_REUSE_WS; NVFP4 weights, W's amax computed, bf16
    activations), one C-ABI call each, in the layer's order: the forward quantizes W once into
    its packed form (codes, scales, S; the saved operand) and its bf16 W_hat, then runs the GEMM,
    which also writes X^T for weights of at most 8192 rows; the backward dequantizes the packed
    W straight into W_hat^T, its dX GEMM also writes dY^T, and it transposes X itself for the
    wider weight."""
    T, N, K = lin["T"], lin["N"], lin["K"]
    X, W, dY = lin["X"], lin["W"], lin["dY"]
    ldm = T + 128 if T % 16384 == 0 else T        # the layer workspace's padded stride
    g = torch.zeros(1, dtype=torch.float32, device=dev)
    S = torch.zeros(1, dtype=torch.float32, device=dev)
    codes = torch.empty(N, K // 2, dtype=torch.uint8, device=dev)
    scales = torch.empty(N, K // 16, dtype=torch.uint8, device=dev)
    what = torch.empty(N, K, dtype=torch.bfloat16, device=dev)
    whatt = torch.empty(K, N, dtype=torch.bfloat16, device=dev)
    xt = torch.empty(K, ldm, dtype=torch.bfloat16, device=dev)
    dyt = torch.empty(N, ldm, dtype=torch.bfloat16, device=dev)
    Y = torch.empty(T, N, dtype=torch.bfloat16, device=dev)
    dX = torch.empty(T, K, dtype=torch.bfloat16, device=dev)
    dW = torch.empty(N, K, dtype=torch.float32, device=dev)
    gws = qf.gemm_workspace(N, K, 1)
    nm = lin["name"]
    calls = [
        (f"{nm}.amax_W", 0.0, lambda: qf.amax(W, g)),
        (f"{nm}.quant_W", 0.0,
         lambda: qf.fakequant_nvfp4(W, g, qf.AMAX_GIVEN, S, codes, scales, what)),
    ]
    if (N + 255) // 256 <= 32:     # the layer's forward GEMM also writes X^T (kept workspace)
        calls.append((f"{nm}.gemm_fwd_and_X_transposed", 2.0 * T * N * K,
                      lambda: qf.gemm_bf16_at(T, N, K, X, K, what, K, Y, N, xt, ldm)))
    else:                          # ... else the backward transposes X
        calls.append((f"{nm}.gemm_fwd", 2.0 * T * N * K,
                      lambda: qf.gemm_bf16(T, N, K, X, K, 1, what, K, 1, Y, N, 0)))
    calls += [
        (f"{nm}.dequant_W_transposed", 0.0,
         lambda: qf.dequantize_transposed("nvfp4", codes, scales, S, N, K, whatt)),
        (f"{nm}.gemm_dX_and_dY_transposed", 2.0 * T * N * K,
         lambda: qf.gemm_bf16_at(T, K, N, dY, N, whatt, N, dX, K, dyt, ldm)),
    ]
    if (N + 255) // 256 > 32:
        calls.append((f"{nm}.transpose_X", 0.0, lambda: qf.transpose_bf16(X, xt)))
    calls.append((f"{nm}.gemm_dW", 2.0 * T * N * K,
                  lambda: qf.gemm_bf16(N, K, T, dyt, ldm, 1, xt, ldm, 1, dW, K, 1, ws=gws)))
    return calls


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

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    qf.lib()
    if args.rows:
        print(json.dumps({"rows": other_rows(qf, torch, dev, set(args.rows.split(",")))}),
              flush=True)
        return
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0)
    lins = dense_layer_inputs(torch, dev, gen)

    if args.phases_once:
        calls = [c for lin in lins for c in dense_phase_calls(qf, torch, dev, lin)]
        torch.cuda.synchronize()
        for name, _, fn in calls:
            print(name, flush=True)
            fn()
            torch.cuda.synchronize()
        print(json.dumps({"phases_once": [c[0] for c in calls]}), flush=True)
        return

    # ---- the timed step: the four linears' C-ABI calls, forward then STE backward ---------
    layer = []
    flops = 0.0
    for lin in lins:
        T, N, K = lin["T"], lin["N"], lin["K"]
        # the workspace is kept from forward to backward: the forward GEMM also writes X^T
        d = qf.qlinear_desc(T, N, K, "nvfp4", "none", flags=qf.FLAG_REUSE_WS)
        layer.append((d, lin["X"], lin["W"], lin["dY"],
                      torch.empty(T, N, dtype=torch.bfloat16, device=dev),
                      torch.empty(T, K, dtype=torch.bfloat16, device=dev),
                      torch.empty(N, K, dtype=torch.float32, device=dev), qf.workspace(d),
                      qf.saved_buffer(d)))
        flops += 3 * 2.0 * T * N * K

    def layer_step():
        # forward saves the packed W_hat; the backward dequantizes it (Sec. 3.2.1)
        for d, X, W, dY, Y, dX, dW, ws, sv in layer:
            qf.qlinear_fwd(d, X, W, Y, ws, saved=sv)
            qf.qlinear_bwd_ste(d, dY, X, W, dX, dW, ws, saved=sv)

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
    ab = fused_ab(qf, torch, layer)
    ms_step = float(np.mean(step_ms))
    tflops = flops / (ms_step * 1e-3) / 1e12
    del layer
    torch.cuda.empty_cache()

    # ---- per-call pass: the same kernels, one C-ABI call each, each bracketed by HIP events
    # on the stream it runs on (torch's current stream, where the binding launches) --------
    calls = [c for lin in lins for c in dense_phase_calls(qf, torch, dev, lin)]
    reps = max(3, args.steps // 4)

    def one_pass(ev=None):
        for i, (_, _, fn) in enumerate(calls):
            if ev is not None:
                ev[i].record()
            fn()
        if ev is not None:
            ev[len(calls)].record()

    for _ in range(2):
        one_pass()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)] for _ in range(reps)]
    for r in range(reps):
        one_pass(evs[r])
    torch.cuda.synchronize()
    per = np.zeros(len(calls))
    for ev in evs:
        per += [ev[i].elapsed_time(ev[i + 1]) for i in range(len(calls))]
    per /= reps
    phases = {c[0]: round(float(per[i]), 4) for i, c in enumerate(calls)}
    gemms = [(c[0], c[1], float(per[i])) for i, c in enumerate(calls) if c[1] > 0]
    dom, dom_flops, dom_ms = max(gemms, key=lambda t: t[2])
    achieved = dom_flops / (dom_ms * 1e-3) / 1e12
    gemm_ms = sum(t[2] for t in gemms)
    del calls
    torch.cuda.empty_cache()

    rows = None
    if not args.main_only:
        del lins
        torch.cuda.empty_cache()
        rows = other_rows(qf, torch, dev)
    cpu = None
    if not args.no_cpu_baseline and not args.main_only:
        cpu = cpu_baseline(args.cpu_rows)

    out = {
        "metric": METRIC,
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
        "data": "synthetic (seeded on the GPU: x = N(0,1) * |Student-t(3)| per channel, "
                "N(0,0.02) weights, N(0,1) upstream gradients)",
        "config": {"workload": "dense_9b_layer_32k_nvfp4: one 32768-token sequence, hidden "
                               "4096, QKV 4096->6144 (tied scale), O 4096->4096, gate/up "
                               "4096->2x12288 (tied scale), down 12288->4096; NVFP4 weight-only "
                               "fake quant, all seven projections fwd + STE bwd",
                   "T": 32768, "linears": [[n, k] for _, n, k in __import__("workloads").DENSE_LINEARS],
                   "wfmt": "nvfp4", "afmt": "none", "step_tflop": round(flops / 1e12, 3)},
        "roofline": {"bound": "mfma", "kernel": "gemm_nt_kernel", "launch": dom,
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic("dense_layer_32k_nvfp4_traffic.json", dom),
                     "traffic_unit": "bytes per launch",
                     "launch_ms": round(dom_ms, 4), "launch_flop": dom_flops},
        "gemm_share": {"gemm_ms": round(gemm_ms, 4), "phases_sum_ms": round(float(per.sum()), 4),
                       "gemm_TFLOPs": round(flops / (gemm_ms * 1e-3) / 1e12, 1)},
        "phases_ms": phases,
        "fused_decode_ab": ab,
        "wall_s_timed": round(wall, 3),
        "rows": rows,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def fused_ab(qf, torch, layer, reps=10):
    """Same-run A/B of the layer calls: the forward that decodes the packed weight inside the
    GEMM (QF_FLAG_DECODE_IN_GEMM) against the default one that writes W_hat in bf16 and runs a
    plain GEMM (and the same writing X^T for a kept workspace), and the backward from the saved
    packed operands (with and without the forward's X^T) against the one that quantizes W
    again."""
    out = {}
    tot = {"fwd_fused": 0.0, "fwd_materialized": 0.0, "fwd_materialized_writing_Xt": 0.0,
           "bwd_from_saved": 0.0, "bwd_from_saved_and_Xt": 0.0, "bwd_requantize": 0.0}
    for d, X, W, dY, Y, dX, dW, ws, sv in layer:
        df = qf.qlinear_desc(d.M, d.N, d.K, "nvfp4", "none", flags=qf.FLAG_DECODE_IN_GEMM)
        d0 = qf.qlinear_desc(d.M, d.N, d.K, "nvfp4", "none")     # no workspace kept
        r = {"fwd_fused": _time(torch, lambda: qf.qlinear_fwd(df, X, W, Y, ws, saved=sv), reps, 2),
             "fwd_materialized": _time(torch, lambda: qf.qlinear_fwd(d0, X, W, Y, ws, saved=sv),
                                       reps, 2),
             "fwd_materialized_writing_Xt": _time(
                 torch, lambda: qf.qlinear_fwd(d, X, W, Y, ws, saved=sv), reps, 2),
             "bwd_from_saved": _time(torch, lambda: qf.qlinear_bwd_ste(d0, dY, X, W, dX, dW, ws,
                                                                       saved=sv), reps, 2),
             "bwd_from_saved_and_Xt": _time(
                 torch, lambda: qf.qlinear_bwd_ste(d, dY, X, W, dX, dW, ws, saved=sv), reps, 2),
             "bwd_requantize": _time(torch, lambda: qf.qlinear_bwd_ste(d0, dY, X, W, dX, dW, ws),
                                     reps, 2)}
        qf.qlinear_fwd(d, X, W, Y, ws, saved=sv)      # leave the saved buffer consistent
        for k in tot:
            tot[k] += r[k]
        out[f"{d.N}x{d.K}"] = {k: round(v, 4) for k, v in r.items()}
    out["total_ms"] = {k: round(v, 4) for k, v in tot.items()}
    return out


def mlp_up_row(qf, torch, dev):
    """The MXFP4 W4A4 MLP up-projection (X 8192x4096, W 14336x4096, dY 8192x14336, seeded on
    the host): the layer's two C-ABI calls per step (20 steps after 10 untimed), the per-call
    breakdown with its roofline record, and the MXFP4 quantizer over rotating buffers."""
    import workloads
    w = workloads.mlp_up(seed=0)
    M, N, K = w["M"], w["N"], w["K"]

    def up(a):
        return torch.from_numpy(a.view(np.int16)).to(dev)

    X, W, dY = up(w["X"]), up(w["W"]), up(w["dY"])
    Y = torch.empty(M, N, dtype=torch.int16, device=dev)
    dX = torch.empty(M, K, dtype=torch.int16, device=dev)
    dW = torch.empty(N, K, dtype=torch.float32, device=dev)
    desc = qf.qlinear_desc(M, N, K, "mxfp4", "mxfp4")
    ws = qf.workspace(desc)
    sv = qf.saved_buffer(desc)

    def layer_step():
        qf.qlinear_fwd(desc, X, W, Y, ws, saved=sv)
        qf.qlinear_bwd_ste(desc, dY, X, W, dX, dW, ws, saved=sv)

    ms_step = _time(torch, layer_step, reps=20, warm=10)
    gemm_flops = 2.0 * M * N * K
    del ws, sv
    wc = torch.empty(N, K // 2, dtype=torch.uint8, device=dev)
    wsc = torch.empty(N, K // 32, dtype=torch.uint8, device=dev)
    xc = torch.empty(M, K // 2, dtype=torch.uint8, device=dev)
    xsc = torch.empty(M, K // 32, dtype=torch.uint8, device=dev)
    xhat = torch.empty(M, K, dtype=torch.int16, device=dev)
    what = torch.empty(N, K, dtype=torch.int16, device=dev)
    whatt = torch.empty(K, N, dtype=torch.int16, device=dev)
    xhatt = torch.empty(K, M, dtype=torch.int16, device=dev)
    dYt = torch.empty(N, M, dtype=torch.int16, device=dev)
    gws = qf.gemm_workspace(N, K, 1)
    # the kernels of the two layer calls with a saved buffer, one C-ABI call each
    phases = ["quant_W", "quant_X", "gemm_fwd", "dequant_W_transposed",
              "gemm_dX_and_dY_transposed", "dequant_X_transposed", "gemm_dW"]
    calls = [
        lambda: qf.fakequant_mxfp4(W, wc, wsc, what),
        lambda: qf.fakequant_mxfp4(X, xc, xsc, xhat),
        lambda: qf.gemm_bf16(M, N, K, xhat, K, 1, what, K, 1, Y, N, 0),
        lambda: qf.dequantize_transposed("mxfp4", wc, wsc, None, N, K, whatt),
        lambda: qf.gemm_bf16_at(M, K, N, dY, N, whatt, N, dX, K, dYt, M),
        lambda: qf.dequantize_transposed("mxfp4", xc, xsc, None, M, K, xhatt),
        lambda: qf.gemm_bf16(N, K, M, dYt, M, 1, xhatt, M, 1, dW, K, 1, ws=gws),
    ]
    steps = 10

    def step(ev=None):
        for i, c in enumerate(calls):
            if ev is not None:
                ev[i].record()
            c()
        if ev is not None:
            ev[len(calls)].record()

    for _ in range(5):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(len(phases) + 1)]
              for _ in range(steps)]
    for s_ in range(steps):
        step(events[s_])
    torch.cuda.synchronize()
    per_phase = np.zeros(len(phases))
    for ev in events:
        per_phase += [ev[i].elapsed_time(ev[i + 1]) for i in range(len(phases))]
    per_phase /= steps
    gemm_ms = {p: float(per_phase[i]) for i, p in enumerate(phases) if p.startswith("gemm")}
    dom = max(gemm_ms, key=gemm_ms.get)
    achieved = gemm_flops / (gemm_ms[dom] * 1e-3) / 1e12
    del X, W, dY, wc, wsc, xc, xsc, xhat, what, whatt, xhatt, dYt, Y, dX, dW, gws
    torch.cuda.empty_cache()
    return {"ms": round(ms_step, 4), "TFLOPs": round(3 * gemm_flops / (ms_step * 1e-3) / 1e12, 1),
            "roofline": {"bound": "mfma", "launch": dom, "achieved": round(achieved, 2),
                         "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                         "traffic": None},       # HBM counters are kept for the headline workload
            "phases_ms": {p: round(float(per_phase[i]), 4) for i, p in enumerate(phases)},
            "work": "MXFP4 W4A4 MLP up-projection X 8192x4096, W 14336x4096, dY 8192x14336; "
                    "fwd + STE bwd (20 steps after 10 untimed)"}


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
    """Throughput of the other configurations on their own workloads (seeded synthetic data):
    the MXFP4 W4A4 MLP up-projection step, every quantizer and the amax pass over W-shaped
    tensors through rotating buffers, the transpose, the 128-expert grouped layer (NVFP4
    weights, Zipf(1.1) top-8 routing), the LoRA-QAD layers, the QAD loss and the Q4_K export
    packing + forward GEMM."""
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

    if want("single"):
        # ---- the single NVFP4 linear (W 512x512, X 256x512): a latency-bound correctness shape --
        w = workloads.single_linear(seed=0)
        X1, W1, dY1 = (torch.from_numpy(w[k].view(np.int16)).to(dev) for k in ("X", "W", "dY"))
        d1 = qf.qlinear_desc(256, 512, 512, "nvfp4", "none")
        ws1, sv1 = qf.workspace(d1), qf.saved_buffer(d1)
        Y1 = torch.empty(256, 512, dtype=torch.bfloat16, device=dev)
        dX1 = torch.empty(256, 512, dtype=torch.bfloat16, device=dev)
        dW1 = torch.empty(512, 512, dtype=torch.float32, device=dev)

        def single_step():
            qf.qlinear_fwd(d1, X1, W1, Y1, ws1, saved=sv1)
            qf.qlinear_bwd_ste(d1, dY1, X1, W1, dX1, dW1, ws1, saved=sv1)

        ms = _time(torch, single_step, reps=200, warm=20)
        # the same calls captured once in a HIP graph and replayed (the launch floor); the
        # replay's outputs are checked against the eager calls' first
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            single_step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        ref = (Y1.clone(), dX1.clone(), dW1.clone())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            single_step()
        graph.replay()
        torch.cuda.synchronize()
        same = all(torch.equal(a, b) for a, b in zip(ref, (Y1, dX1, dW1)))
        gms = _time(torch, graph.replay, reps=500, warm=20)
        out["single_linear_nvfp4"] = {
            "us": round(ms * 1e3, 2), "fwd_us": round(_time(
                torch, lambda: qf.qlinear_fwd(d1, X1, W1, Y1, ws1, saved=sv1), 200, 20) * 1e3, 2),
            "graph_us": round(gms * 1e3, 2), "graph_matches_eager": same,
            "work": "X 256x512, W 512x512 NVFP4 (amax computed), fwd + STE bwd: 0.403 GFLOP; "
                    "bound by its chain of small dependent kernels on the GPU (graph_us: the same "
                    "calls replayed from a HIP graph, no faster, so not by host launches)"}
        del graph

    if want("mlp_up"):
        # ---- the MXFP4 W4A4 MLP up-projection (8B-class) -------------------------------------
        out["mlp_up_mxfp4"] = mlp_up_row(qf, torch, dev)

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
                            torch.empty(E, n, k, dtype=torch.float32, device=dev), qf.grouped_workspace(d),
                            qf.grouped_saved_buffer(d)))
            gflops += 3 * 2.0 * Tm * n * k

        def moe_step():
            # the forward saves the experts' packed W_hat; the backward dequantizes it
            for d, Xg, Wg, dYg, Yg, dXg, dWg, ws, sv in glayers:
                qf.qlinear_grouped_fwd(d, off, Xg, Wg, Yg, ws, saved=sv)
                qf.qlinear_grouped_bwd_ste(d, off, dYg, Xg, Wg, dXg, dWg, ws, saved=sv)

        ms = _time(torch, moe_step, reps=10, warm=5)
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

    if want("blas"):
        # ---- context: this library's NT GEMM against hipBLASLt (torch's F.linear) on the 9B
        # layer's forward shapes and the MLP up shape, same operands, same run -------------------
        import torch.nn.functional as F
        shapes = {"qkv": (32768, 6144, 4096), "o": (32768, 4096, 4096), "gate_up": (32768, 24576, 4096),
                  "down": (32768, 4096, 12288), "mlp_up": (8192, 14336, 4096)}
        ctx = {}
        for name, (M, Nn, Kk) in shapes.items():
            A = _randn_bf16(torch, gen, (M, Kk))
            B = _randn_bf16(torch, gen, (Nn, Kk), 0.02)
            C = torch.empty(M, Nn, dtype=torch.bfloat16, device=dev)
            ws = qf.gemm_workspace(M, Nn, 0)
            ours = _time(torch, lambda: qf.gemm_bf16(M, Nn, Kk, A, Kk, 1, B, Kk, 1, C, Nn, 0, ws=ws), reps=10, warm=3)
            blas = _time(torch, lambda: F.linear(A, B), reps=10, warm=3)
            f = 2.0 * M * Nn * Kk
            ctx[name] = {"shape": f"{M}x{Nn}x{Kk}", "ours_ms": round(ours, 4), "hipblaslt_ms": round(blas, 4),
                         "ours_TFLOPs": round(f / (ours * 1e-3) / 1e12, 1),
                         "hipblaslt_TFLOPs": round(f / (blas * 1e-3) / 1e12, 1)}
            del A, B, C, ws
        out["gemm_vs_hipblaslt"] = ctx
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


def cpu_baseline(rows):
    """The CPU oracle (test infrastructure, as it stands) on a bounded sample of the headline
    step, on the host's cores (threads over row chunks, each an oracle call; numpy's BLAS for
    the FP64 products):
      - NVFP4 fake quant with the tensor amax computed (codes, scales, S and x_hat) of the 9B
        layer's four weights, all 193 M elements, on all threads; and of the QKV weight's first
        2048 rows on one thread -> GB/s of the 4.5625-byte model;
      - the FP64 products of `rows` token rows through the four linears (their rows of Y and
        dX and their rank-`rows` share of dW: 3 * 2 * rows * N * K flops per linear), on one
        thread and on all threads -> GFLOP/s.
    `value` is the sample's GEMM flops over the all-thread time of its quantization + GEMMs
    (TFLOP/s); `full_step_s_estimate` extrapolates the full 32768-token step."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    import workloads
    from threadpoolctl import threadpool_limits

    ncpu = os.cpu_count() or 1
    threads = max(1, min(ncpu, int(os.environ.get("OMP_NUM_THREADS", ncpu))))
    rng = np.random.default_rng(0)
    lins = []
    for name, n, k in workloads.DENSE_LINEARS:
        tau = np.abs(rng.standard_t(3.0, size=k)).astype(np.float32)
        lins.append({"name": name, "N": n, "K": k,
                     "W": workloads.normal_bf16(rng, (n, k), 0.02),
                     "X": workloads.normal_bf16(rng, (rows, k), 1.0, col_scale=tau),
                     "dY": workloads.normal_bf16(rng, (rows, n), 1.0)})
    nel = sum(l["N"] * l["K"] for l in lins)

    def quant_rows(W, g, r0, r1):
        return oracle.nvfp4(np.ascontiguousarray(W[r0:r1]), amax_in=g)["xhat"]

    # one thread: the QKV weight's first 2048 rows (its tensor amax over the whole weight)
    W0 = lins[0]["W"]
    t = time.perf_counter()
    g0 = oracle.amax(W0)
    quant_rows(W0, g0, 0, 2048)
    q1_s = time.perf_counter() - t
    q1_gbps = 2048 * W0.shape[1] * 4.5625 / q1_s / 1e9
    # all threads: every weight in full, chunks of 256 rows
    t = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as ex:
        for l in lins:
            g = oracle.amax(l["W"])
            parts = list(ex.map(lambda r0: quant_rows(l["W"], g, r0, min(l["N"], r0 + 256)),
                                range(0, l["N"], 256)))
            l["what"] = np.concatenate(parts)
    qn_s = time.perf_counter() - t
    qn_gbps = nel * 4.5625 / qn_s / 1e9

    def gemms():
        for l in lins:
            oracle.linear_fwd(l["X"], l["what"])
            oracle.linear_dx(l["dY"], l["what"])
            oracle.linear_dw(l["dY"], l["X"])

    flops = sum(3 * 2.0 * rows * l["N"] * l["K"] for l in lins)
    with threadpool_limits(limits=1):
        t = time.perf_counter()
        gemms()
        g1_s = time.perf_counter() - t
    with threadpool_limits(limits=threads):
        t = time.perf_counter()
        gemms()
        gn_s = time.perf_counter() - t
    full_flops = sum(3 * 2.0 * 32768 * l["N"] * l["K"] for l in lins)
    return {"value": round(flops / (qn_s + gn_s) / 1e12, 6), "unit": "TFLOP/s",
            "cores": threads, "host_cpu_count": ncpu, "kind": "oracle",
            "sample": f"{rows} of 32768 token rows through the 9B layer's four linears (FP64 "
                      f"fwd, dX, dW share) after NVFP4 fake quant of all four full weights "
                      f"({nel / 1e6:.0f} M elements)",
            "fakequant_nvfp4": {"GBps_1_thread": round(q1_gbps, 4), "s_1_thread": round(q1_s, 2),
                                "elements_1_thread": 2048 * W0.shape[1],
                                "GBps_all_threads": round(qn_gbps, 4), "s_all_threads": round(qn_s, 2),
                                "elements_all_threads": nel, "bytes_per_elem": 4.5625},
            "gemm_fp64": {"GFLOPs_1_thread": round(flops / g1_s / 1e9, 2), "s_1_thread": round(g1_s, 2),
                          "GFLOPs_all_threads": round(flops / gn_s / 1e9, 2),
                          "s_all_threads": round(gn_s, 2), "flop": flops},
            "full_step_s_estimate": round(qn_s + full_flops / (flops / gn_s), 1)}


if __name__ == "__main__":
    main()
