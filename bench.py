#!/usr/bin/env python3
"""Throughput of the Rollout-ResQ FP4 linear layer on one MI355X.

A default run prints one JSON line whose headline (value, roofline, cpu_baseline) is the
default workload below, and which carries, under one key each (EXTRA_ENTRIES), the same
measurement of the rest of the metric taken in the same process: MXFP4 on the same block,
the Qwen2.5-7B block at m = 512 with the channel, 32x64-block and element-wise residuals in
both formats, the m = 8192 prefill linears and the m = 8192 training backward in both formats.

A step is one rollout forward of every linear projection of one transformer block (the hot
path of Eq. 4): for each linear, quantize the bf16 activations, form and quantize the
residual, apply S, and run the FP4 GEMM with the residual term, writing float32 Y.  Q(W) is
computed once before timing: the weights change once per policy update, not per decode step.

Default workload: the four linears of one Qwen2.5-3B block (qkv 2048->2560, o 2048->2048,
gate_up 2048->22016, down 11008->2048) at m = 256 tokens, HiF4 with the S_2:4 residual,
seeded synthetic bf16 activations with 1% outlier channels (x50) and N(0, 0.02) weights.

Steps are timed as eager launches on one stream (--graph 1 also times HIP graph replays of
the same launches and reports them beside).  Inputs are resident in HBM when timing starts.  Weight and activation copies rotate across
steps so that the 256 MB last-level cache cannot serve a step from the previous one.

Prints one JSON line: the layer's algorithmic TFLOP/s (value), the roofline of the dominant
kernel (the GEMM, timed with HIP events on its stream through the library's profiler) and
the oracle timed on this host on a bounded sample of the same workload (cpu_baseline).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP4_PEAK_TFLOPS = 10100.0      # MI355X dense MXFP4 / MXFP6 MFMA
LLC_BYTES = 256 << 20          # MI355X last-level (Infinity) cache

BYTES_PER_ELEM = {"hif4": 36 / 64, "mxfp4": 17 / 32}  # codes + block scales
METRIC = "ResQ FP4 linear TFLOP/s + % roofline (HBM GB/s decode, MFMA FP4 prefill)"
DEFAULT_WORKLOAD = "qwen3b_layer_m256"
# Entries measured after the headline in a default run: (key, workload, format, sparsity)
EXTRA_ENTRIES = (
    ("qwen3b_layer_m256_mxfp4", "qwen3b_layer_m256", "mxfp4", "2:4"),
    ("qwen7b_layer_m512_hif4_block", "qwen7b_layer_m512", "hif4", "block32x64_50"),
    ("qwen7b_layer_m512_mxfp4_block", "qwen7b_layer_m512", "mxfp4", "block32x64_50"),
    ("qwen7b_layer_m512_hif4_unstructured", "qwen7b_layer_m512", "hif4", "unstructured50"),
    ("qwen7b_layer_m512_mxfp4_unstructured", "qwen7b_layer_m512", "mxfp4", "unstructured50"),
    ("qwen7b_layer_m512_hif4_channel", "qwen7b_layer_m512", "hif4", "channel50"),
    ("qwen7b_layer_m512_mxfp4_channel", "qwen7b_layer_m512", "mxfp4", "channel50"),
    ("qwen7b_prefill_m8192_hif4", "qwen7b_prefill_m8192", "hif4", "2:4"),
    ("qwen7b_prefill_m8192_mxfp4", "qwen7b_prefill_m8192", "mxfp4", "2:4"),
    ("qwen3b_gateup_bwd_m8192_hif4", "qwen3b_gateup_bwd_m8192", "hif4", "none"),
    ("qwen3b_gateup_bwd_m8192_mxfp4", "qwen3b_gateup_bwd_m8192", "mxfp4", "none"),
    # the mixed-precision alternatives of Table 1 on the default block
    ("qwen3b_layer_m256_hif4_w4a16", "qwen3b_layer_m256", "hif4", "w4a16"),
    ("qwen3b_layer_m256_hif4_w16a4", "qwen3b_layer_m256", "hif4", "w16a4"),
    ("qwen3b_layer_m256_mxfp4_w4a16", "qwen3b_layer_m256", "mxfp4", "w4a16"),
    ("qwen3b_layer_m256_mxfp4_w16a4", "qwen3b_layer_m256", "mxfp4", "w16a4"),
)


def kept_fraction(sp):
    """Nominal fraction of the residual a sparsity keeps: k/g for "k:g", p/100 for the
    "channel<p>", "block32x64_<p>" and "unstructured<p>" levels."""
    if sp in ("none", "identity"):
        return 0.0 if sp == "none" else 1.0
    if ":" in sp:
        k, g = (int(v) for v in sp.split(":"))
        return k / g
    return int(sp.replace("block32x64_", "").replace("channel", "").replace("unstructured", "")) / 100


def alg_flops(m, d, n, sp):
    """Sec. 5.4: 2mdn for the main GEMM; a 50% residual adds mdn, the dense one 2mdn (other
    levels: their kept fraction of 2mdn)."""
    return 2 * m * d * n + round(2 * m * d * n * kept_fraction(sp))


def executed_flops(m, d, n, sp):
    """Sec. 5.4 work as the GEMM executes it on gfx950: 2mdn per term; every residual kind
    runs as a dense FP4 operand (no FP4 sparse MFMA), so a residual adds a full 2mdn."""
    return 2 * m * d * n * (1 if sp == "none" else 2)


def issued_mfma_flops(m, d, n, fmt, sp):
    """MFMA work the GEMM issues at the FP4/FP6 rate: the executed work, twice for HiF4
    (each HiF4 term runs as two E2M3 operands, hi and lo, so its level-1 scale fits)."""
    return executed_flops(m, d, n, sp) * (2 if fmt == "hif4" else 1)


def step_bytes(m, d, n, fmt, y_bytes=4):
    """Algorithmic HBM bytes of one linear: X (bf16) in, Q(W) in, Y (fp32 or bf16) out."""
    return 2 * m * d + BYTES_PER_ELEM[fmt] * n * d + y_bytes * m * n


def gemm_bytes(m, d, n, fmt, sp, y_bytes=4):
    """Algorithmic bytes of the GEMM launch: Q(W), Q(X) and S(Q(dX)) read once, Y written."""
    terms = 1 if sp == "none" else 2
    return BYTES_PER_ELEM[fmt] * (n * d + terms * m * d) + y_bytes * m * n


def gemm_traffic(workload, fmt, sp, out="f32"):
    """HBM bytes per GEMM launch from the committed rocprofv3 counter summary, or None when
    the summary does not cover this workload or the GEMM source (gemm.hip and gemm_geo.h)
    changed since it was taken."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "gemm_traffic.json")))
        h = hashlib.sha256()
        for f in ("gemm.hip", "gemm_geo.h"):  # the GEMM kernel's sources
            h.update(open(os.path.join(ROOT, "paper_2607_26515_amd", "csrc", f), "rb").read())
    except OSError:
        return None
    if rec.get("gemm_source_sha256") != h.hexdigest():
        return None
    key = f"{workload}/{fmt}/{sp}" + ("" if out == "f32" else f"/{out}")
    entry = rec.get("entries", {}).get(key)
    return None if entry is None else round(entry["bytes_per_launch"])


def cpu_baseline(wl, fmt, sp, n_sample, n_rows, min_seconds):
    """The oracle, as it stands, on a bounded sample of the same workload (host cores)."""
    import numpy as np
    from oracle import formats as F
    from oracle import resq as Q
    from synth import bf16_bits_to_f32, workload_tensors

    cores = len(os.sched_getaffinity(0))
    blas_threads = None
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=None)
    except Exception:
        pass
    rows = min(wl.m, n_rows)
    prepared = []
    for lin in wl.linears:
        t = workload_tensors(wl, lin, m=rows, n_w=n_sample)
        if wl.backward:
            xb, wb, gb = t
            prepared.append((bf16_bits_to_f32(xb), bf16_bits_to_f32(wb[:n_sample]),
                             bf16_bits_to_f32(gb[:, :n_sample])))
        else:
            xb, wb = t
            w = bf16_bits_to_f32(wb[:n_sample])
            what = F.dequantize(fmt, *F.quantize(fmt, w))  # Q(W): once per policy update, untimed
            prepared.append((bf16_bits_to_f32(xb), what, None))
    flops = 0
    t0 = time.perf_counter()
    reps = 0
    while True:
        for x, w, gy in prepared:
            if wl.backward:
                Q.resq_backward(fmt, gy, x, w)
                flops += 4 * x.shape[0] * x.shape[1] * w.shape[0]
            else:
                out = Q.resq_quantize_residual(fmt, sp, x)
                y = out["xhat"] @ w.T
                if sp != "none":
                    y = y + out["srhat"] @ w.T
                y.astype(np.float32)
                flops += alg_flops(x.shape[0], x.shape[1], w.shape[0], sp)
        reps += 1
        if time.perf_counter() - t0 >= min_seconds:
            break
    dt = time.perf_counter() - t0
    what_ = ("dY, X and W restricted to" if wl.backward else "X restricted to")
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(blas_threads or cores),
        "kind": "oracle",
        "sample": (f"{wl.name}: {what_} the first {rows} rows and the first {n_sample} output "
                   f"features of every linear, {reps} repetition(s), {dt:.1f} s"
                   f"{'' if wl.backward else '; Q(W) untimed'}; numpy fp64 (quantizers "
                   f"single-threaded, matmul on {blas_threads or '?'} BLAS threads of {cores} cores)"),
    }


def bench_diagnostics(args, P, torch, np, wl, fmt, dev, sptr):
    """--op diagnostics: resq_diagnostics (the Figs. 2-4 statistics) over every linear's input
    X of the workload; algorithmic bytes = X read once (2 B per element)."""
    from synth import workload_tensors
    f = P.FORMATS[fmt]
    per_copy = sum(2 * wl.m * l.d for l in wl.linears)
    copies = int(min(64, max(2, -(-2 * LLC_BYTES // per_copy) + 1)))
    ws_bytes = max(P.resq_workspace_size(P.OP_DIAGNOSTICS, f, 0, wl.m, l.d, 0) for l in wl.linears)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    stats = torch.empty(len(P.DIAG_STATS), dtype=torch.float64, device=dev)
    xs = []
    for lin in wl.linears:
        xb, _ = workload_tensors(wl, lin)
        x0 = torch.from_numpy(xb.view(np.int16)).to(dev)
        xs.append((lin, [x0.clone() for _ in range(copies)]))
    lib = P.load()
    thr = args.outlier_threshold

    def step(i):
        for lin, xc in xs:
            rc = lib.resq_diagnostics(f, int(xc[i % copies].data_ptr()), wl.m, lin.d, lin.d, thr,
                                      int(stats.data_ptr()), int(ws.data_ptr()), ws_bytes, sptr)
            if rc != 0:
                raise P.ResqError(f"resq_diagnostics: {P.resq_last_error()}", rc)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    P.resq_profile_enable(True)
    P.resq_profile_reset()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    n_launch, k_ms = P.resq_profile_read("diagnostics")
    P.resq_profile_enable(False)
    nbytes = per_copy
    launch_s = k_ms / n_launch * 1e-3
    achieved = nbytes / len(wl.linears) / launch_s / 1e9
    out = {
        "metric": "Figs. 2-4 activation statistics pass (zeros, outlier blocks, S_2:4 error), GB/s of X",
        "value": round(nbytes * args.steps / dt / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3 / args.steps, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "fp4", "data": "synthetic",
        "config": {"workload": wl.name, "format": fmt, "op": "diagnostics", "m": wl.m,
                   "inputs": {l.name: [wl.m, l.d] for l in wl.linears},
                   "outlier_threshold": thr, "copies_rotated": copies},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": f"diag_kernel + diag_finish_kernel ({len(wl.linears)} calls per step)",
                     "alg_bytes_per_launch": round(nbytes / len(wl.linears)),
                     "avg_launch_us": round(launch_s * 1e6, 2)},
    }
    if not args.no_cpu_baseline:
        from oracle import diagnostics as OD
        from synth import bf16_bits_to_f32
        rows = min(wl.m, args.cpu_sample_rows)
        xs_cpu = [bf16_bits_to_f32(workload_tensors(wl, l, m=rows)[0]) for l in wl.linears]
        t0, reps, nb = time.perf_counter(), 0, 0
        while True:
            for x in xs_cpu:
                OD.diagnostics(fmt, x, thr)
                nb += 2 * x.size
            reps += 1
            if time.perf_counter() - t0 >= args.cpu_seconds:
                break
        cdt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(nb / cdt / 1e9, 4), "unit": "GB/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{wl.name}: the first {rows} rows of every linear's X, "
                                         f"{reps} repetition(s), {cdt:.1f} s, numpy (single-threaded)"}
    print(json.dumps(out), flush=True)
    return 0


def bench_swiglu_down(args, P, torch, np, wl, fmt, sp, dev, sptr):
    """--op swiglu_down: the workload's down projection with its SwiGLU input formed inside the
    quantization pass (resq_linear_fwd_prepared_swiglu, G and U bf16), against the same linear
    fed by a separate torch silu * mul kernel that writes X (bf16) first."""
    from synth import activations, rng_tree, workload_tensors
    lin = next(l for l in wl.linears if l.name == "down")
    m, d, n = wl.m, lin.d, lin.n
    f, s = P.FORMATS[fmt], P.sparsity_code(sp)
    _, wb = workload_tensors(wl, lin)
    w0 = torch.from_numpy(wb.view(np.int16)).to(dev)
    qc, qs = P.quantize(w0, fmt, axis=1)
    per_copy = P.resq_prepared_weights_size(f, n, d) + 2 * 2 * m * d
    copies = int(min(32, max(2, -(-2 * LLC_BYTES // per_copy) + 1)))
    wps = [P.prepare_weights(qc, qs, fmt) for _ in range(copies)]
    rg, ru = rng_tree(7, 2)
    g0 = torch.from_numpy(activations(rg, m, d, 0.01, 8.0).view(np.int16)).to(dev)
    u0 = torch.from_numpy(activations(ru, m, d, 0.01, 30.0).view(np.int16)).to(dev)
    gs = [g0.clone() for _ in range(copies)]
    us = [u0.clone() for _ in range(copies)]
    y = torch.empty((m, n), dtype=torch.float32, device=dev)
    ws_bytes = P.resq_workspace_size(P.OP_LINEAR_FWD_PREPARED, f, s, m, d, n)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    lib = P.load()

    def fused(i):
        c = i % copies
        rc = lib.resq_linear_fwd_prepared_swiglu(f, s, int(gs[c].data_ptr()), int(us[c].data_ptr()),
                                                 P.IN_BF16, m, d, d, d, int(wps[c].data_ptr()), n,
                                                 int(y.data_ptr()), n, int(ws.data_ptr()), ws_bytes, sptr)
        if rc != 0:
            raise P.ResqError(f"resq_linear_fwd_prepared_swiglu: {P.resq_last_error()}", rc)

    def unfused(i):
        c = i % copies
        g, u = gs[c].view(torch.bfloat16), us[c].view(torch.bfloat16)
        x = (torch.nn.functional.silu(g.float()) * u.float()).to(torch.bfloat16).view(torch.int16)
        rc = lib.resq_linear_fwd_prepared(f, s, int(x.data_ptr()), m, d, d, int(wps[c].data_ptr()), n,
                                          int(y.data_ptr()), n, int(ws.data_ptr()), ws_bytes, sptr)
        if rc != 0:
            raise P.ResqError(f"resq_linear_fwd_prepared: {P.resq_last_error()}", rc)

    def timed(fn):
        for i in range(args.warmup):
            fn(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            fn(i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / args.steps

    t_f, t_u = timed(fused), timed(unfused)
    P.resq_profile_enable(True)
    P.resq_profile_reset()
    for i in range(args.steps):
        fused(i)
    torch.cuda.synchronize()
    res = P.resq_profile_read("residual")
    P.resq_profile_enable(False)
    flops = alg_flops(m, d, n, sp)
    out = {
        "metric": "ResQ down projection with the SwiGLU producer fused into its quantization pass, TFLOP/s",
        "value": round(flops / t_f / 1e12, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(t_f * 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "fp4",
        "data": "synthetic",
        "config": {"workload": wl.name, "linear": f"down {d}->{n}", "m": m, "format": fmt,
                   "sparsity": sp, "op": "swiglu_down", "inputs": "G, U bf16", "copies_rotated": copies},
        "unfused_ms": round(t_u * 1e3, 5),
        "speedup_vs_unfused": round(t_u / t_f, 3),
        "fused_activation_pass_us": round(res[1] / res[0] * 1e3, 2) if res[0] else None,
    }
    print(json.dumps(out), flush=True)
    return 0


def bench_rmsnorm_in(args, P, torch, np, wl, fmt, sp, dev, sptr):
    """--op rmsnorm_in: the workload's qkv and gate_up projections (the linears that take an
    RMSNorm output) with the RMSNorm of H formed inside the quantization pass
    (resq_linear_fwd_prepared_rmsnorm: one launch for the per-row factors, then the activation
    pass and the GEMM), against the same linears fed by a torch RMSNorm (float32 statistics)
    that writes X (bf16) first.  A step is both linears."""
    from synth import activations, rng_tree, workload_tensors
    lins = [l for l in wl.linears if l.name in ("qkv", "gate_up")]
    m = wl.m
    f, s = P.FORMATS[fmt], P.sparsity_code(sp)
    eps = 1e-6
    per_copy = sum(P.resq_prepared_weights_size(f, l.n, l.d) + 2 * m * l.d for l in lins)
    copies = int(min(32, max(2, -(-2 * LLC_BYTES // per_copy) + 1)))
    state = []
    for k, lin in enumerate(lins):
        _, wb = workload_tensors(wl, lin)
        qc, qs = P.quantize(torch.from_numpy(wb.view(np.int16)).to(dev), fmt, axis=1)
        rh, rg = rng_tree(11 + k, 2)
        h0 = torch.from_numpy(activations(rh, m, lin.d, 0.01, 20.0).view(np.int16)).to(dev)
        gamma = (1.0 + 0.2 * torch.randn(lin.d, generator=torch.Generator().manual_seed(k))) \
            .to(torch.bfloat16).view(torch.int16).to(dev)
        ws_bytes = P.resq_workspace_size(P.OP_LINEAR_FWD_RMSNORM, f, s, m, lin.d, lin.n)
        state.append({
            "lin": lin, "wps": [P.prepare_weights(qc, qs, fmt) for _ in range(copies)],
            "hs": [h0.clone() for _ in range(copies)], "gamma": gamma,
            "y": torch.empty((m, lin.n), dtype=torch.float32, device=dev),
            "ws": torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev), "ws_bytes": ws_bytes,
        })
    lib = P.load()

    def fused(i):
        c = i % copies
        for st in state:
            l = st["lin"]
            rc = lib.resq_linear_fwd_prepared_rmsnorm(
                f, s, int(st["hs"][c].data_ptr()), m, l.d, l.d, int(st["gamma"].data_ptr()), eps,
                int(st["wps"][c].data_ptr()), l.n, int(st["y"].data_ptr()), l.n,
                int(st["ws"].data_ptr()), st["ws_bytes"], sptr)
            if rc != 0:
                raise P.ResqError(f"resq_linear_fwd_prepared_rmsnorm: {P.resq_last_error()}", rc)

    def unfused(i):
        c = i % copies
        for st in state:
            l = st["lin"]
            h = st["hs"][c].view(torch.bfloat16).float()
            r = torch.rsqrt(h.pow(2).mean(-1, keepdim=True) + eps)
            x = (h * r * st["gamma"].view(torch.bfloat16).float()).to(torch.bfloat16).view(torch.int16)
            rc = lib.resq_linear_fwd_prepared(f, s, int(x.data_ptr()), m, l.d, l.d,
                                              int(st["wps"][c].data_ptr()), l.n, int(st["y"].data_ptr()),
                                              l.n, int(st["ws"].data_ptr()), st["ws_bytes"], sptr)
            if rc != 0:
                raise P.ResqError(f"resq_linear_fwd_prepared: {P.resq_last_error()}", rc)

    def timed(fn):
        for i in range(args.warmup):
            fn(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            fn(i)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / args.steps

    t_f, t_u = timed(fused), timed(unfused)
    P.resq_profile_enable(True)
    P.resq_profile_reset()
    for i in range(args.steps):
        fused(i)
    torch.cuda.synchronize()
    res = P.resq_profile_read("residual")
    P.resq_profile_enable(False)
    flops = sum(alg_flops(m, l.d, l.n, sp) for l in lins)
    out = {
        "metric": "ResQ qkv and gate_up projections with the RMSNorm producer fused into their "
                  "quantization pass, TFLOP/s",
        "value": round(flops / t_f / 1e12, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(t_f * 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "fp4",
        "data": "synthetic",
        "config": {"workload": wl.name, "linears": {l.name: [l.d, l.n] for l in lins}, "m": m,
                   "format": fmt, "sparsity": sp, "op": "rmsnorm_in", "inputs": "H, gamma bf16",
                   "eps": eps, "copies_rotated": copies},
        "unfused_ms": round(t_u * 1e3, 5),
        "speedup_vs_unfused": round(t_u / t_f, 3),
        "rms_and_activation_pass_us_per_step": round(res[1] / args.steps * 1e3, 2),
    }
    print(json.dumps(out), flush=True)
    return 0


BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA


def measure_mixed(args, P, torch, np, wl, fmt, op, dev, sptr, cpu_seconds):
    """The mixed-precision rollout linears of Table 1 on every linear of a forward workload:
    op "w4a16" (Y = X Q(W)^T, Q(W) K-major, computed once before timing) or "w16a4" (Y =
    Q(X) W^T, W bf16).  Both run on the bf16 MFMA; the roofline is the larger of the HBM time
    of their algorithmic bytes and the bf16 MFMA time of 2mdn per linear."""
    from synth import workload_tensors
    f = P.FORMATS[fmt]
    w4 = op == "w4a16"
    wbytes = BYTES_PER_ELEM[fmt] if w4 else 2.0
    per_copy = sum(wbytes * l.n * l.d + 2 * wl.m * l.d for l in wl.linears)
    copies = int(min(64, max(2, -(-2 * LLC_BYTES // int(per_copy)) + 1)))
    ws_bytes = max(P.resq_workspace_size(P.OP_LINEAR_W16A4, f, 0, wl.m, l.d, l.n) for l in wl.linears)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    lib = P.load()
    state = []
    for lin in wl.linears:
        xb, wb = workload_tensors(wl, lin)
        x0 = torch.from_numpy(xb.view(np.int16)).to(dev)
        w0 = torch.from_numpy(wb.view(np.int16)).to(dev)
        xs = [x0.clone() for _ in range(copies)]
        ops = [P.quantize(w0, fmt, axis=1) for _ in range(copies)] if w4 else [w0.clone() for _ in range(copies)]
        y = torch.empty((wl.m, lin.n), dtype=torch.float32, device=dev)
        state.append((lin, xs, ops, y))
        del x0, w0
    torch.cuda.synchronize()

    def step(i):
        c = i % copies
        for lin, xs, ops, y in state:
            x = xs[c]
            if w4:
                qc, qs = ops[c]
                rc = lib.resq_linear_w4a16(f, int(x.data_ptr()), wl.m, lin.d, lin.d, int(qc.data_ptr()),
                                           int(qs.data_ptr()), lin.n, int(y.data_ptr()), lin.n, sptr)
            else:
                rc = lib.resq_linear_w16a4(f, int(x.data_ptr()), wl.m, lin.d, lin.d, int(ops[c].data_ptr()),
                                           lin.d, lin.n, int(y.data_ptr()), lin.n, int(ws.data_ptr()),
                                           ws_bytes, sptr)
            if rc != 0:
                raise P.ResqError(f"resq_linear_{op}: {P.resq_last_error()}", rc)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    P.resq_profile_enable(True)
    P.resq_profile_reset()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    n_mixed, ms_mixed = P.resq_profile_read("mixed")
    n_q, ms_q = P.resq_profile_read("quant_rows")
    P.resq_profile_enable(False)
    del state
    torch.cuda.empty_cache()
    flops = sum(2 * wl.m * l.d * l.n for l in wl.linears)
    gbytes = sum(2 * wl.m * l.d + wbytes * l.n * l.d + 4 * wl.m * l.n for l in wl.linears)
    gemm_s = ms_mixed / args.steps * 1e-3
    t_hbm, t_mfma = gbytes / (HBM_PEAK_GBS * 1e9), flops / (BF16_PEAK_TFLOPS * 1e12)
    mfma_bound = t_mfma > t_hbm
    achieved = (flops / gemm_s / 1e12) if mfma_bound else (gbytes / gemm_s / 1e9)
    peak = BF16_PEAK_TFLOPS if mfma_bound else HBM_PEAK_GBS
    res = {
        "value": round(flops * args.steps / dt / 1e12, 3),
        "unit": "TFLOP/s",
        "ms_per_step": round(dt * 1e3 / args.steps, 5),
        "config": {"workload": wl.name, "format": fmt, "op": op,
                   "precision": "weights FP4, activations bf16" if w4 else "activations FP4, weights bf16",
                   "m": wl.m, "linears": {l.name: [l.d, l.n] for l in wl.linears}, "copies_rotated": copies},
        "kernel_ms_per_step": {"mixed_gemm": round(ms_mixed / args.steps, 5),
                               "quant_rows": round(ms_q / args.steps, 5)},
        "roofline": {"bound": "mfma" if mfma_bound else "hbm", "achieved": round(achieved, 1), "peak": peak,
                     "unit": "TFLOP/s" if mfma_bound else "GB/s", "frac": round(achieved / peak, 4),
                     "traffic": None,
                     "kernel": f"mixed_gemm_kernel ({len(wl.linears)} launches per step, bf16 MFMA)",
                     "alg_bytes_per_launch": round(gbytes / len(wl.linears)),
                     "alg_flops_per_launch": round(flops / len(wl.linears)),
                     "avg_launch_us": round(gemm_s / len(wl.linears) * 1e6, 2)},
    }
    if not args.no_cpu_baseline:
        from oracle import resq as Q
        from synth import bf16_bits_to_f32
        rows, cols = min(wl.m, args.cpu_sample_rows), args.cpu_sample_cols
        sample = []
        for lin in wl.linears:
            xb, wb = workload_tensors(wl, lin, m=rows, n_w=cols)
            sample.append((bf16_bits_to_f32(xb), bf16_bits_to_f32(wb)))
        fn = Q.w4a16_forward if w4 else Q.w16a4_forward
        t0, reps, fl = time.perf_counter(), 0, 0
        while True:
            for x, w in sample:
                fn(fmt, x, w)
                fl += 2 * x.shape[0] * x.shape[1] * w.shape[0]
            reps += 1
            if time.perf_counter() - t0 >= cpu_seconds:
                break
        cdt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": fl / cdt / 1e12, "unit": "TFLOP/s",
                               "cores": len(os.sched_getaffinity(0)), "kind": "oracle",
                               "sample": f"{wl.name}: the first {rows} rows and {cols} output features of "
                                         f"every linear, {reps} repetition(s), {cdt:.1f} s; numpy fp64"}
    return res


def setup_forward(P, torch, np, wl, fmt, sp, dev, sptr, out="f32"):
    """Inputs resident in HBM (enough rotating copies to defeat the last-level cache) and a
    step function running every linear of the workload through resq_linear_fwd_prepared
    (float32 Y) or resq_linear_fwd_prepared_bf16 (bf16 Y)."""
    from synth import workload_tensors
    f, s = P.FORMATS[fmt], P.sparsity_code(sp)
    per_copy = sum(P.resq_prepared_weights_size(f, l.n, l.d) + 2 * wl.m * l.d for l in wl.linears)
    copies = int(min(64, max(2, -(-2 * LLC_BYTES // int(per_copy)) + 1)))
    ws_bytes = max(P.resq_workspace_size(3, f, s, wl.m, l.d, l.n) for l in wl.linears)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    lin_state = []
    for lin in wl.linears:
        xb, wb = workload_tensors(wl, lin)
        x0 = torch.from_numpy(xb.view(np.int16)).to(dev)
        w0 = torch.from_numpy(wb.view(np.int16)).to(dev)
        xs, wps = [], []
        for c in range(copies):
            xs.append(x0.clone())
            qc, qs = P.quantize(w0, fmt, axis=1)  # Q(W) and its GEMM layout: once per policy update
            wps.append(P.prepare_weights(qc, qs, fmt))
            del qc, qs
        del w0, x0
        y = torch.empty((wl.m, lin.n), dtype=torch.float32 if out == "f32" else torch.int16,
                        device=dev)
        lin_state.append(dict(lin=lin, xs=xs, wps=wps, y=y, xp=[int(t.data_ptr()) for t in xs],
                              wp=[int(t.data_ptr()) for t in wps]))
    torch.cuda.synchronize()
    lib = P.load()
    entry = lib.resq_linear_fwd_prepared if out == "f32" else lib.resq_linear_fwd_prepared_bf16

    def run_linear(st, i):
        lin, c = st["lin"], i % copies
        rc = entry(f, s, st["xp"][c], wl.m, lin.d, lin.d, st["wp"][c], lin.n,
                   int(st["y"].data_ptr()), lin.n, int(ws.data_ptr()), ws_bytes, sptr)
        if rc != 0:
            raise P.ResqError(f"{entry.__name__}: {P.resq_last_error()}", rc)

    return lin_state, run_linear, copies


def setup_backward(P, torch, np, wl, fmt, dev, sptr):
    """dY, X, W resident in HBM (rotating copies) and a step running resq_linear_bwd."""
    from synth import workload_tensors
    f = P.FORMATS[fmt]
    lin = wl.linears[0]
    m, d, n = wl.m, lin.d, lin.n
    per_copy = 2 * (m * n + m * d + n * d)
    copies = int(min(16, max(2, -(-2 * LLC_BYTES // per_copy) + 1)))
    xb, wb, gb = workload_tensors(wl, lin)
    base = [torch.from_numpy(a.view(np.int16)).to(dev) for a in (gb, xb, wb)]
    sets = [[t.clone() for t in base] for _ in range(copies)]
    del base
    dx = torch.empty((m, d), dtype=torch.float32, device=dev)
    dw = torch.empty((n, d), dtype=torch.float32, device=dev)
    ws_bytes = P.resq_workspace_size(P.OP_LINEAR_BWD, f, 0, m, d, n)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    lib = P.load()
    st = dict(lin=lin)

    def run_linear(_st, i):
        g, x, w = sets[i % copies]
        rc = lib.resq_linear_bwd(f, int(g.data_ptr()), int(x.data_ptr()), int(w.data_ptr()), m, d, n,
                                 int(dx.data_ptr()), int(dw.data_ptr()), int(ws.data_ptr()), ws_bytes,
                                 sptr)
        if rc != 0:
            raise P.ResqError(f"resq_linear_bwd: {P.resq_last_error()}", rc)

    return [st], run_linear, copies


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--format", default="hif4", choices=["hif4", "mxfp4"])
    ap.add_argument("--sparsity", default="2:4")
    ap.add_argument("--op", default="linear",
                    choices=["linear", "diagnostics", "swiglu_down", "rmsnorm_in", "w4a16", "w16a4"],
                    help="linear: the ResQ layer step; diagnostics: the Figs. 2-4 statistics pass; "
                         "swiglu_down: the down projection with its SwiGLU input fused; "
                         "rmsnorm_in: the qkv and gate_up projections with their RMSNorm input "
                         "fused; w4a16 / w16a4: the mixed-precision linears of Table 1 on every "
                         "linear")
    ap.add_argument("--outlier-threshold", type=float, default=10.0,
                    help="--op diagnostics: |x| above which a block counts as holding an outlier")
    ap.add_argument("--out", default="f32", choices=["f32", "bf16"],
                    help="forward output type: float32, or its bf16 rounding written by the GEMM")
    ap.add_argument("--graph", type=int, default=0, choices=[0, 1],
                    help="linear op: time the steps as eager launches (0), or also as HIP graph "
                         "replays, one graph per rotated input copy (1; measured slower on "
                         "ROCm 7, reported beside the eager time, which stays the value)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="measure only the selected workload (a default run also measures the "
                         "entries of EXTRA_ENTRIES and adds them to the JSON line)")
    ap.add_argument("--extra-cpu-seconds", type=float, default=4.0,
                    help="oracle time per extra entry's cpu_baseline")
    ap.add_argument("--cpu-sample-cols", type=int, default=1024)
    ap.add_argument("--cpu-sample-rows", type=int, default=512)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-sized device buffer once (HBM counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: the benchmark runs the layer on one GPU; --gpus {args.gpus} is not "
              f"supported (how the layer shards over several GPUs is described, not run).",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2607_26515_amd as P
    from synth import WORKLOADS

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n}), flush=True)
        return 0
    P.load()  # fails loudly when libresq.so is missing
    dev = torch.device("cuda:0")
    # one stream of the default priority for the whole run (graph capture needs a stream
    # other than the null stream)
    run_stream = torch.cuda.Stream()
    torch.cuda.set_stream(run_stream)
    sptr = int(run_stream.cuda_stream)
    wl = WORKLOADS[args.workload]
    fmt = args.format
    if args.op == "diagnostics":
        if wl.backward:
            print("bench.py: --op diagnostics needs a forward workload", file=sys.stderr)
            return 2
        return bench_diagnostics(args, P, torch, np, wl, args.format, dev, sptr)
    if args.op == "swiglu_down":
        if wl.backward or not any(l.name == "down" for l in wl.linears):
            print("bench.py: --op swiglu_down needs a forward workload with a down projection", file=sys.stderr)
            return 2
        return bench_swiglu_down(args, P, torch, np, wl, args.format, args.sparsity, dev, sptr)
    if args.op == "rmsnorm_in":
        if wl.backward or not any(l.name in ("qkv", "gate_up") for l in wl.linears):
            print("bench.py: --op rmsnorm_in needs a forward workload with a qkv or gate_up "
                  "projection", file=sys.stderr)
            return 2
        return bench_rmsnorm_in(args, P, torch, np, wl, args.format, args.sparsity, dev, sptr)
    if args.op in ("w4a16", "w16a4"):
        if wl.backward:
            print(f"bench.py: --op {args.op} needs a forward workload", file=sys.stderr)
            return 2
        r = measure_mixed(args, P, torch, np, wl, fmt, args.op, dev, sptr, args.cpu_seconds)
        out = {"metric": f"{args.op} rollout linear (Table 1) TFLOP/s", "value": r.pop("value"),
               "unit": r.pop("unit"), "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
               "ms_per_step": r.pop("ms_per_step"), "higher_is_better": True, "scaling": "weak",
               "vs_baseline": None, "dtype": "bf16", "data": "synthetic"}
        out.update(r)
        print(json.dumps(out), flush=True)
        return 0
    result = measure(args, P, torch, np, wl, fmt, args.sparsity, args.out, dev, sptr, run_stream,
                     args.cpu_seconds, graph=bool(args.graph))
    out = {
        "metric": METRIC,
        "value": result.pop("value"),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": result.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp4",
        "data": "synthetic",
    }
    out.update(result)
    if not args.no_extra and args.workload == DEFAULT_WORKLOAD:
        # the rest of the metric, measured in the same process: the other format on the
        # same workload, the m = 512 block, prefill and the training backward
        for name, wl_name, f, sp in EXTRA_ENTRIES:
            torch.cuda.empty_cache()
            if wl_name == args.workload and f == fmt and sp == args.sparsity:
                continue  # the headline itself
            if sp in ("w4a16", "w16a4"):
                e = measure_mixed(args, P, torch, np, WORKLOADS[wl_name], f, sp, dev, sptr,
                                  args.extra_cpu_seconds)
            else:
                e = measure(args, P, torch, np, WORKLOADS[wl_name], f, sp, "f32", dev, sptr, run_stream,
                            args.extra_cpu_seconds)
            out[name] = e
            print(f"bench.py: {name}: {e['ms_per_step']} ms/step, roofline frac "
                  f"{e['roofline']['frac']}", file=sys.stderr, flush=True)
    print(json.dumps(out), flush=True)
    return 0


def measure(args, P, torch, np, wl, fmt, sparsity, out_t, dev, sptr, run_stream, cpu_seconds,
            graph=False):
    """One workload: setup (inputs resident in HBM, rotated copies), warmup, the timed steps,
    kernel times from the library profiler, roofline of the GEMM and the oracle baseline.
    Returns the result fields (value, ms_per_step, config, roofline, cpu_baseline, ...)."""
    sp = "none" if wl.backward else sparsity
    out_t = "f32" if wl.backward else out_t
    y_bytes = 4 if out_t == "f32" else 2
    if wl.backward:
        lin_state, run_linear, copies = setup_backward(P, torch, np, wl, fmt, dev, sptr)
    else:
        lin_state, run_linear, copies = setup_forward(P, torch, np, wl, fmt, sp, dev, sptr, out_t)

    def run_step(i):
        for st in lin_state:
            run_linear(st, i)

    def timed_loop(step):
        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            step(i)
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    dt = timed_loop(run_step)
    ms_per_step = dt * 1e3 / args.steps
    ms_graph = None
    if graph:
        # The same launches, captured once per rotated copy and replayed.
        graphs = []
        for c in range(copies):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=run_stream):
                run_step(c)
            graphs.append(g)
        ms_graph = timed_loop(lambda i: graphs[i % copies].replay()) * 1e3 / args.steps
        del graphs

    # ---- kernel times: HIP events on the launch stream via the library profiler ----
    kinds = ("quant_rows", "quant_cols", "pack_hif4", "gemm") if wl.backward else \
            ("residual", "pack_hif4", "select", "gemm")
    P.resq_profile_enable(True)
    P.resq_profile_reset()
    for i in range(args.steps):
        run_step(i)
    torch.cuda.synchronize()
    prof = {k: P.resq_profile_read(k) for k in kinds}
    per_linear = {}
    if len(lin_state) > 1:
        for st in lin_state:
            P.resq_profile_reset()
            for i in range(args.steps):
                run_linear(st, i)
            torch.cuda.synchronize()
            per_linear[st["lin"].name] = {k: round(P.resq_profile_read(k)[1] / args.steps * 1e3, 2)
                                          for k in kinds}
    P.resq_profile_enable(False)
    del lin_state, run_linear

    lins = wl.linears
    if wl.backward:
        flops = sum(4 * wl.m * l.d * l.n for l in lins)  # dX and dW, 2mdn each
        gexec = flops                                    # no residual in the backward
        gissued = flops * (2 if fmt == "hif4" else 1)
        gbytes = sum(BYTES_PER_ELEM[fmt] * 2 * (wl.m * l.n + l.n * l.d + wl.m * l.d)
                     + 4 * (wl.m * l.d + l.n * l.d) for l in lins)
        sbytes = sum(2 * (wl.m * l.n + wl.m * l.d + l.n * l.d) + 4 * (wl.m * l.d + l.n * l.d)
                     for l in lins)
        n_launch = 2 * len(lins)
    else:
        flops = sum(alg_flops(wl.m, l.d, l.n, sp) for l in lins)
        gexec = sum(executed_flops(wl.m, l.d, l.n, sp) for l in lins)
        gissued = sum(issued_mfma_flops(wl.m, l.d, l.n, fmt, sp) for l in lins)
        gbytes = sum(gemm_bytes(wl.m, l.d, l.n, fmt, sp, y_bytes) for l in lins)
        sbytes = sum(step_bytes(wl.m, l.d, l.n, fmt, y_bytes) for l in lins)
        n_launch = len(lins)
    value = flops * args.steps / dt / 1e12
    g_launch, g_ms = prof["gemm"]
    gemm_ms_step = g_ms / args.steps
    launch_s = gemm_ms_step / n_launch * 1e-3  # average GEMM launch
    exec_tflops = gexec / (gemm_ms_step * 1e-3) / 1e12
    hbm_gbs = gbytes / n_launch / launch_s / 1e9  # algorithmic bytes per launch / launch time
    mfma_bound = wl.backward or wl.m >= 2048
    roofline = {
        "bound": "mfma" if mfma_bound else "hbm",
        "achieved": round(exec_tflops if mfma_bound else hbm_gbs, 1),
        "peak": FP4_PEAK_TFLOPS if mfma_bound else HBM_PEAK_GBS,
        "unit": "TFLOP/s" if mfma_bound else "GB/s",
        "frac": round(exec_tflops / FP4_PEAK_TFLOPS if mfma_bound else hbm_gbs / HBM_PEAK_GBS, 4),
        "traffic": gemm_traffic(wl.name, fmt, sp, out_t),
        "kernel": f"gemm_kernel ({n_launch} launches per step)",
        "alg_bytes_per_launch": round(gbytes / n_launch),
        "exec_flops_per_launch": round(gexec / n_launch),
        "flops_counted": "executed: 2mnd per term, the residual as a dense FP4 operand (Sec. 5.4 on gfx950)",
        "avg_launch_us": round(launch_s * 1e6, 2),
        "hbm_gbs": round(hbm_gbs, 1),
        "exec_tflops": round(exec_tflops, 1),
        "exec_frac": round(exec_tflops / FP4_PEAK_TFLOPS, 4),
        "alg_tflops": round(flops / (gemm_ms_step * 1e-3) / 1e12, 1),
        "mfma_issued_tflops": round(gissued / (gemm_ms_step * 1e-3) / 1e12, 1),
    }
    res = {
        "value": round(value, 3),
        "ms_per_step": round(ms_per_step, 5),
        "config": {
            "workload": wl.name,
            "format": fmt,
            "sparsity": sp,
            "pass": "backward (dX, dW)" if wl.backward else "forward",
            "output": "float32" if out_t == "f32" else "bf16",
            "m": wl.m,
            "linears": {l.name: [l.d, l.n] for l in lins},
            "copies_rotated": copies,
        },
        "step_hbm": {
            "alg_bytes": int(sbytes),
            "achieved_gbs": round(sbytes / (ms_per_step * 1e-3) / 1e9, 1),
            "frac": round(sbytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        },
        "kernel_ms_per_step": {k: round(v[1] / args.steps, 5) for k, v in prof.items()},
        "per_linear_us": per_linear,
        "roofline": roofline,
    }
    if ms_graph is not None:
        res["ms_per_step_graph_replay"] = round(ms_graph, 5)
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, fmt, sp, args.cpu_sample_cols, args.cpu_sample_rows,
                                           cpu_seconds)
    return res


if __name__ == "__main__":
    sys.exit(main())
