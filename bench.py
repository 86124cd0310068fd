#!/usr/bin/env python3
"""Benchmark: fused bf16 GEMM + GELU-tanh/clamp tail on one MI355X.

Workload (the configuration the headline metric is quoted on):
x[1024, 8192] ~ N(0,1), W[8192, 8192] and b[8192] ~ U(±1/√8192), bf16 inputs,
y = clamp(GELU_tanh((x·Wᵀ + b)·0.5), −1, 1), bf16 output, fp32 accumulation.
One step = one fused launch over that batch, inputs resident in HBM.

Prints ONE JSON line with the fused kernel's TFLOP/s (``value``), its
roofline fraction against the dense bf16 MFMA peak, the unfused sequence
(vendor GEMM + one eager kernel per tail op) and the GEMM alone timed beside
it, and the fp64 CPU oracle timed on a bounded sample of rows.

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
                       [--workload gelu_clamp|gelu_clamp_e4m3|lse|silu_gn|tiny_f32|scale_lse_mish|gn_swish_mul_swish|
                                   gn_lrelu_sum|swish_sum_gn|moe_{prefill,decode}_{bf16,e4m3}|
                                   moe_finalize|add_rmsnorm|rope_kv]
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, published
PEAK_FP8_TFLOPS = 5000.0       # MI355X dense fp8 MFMA, published
PEAK_HBM_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ["fg_tile.hpp", "fg_epilogue.hpp", "fgemm.hip"]
MOE_KERNEL_SOURCES = ["fg_tile.hpp", "fg_quant.hpp", "moe.hip", "quant.hip"]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--warmup-seconds", type=float, default=1.0,
                    help="extra untimed work first, so clocks settle before timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target oracle sample time")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after the measurement, run a plain device-to-device copy of this many MiB "
                         "(3 times); its HBM counters calibrate rocprofv3 FETCH_SIZE/WRITE_SIZE")
    ap.add_argument("--workload", default="gelu_clamp",
                    choices=["gelu_clamp", "gelu_clamp_e4m3", "lse", "silu_gn", "tiny_f32", "scale_lse_mish",
                             "gn_swish_mul_swish", "gn_lrelu_sum", "swish_sum_gn", "moe_prefill_bf16",
                             "moe_prefill_e4m3", "moe_decode_bf16", "moe_decode_e4m3", "moe_finalize", "add_rmsnorm",
                             "rope_kv"],
                    help="gelu_clamp (default) is the headline workload; the others are the "
                         "remaining configurations, measured the same way")
    return ap.parse_args()


def kernel_source_hash(sources=KERNEL_SOURCES):
    """Hash of the kernel sources with comments and whitespace removed, so
    that committed counter summaries stay valid across comment edits but not
    across code changes."""
    import re
    h = hashlib.sha256()
    for f in sources:
        with open(os.path.join(ROOT, "paper_2606_02963_amd", "csrc", f), encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(name, sources=KERNEL_SOURCES):
    """HBM bytes per launch from committed rocprofv3 --pmc summaries
    (FETCH_SIZE + WRITE_SIZE, copy-kernel calibrated) if they were taken on
    the current kernel sources; None otherwise."""
    path = os.path.join(PROFILES, f"{name}.pmc.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        d = json.load(fh)
    if d.get("kernel_source_hash") != kernel_source_hash(sources):
        return None
    return d.get("hbm_bytes_per_launch")


def settle(fn, seconds, torch):
    """Run untimed work for about `seconds` so the clocks reach steady state."""
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            fn()
        torch.cuda.synchronize()


def time_steps(fn, steps, warmup, torch):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        fn()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps      # ms per step


def repeat_stats(fn, steps, torch, count=7):
    """Seven further timings of `steps` steps each, after the reported one:
    the median step time and the coefficient of variation across them (the
    run-to-run spread on one box; the reported value is the first timing)."""
    import statistics
    ms = [time_steps(fn, steps, 0, torch) for _ in range(count)]
    med = statistics.median(ms)
    cv = statistics.pstdev(ms) / statistics.fmean(ms)
    return {"count": count, "ms_per_step_median": round(med, 5), "cv": round(cv, 5)}


FGEMM_WORKLOADS = {"gelu_clamp": "bf16_gelu_clamp", "lse": "bf16_lse", "silu_gn": "bf16_silu_gn",
                   "tiny_f32": "tiny_f32_relu_x2", "scale_lse_mish": "bf16_scale_lse_mish",
                   "gn_swish_mul_swish": "bf16_gn_swish_mul_swish", "gn_lrelu_sum": "bf16_gn_lrelu_sum",
                   "swish_sum_gn": "bf16_swish_sum_gn", "gelu_clamp_e4m3": "e4m3_gelu_clamp"}
MOE_WORKLOADS = {"moe_prefill_bf16", "moe_prefill_e4m3", "moe_decode_bf16", "moe_decode_e4m3"}
TAIL_TEXT = {"bf16_gelu_clamp": "(x0.5, GELU_tanh, clamp[-1,1])", "bf16_lse": "(-0.25, row logsumexp)",
             "bf16_silu_gn": "(SiLU, GroupNorm 32x128)", "tiny_f32_relu_x2": "(ReLU, x2)",
             "bf16_scale_lse_mish": "(x2, row logsumexp, Mish)",
             "bf16_gn_swish_mul_swish": "(GroupNorm 32x128, SiLU, x1.5, SiLU)",
             "bf16_gn_lrelu_sum": "(GroupNorm 32x128, LeakyReLU 0.01, x+x)",
             "bf16_swish_sum_gn": "(SiLU, +0.25, GroupNorm 32x128)",
             "e4m3_gelu_clamp": "(per-row scales, x0.5, GELU_tanh, clamp[-1,1])"}


def base_result(args, metric_value, ms, dtype, data, config, roofline):
    return {
        "metric": "fused GEMM+epilogue TFLOP/s (% of MI355X MFMA peak) vs unfused sequence",
        "value": round(metric_value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": data, "config": config,
        "roofline": roofline,
    }


def bench_fgemm(args, torch, np):
    import torch.nn.functional as F
    from paper_2606_02963_amd import api
    from paper_2606_02963_amd.synth import FGEMM_SPECS, make_fgemm_inputs

    spec = FGEMM_SPECS[FGEMM_WORKLOADS[args.workload]]
    inp = make_fgemm_inputs(spec, seed=0)
    dev = torch.device("cuda", 0)
    sx = sw = None
    if spec.dtype == "f32":
        x, W = torch.from_numpy(inp["x"]).to(dev), torch.from_numpy(inp["W"]).to(dev)
    elif spec.dtype == "e4m3":
        x, W = torch.from_numpy(inp["x"]).to(dev), torch.from_numpy(inp["W"]).to(dev)
        sx, sw = torch.from_numpy(inp["x_scale"]).to(dev), torch.from_numpy(inp["w_scale"]).to(dev)
    else:
        x = torch.from_numpy(inp["x"].view(np.int16)).view(torch.bfloat16).to(dev)
        W = torch.from_numpy(inp["W"].view(np.int16)).view(torch.bfloat16).to(dev)
    b = torch.from_numpy(inp["b"]).to(dev)
    g = torch.from_numpy(inp["gamma"]).to(dev) if "gamma" in inp else None
    be = torch.from_numpy(inp["beta"]).to(dev) if "beta" in inp else None
    out_dt = torch.float32 if spec.out == "f32" else torch.bfloat16
    out = torch.empty((spec.M,) if spec.reduction == "lse" else (spec.M, spec.N), dtype=out_dt, device=dev)
    plan = api.get_plan(spec.M, spec.N, spec.K, spec.dtype, spec.out, True, spec.ops, spec.reduction,
                        spec.gn_groups, spec.gn_eps, spec.post_ops)
    info = plan.info()
    ws = torch.empty(max(plan.workspace_bytes(), 16), dtype=torch.uint8, device=dev)

    def fused():
        api.linear_epilogue(x, W, b, spec.ops, spec.reduction, spec.gn_groups, spec.gn_eps, g, be,
                            out_dtype=spec.out, out=out, workspace=ws, post_ops=spec.post_ops,
                            x_scale=sx, w_scale=sw)

    settle(fused, args.warmup_seconds, torch)
    ms = time_steps(fused, args.steps, args.warmup, torch)
    reps = repeat_stats(fused, args.steps, torch)
    flops = spec.flops()
    tflops = flops / (ms * 1e-3) / 1e12
    peak = {"bf16": PEAK_BF16_TFLOPS, "e4m3": PEAK_FP8_TFLOPS, "f32": 157.3}[spec.dtype]
    # the GEMM launch dominates; with a row LogSumExp the step also holds the
    # small combine launch, so the step time bounds the GEMM launch from above
    achieved = tflops
    name = f"fgemm_{spec.name}_{spec.M}x{spec.N}x{spec.K}"
    result = base_result(
        args, tflops, ms, spec.dtype,
        "synthetic (seeded: x ~ N(0,1), W, b ~ U(+-a); see paper_2606_02963_amd/synth.py)",
        {"workload": f"{spec.dtype} GEMM + {TAIL_TEXT[spec.name]} tail, x[{spec.M},{spec.K}] "
                     f"W[{spec.N},{spec.K}] -> {spec.out}"
                     f"[{spec.M}{'' if spec.reduction == 'lse' else ',' + str(spec.N)}]",
         "M": spec.M, "N": spec.N, "K": spec.K, "tile": f"{info['tile_m']}x{info['tile_n']}",
         "workgroups": info["workgroups"], "launches_per_step": info["launches"]},
        {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
         "frac": round(achieved / peak, 4), "traffic": measured_traffic(name),
         "algorithmic_flops_per_launch": flops, "algorithmic_bytes_per_launch": spec.bytes()})
    result["repeats"] = reps

    if not args.no_unfused:
        tdt = torch.float32 if spec.dtype == "f32" else torch.bfloat16
        bb = b.to(tdt)

        def eager_ops(z, ops):
            for op in ops:
                if op[0] == "scale":
                    z = z * op[1]
                elif op[0] == "add":
                    z = z + op[1]
                elif op[0] == "relu":
                    z = torch.relu(z)
                elif op[0] == "gelu_tanh":
                    z = F.gelu(z, approximate="tanh")
                elif op[0] == "silu":
                    z = F.silu(z)
                elif op[0] == "clamp":
                    z = torch.clamp(z, op[1], op[2])
                elif op[0] == "mish":
                    z = F.mish(z)
                elif op[0] == "leaky_relu":
                    z = F.leaky_relu(z, op[1])
            return z

        if spec.dtype == "e4m3":
            # vendor fp8 GEMM with row-wise scales (hipBLASLt through
            # torch._scaled_mm), bf16 result
            x8, W8 = x.view(torch.float8_e4m3fn), W.view(torch.float8_e4m3fn)
            sa, sb = sx.view(-1, 1), sw.view(1, -1)

            def vendor_mm():
                return torch._scaled_mm(x8, W8.t(), scale_a=sa, scale_b=sb, out_dtype=torch.bfloat16)
        else:
            def vendor_mm():
                return torch.mm(x, W.t())

        def unfused():
            z = vendor_mm()
            z = eager_ops(z + bb, spec.ops)
            if spec.reduction == "lse":
                z = torch.logsumexp(z.float(), dim=1)
            elif spec.reduction == "groupnorm":
                z = F.group_norm(z, spec.gn_groups, g.to(tdt), be.to(tdt), spec.gn_eps)
            return eager_ops(z, spec.post_ops)

        try:
            ms_u = time_steps(unfused, args.steps, args.warmup, torch)
            ms_g = time_steps(vendor_mm, args.steps, args.warmup, torch)
        except RuntimeError as e:         # a torch build without row-wise fp8 scaling
            result["unfused"] = {"ms": None, "error": str(e).splitlines()[0][:200]}
        else:
            result["unfused"] = {"ms": round(ms_u, 5), "tflops": round(flops / (ms_u * 1e-3) / 1e12, 2),
                                 "sequence": ("torch._scaled_mm (vendor fp8 GEMM, row-wise scales)"
                                              if spec.dtype == "e4m3" else "torch.mm (vendor BLAS)")
                                 + " then one eager kernel per tail op"}
            result["gemm_only"] = {"ms": round(ms_g, 5), "tflops": round(flops / (ms_g * 1e-3) / 1e12, 2)}
            result["speedup_vs_unfused"] = round(ms_u / ms, 3)

    if not args.no_cpu_baseline:
        torch.cuda.synchronize()
        cpu = cpu_oracle_fgemm(spec, inp, args.cpu_seconds, out, np)
        result["cpu_baseline"], rep = cpu
        result["parity_sample"] = {"rel_err": rep.rel_err, "tol": rep.tol, "ok": bool(rep.ok)}
    return result


def cpu_oracle_fgemm(spec, inp, budget_s, out, np):
    """Time the fp64 oracle on a growing sample of rows until ~budget_s."""
    from threadpoolctl import threadpool_info
    from oracle import bf16_decode, compare, e4m3_decode, ref_fgemm

    if spec.dtype == "e4m3":
        x64 = e4m3_decode(inp["x"]) * inp["x_scale"].astype(np.float64)[:, None]
        W64 = e4m3_decode(inp["W"]) * inp["w_scale"].astype(np.float64)[:, None]
    else:
        dec = (lambda a: a.astype(np.float64)) if spec.dtype == "f32" else bf16_decode
        x64, W64 = dec(inp["x"]), dec(inp["W"])
    b = inp["b"].astype(np.float64)
    got = out.float().cpu().numpy().astype(np.float64)
    rows, t_total, flops_total, n_rows, first = 8, 0.0, 0.0, 0, None
    while t_total < budget_s and n_rows < spec.M:
        r = min(rows, spec.M - n_rows)
        sel = slice(n_rows, n_rows + r)
        t0 = time.perf_counter()
        ref = ref_fgemm(x64[sel], W64, b, spec.ops, spec.reduction, spec.gn_groups, spec.gn_eps,
                        inp.get("gamma"), inp.get("beta"), spec.post_ops)
        t_total += time.perf_counter() - t0
        if first is None:
            first = (sel, ref)
        flops_total += 2.0 * r * spec.N * spec.K
        n_rows += r
        rows *= 2
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    rep = compare(got[first[0]], first[1], {"f32": "f32", "bf16": "bf16", "e4m3": "e4m3"}[spec.dtype])
    return ({"value": flops_total / t_total / 1e12, "unit": "TFLOP/s", "cores": int(threads),
             "kind": "oracle",
             "sample": f"{n_rows} of {spec.M} output rows (all {spec.N} columns, K={spec.K}), "
                       f"fp64 numpy matmul + tail, {t_total:.1f} s",
             "seconds": round(t_total, 2)}, rep)


def bench_moe(args, torch, np):
    from paper_2606_02963_amd import api
    from paper_2606_02963_amd.synth import MOE_SPECS, make_moe_activations, make_moe_weights

    spec = MOE_SPECS[args.workload]
    act = make_moe_activations(spec, 0)
    w = make_moe_weights(spec, 0)
    dev = torch.device("cuda", 0)
    bf = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)  # noqa: E731
    x, lg = bf(act["x"]), torch.from_numpy(act["logits"]).to(dev)
    if spec.w_dtype == "bf16":
        wgu, wd, sgu, sd = bf(w["w_gate_up"]), bf(w["w_down"]), None, None
    else:
        wgu, wd = torch.from_numpy(w["w_gate_up"]).to(dev), torch.from_numpy(w["w_down"]).to(dev)
        sgu, sd = torch.from_numpy(w["s_gate_up"]).to(dev), torch.from_numpy(w["s_down"]).to(dev)
    del w
    bufs = api.moe_ffn(x, lg, wgu, wd, sgu, sd, top_k=spec.k)

    def fused():
        api.moe_ffn(x, lg, wgu, wd, sgu, sd, top_k=spec.k, buffers=bufs)

    settle(fused, args.warmup_seconds, torch)
    ms = time_steps(fused, args.steps, args.warmup, torch)
    reps = repeat_stats(fused, args.steps, torch)
    counts = np.diff(bufs.offsets.cpu().numpy())
    active = int(np.sum(counts > 0))
    flops = spec.flops()
    nbytes = spec.bytes(active)
    tflops = flops / (ms * 1e-3) / 1e12
    gbs = nbytes / (ms * 1e-3) / 1e9
    decode = spec.T <= 256
    peak_c = PEAK_BF16_TFLOPS if spec.w_dtype == "bf16" else 5000.0
    roof = ({"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
             "frac": round(gbs / PEAK_HBM_GBS, 4)} if decode else
            {"bound": "mfma", "achieved": round(tflops, 2), "peak": peak_c, "unit": "TFLOP/s",
             "frac": round(tflops / peak_c, 4)})
    roof.update({"traffic": measured_traffic(spec.name, MOE_KERNEL_SOURCES),
                 "scope": "whole step (all launches)",
                 "algorithmic_flops": flops, "algorithmic_bytes": nbytes, "active_experts": active})
    result = base_result(
        args, tflops, ms, "e4m3" if spec.w_dtype == "e4m3" else "bf16",
        "synthetic (seeded: logits, x ~ N(0,1); W ~ N(0,0.02); see paper_2606_02963_amd/synth.py)",
        {"workload": f"MoE expert FFN step T={spec.T} H={spec.H} I={spec.I} E={spec.E} top-{spec.k} "
                     f"{spec.w_dtype} weights, clamped SwiGLU",
         "T": spec.T, "H": spec.H, "I": spec.I, "E": spec.E, "top_k": spec.k}, roof)
    result["hbm_gbs"] = round(gbs, 1)
    result["repeats"] = reps
    if not args.no_cpu_baseline:
        torch.cuda.synchronize()
        cpu, rep = cpu_oracle_moe(spec, act, bufs.out, nbytes, decode, np, torch)
        result["cpu_baseline"] = cpu
        result["parity_sample"] = {"rel_err": rep.rel_err, "tol": rep.tol, "ok": bool(rep.ok)}

    if not args.no_unfused:
        # The eager PyTorch sequence: top-k and softmax, a stable argsort of the
        # slots, the expert sizes brought to the host for the per-expert loop,
        # a gather of token rows, per expert a vendor GEMM, the clamped SwiGLU
        # as separate elementwise kernels and a second vendor GEMM, then the
        # routing-weight multiply, a scatter back to slot order and the sum
        # over the k slots. With e4m3 weights the activations are quantised
        # per row in eager torch and each GEMM is the vendor fp8 GEMM with
        # row-wise scales (torch._scaled_mm).
        k, E, I = spec.k, spec.E, spec.I
        f8 = spec.w_dtype == "e4m3"
        if f8:
            wgu8, wd8 = wgu.view(torch.float8_e4m3fn), wd.view(torch.float8_e4m3fn)

            def q_rows(t):
                a = t.float().abs().amax(dim=1, keepdim=True)
                sc = torch.where(a > 0, a / 448.0, torch.ones_like(a))
                return (t.float() / sc).clamp(-448.0, 448.0).to(torch.float8_e4m3fn), sc

            def mm(a_rows, e, down):
                q, sa = q_rows(a_rows)
                w8, sw_ = (wd8, sd) if down else (wgu8, sgu)
                return torch._scaled_mm(q, w8[e].t(), scale_a=sa, scale_b=sw_[e].view(1, -1),
                                        out_dtype=torch.bfloat16)
        else:
            def mm(a_rows, e, down):
                return torch.mm(a_rows, (wd if down else wgu)[e].t())

        def unfused():
            topv, topi = torch.topk(lg, k, dim=1)
            wts = torch.softmax(topv, dim=1).flatten()
            flat = topi.flatten()
            order = torch.argsort(flat, stable=True)
            offs = [0] + torch.bincount(flat, minlength=E).cumsum(0).tolist()
            xs = x[order // k]
            ys = torch.empty(x.shape[0] * k, spec.H, dtype=torch.bfloat16, device=dev)
            for e in range(E):
                a, b_ = offs[e], offs[e + 1]
                if a == b_:
                    continue
                gu = mm(xs[a:b_], e, False)
                gate = torch.clamp(gu[:, :I], max=spec.limit)
                up = torch.clamp(gu[:, I:], -spec.limit, spec.limit)
                h = (up + 1) * gate * torch.sigmoid(spec.alpha * gate)
                ys[order[a:b_]] = mm(h, e, True)
            ys = ys * wts[:, None].to(torch.bfloat16)
            return ys.view(-1, k, spec.H).float().sum(1).to(torch.bfloat16)

        try:
            ms_u = time_steps(unfused, args.steps, args.warmup, torch)
        except RuntimeError as e:         # a torch build without row-wise fp8 scaling
            result["unfused"] = {"ms": None, "error": str(e).splitlines()[0][:200]}
        else:
            result["unfused"] = {"ms": round(ms_u, 5), "tflops": round(flops / (ms_u * 1e-3) / 1e12, 2),
                                 "hbm_gbs": round(nbytes / (ms_u * 1e-3) / 1e9, 1),
                                 "sequence": "eager torch: topk, softmax, stable argsort, per-expert "
                                             + ("row quantisation + torch._scaled_mm (fp8) + elementwise "
                                                "clamped SwiGLU + row quantisation + torch._scaled_mm"
                                                if f8 else "torch.mm + elementwise clamped SwiGLU + torch.mm")
                                             + ", weighted scatter, slot sum"}
            result["speedup_vs_unfused"] = round(ms_u / ms, 3)
    return result


def cpu_oracle_moe(spec, act, out, step_bytes, decode, np, torch):
    """Time the fp64 oracle's MoE step on the host: the whole step at decode
    size (T = 64), the first 64 tokens of the prefill batch otherwise. The
    oracle decodes each expert's weights to fp64 as part of its work."""
    from threadpoolctl import threadpool_info
    from oracle import bf16_decode, compare, e4m3_decode, ref_moe
    from paper_2606_02963_amd.synth import make_moe_weights

    w = make_moe_weights(spec, 0)
    if spec.w_dtype == "bf16":
        weights = lambda e: (bf16_decode(w["w_gate_up"][e]), bf16_decode(w["w_down"][e]))  # noqa: E731
    else:
        weights = lambda e: (e4m3_decode(w["w_gate_up"][e]) * w["s_gate_up"][e][:, None].astype(np.float64),  # noqa: E731
                             e4m3_decode(w["w_down"][e]) * w["s_down"][e][:, None].astype(np.float64))
    tokens = None if decode else np.arange(min(64, spec.T))
    f8 = spec.w_dtype == "e4m3"
    t0 = time.perf_counter()
    ref = ref_moe(bf16_decode(act["x"]), act["logits"].astype(np.float64), weights, spec.k,
                  storage="e4m3" if f8 else "bf16", act_quant=f8, alpha=spec.alpha, limit=spec.limit,
                  tokens=tokens, with_bound=True)
    sec = time.perf_counter() - t0
    got = bf16_decode(out.view(torch.int16).cpu().numpy().view(np.uint16))
    if tokens is not None:
        got = got[tokens]
    rep = compare(got, ref["out"], "e4m3" if f8 else "bf16", slack=ref["out_bound"])
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    n = spec.T if tokens is None else tokens.size
    if decode:
        value, unit = step_bytes / sec / 1e9, "GB/s"
    else:
        value, unit = 2.0 * n * spec.k * (spec.H * 2 * spec.I + spec.I * spec.H) / sec / 1e12, "TFLOP/s"
    return ({"value": round(value, 4), "unit": unit, "cores": int(threads), "kind": "oracle",
             "sample": (f"the whole T={spec.T} step" if tokens is None else
                        f"{n} of {spec.T} tokens (their {n * spec.k} slots through all experts)") +
                       f", fp64 numpy incl. decoding the expert weights, {sec:.1f} s",
             "seconds": round(sec, 2)}, rep)


def bench_finalize(args, torch, np):
    """The standalone MoE finalize over the batch sizes of paper Table I
    (top-4, H = 2880). Each launch moves a few MB, so launches are captured
    back to back in one HIP graph and the graph is timed; per-launch time is
    the graph time over the launches in it. The headline line is T = 128."""
    from paper_2606_02963_amd import api
    from paper_2606_02963_amd.synth import FINALIZE_BATCHES, FINALIZE_H, FINALIZE_K, make_finalize_inputs

    reps = 50
    H, k = FINALIZE_H, FINALIZE_K
    sweep = {}
    for T in FINALIZE_BATCHES:
        bits = make_finalize_inputs(T)
        y = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()
        out = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
        api.moe_finalize(y, k, out=out)
        torch.cuda.synchronize()
        eager = out.clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                api.moe_finalize(y, k, out=out)
        g.replay()
        torch.cuda.synchronize()
        if not torch.equal(out, eager):
            raise RuntimeError("graph replay of moe_finalize differs from the eager launch")
        settle(g.replay, min(args.warmup_seconds, 0.3), torch)
        ms = time_steps(g.replay, max(args.steps // 5, 5), max(args.warmup // 5, 2), torch) / reps
        nbytes = (T * k * H + T * H) * 2
        sweep[T] = {"us": round(ms * 1e3, 3), "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1), "bytes": nbytes}
    T = FINALIZE_BATCHES[-1]
    head = sweep[T]
    roof = {"bound": "hbm", "achieved": head["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(head["gbs"] / PEAK_HBM_GBS, 4), "traffic": None,
            "algorithmic_bytes_per_launch": head["bytes"]}
    result = {
        "metric": "MoE finalize effective HBM GB/s (paper Table I batch sweep)", "value": head["gbs"],
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(head["us"] / 1e3, 6), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded: y_slot ~ N(0, 0.25); see "
        "paper_2606_02963_amd/synth.py)",
        "config": {"workload": f"MoE finalize y_slot[{T}x{k}, {H}] bf16 -> out[{T}, {H}] bf16, fp32 sum",
                   "T": T, "H": H, "top_k": k, "launches_per_graph": reps},
        "roofline": roof, "sweep": {str(t): v for t, v in sweep.items()}}
    if not args.no_cpu_baseline:
        from oracle import bf16_decode, ref_moe_finalize
        y64 = bf16_decode(make_finalize_inputs(T))
        t0, n = time.perf_counter(), 0
        while time.perf_counter() - t0 < 1.0:
            ref_moe_finalize(y64, k)
            n += 1
        sec = (time.perf_counter() - t0) / n
        result["cpu_baseline"] = {"value": round(head["bytes"] / sec / 1e9, 3), "unit": "GB/s",
                                  "cores": 1, "kind": "oracle",
                                  "sample": f"the whole T={T} finalize, {n} repetitions in ~1 s",
                                  "seconds": round(sec, 6)}
    return result


def bench_add_rmsnorm(args, torch, np):
    """The fused residual add + RMSNorm over the batch sizes of paper Table I
    (H = 2880, eps = 1e-5), timed like the finalize: launches captured back
    to back in one HIP graph. Each launch reads x, the residual and the
    weight and writes the residual and out; the headline line is T = 128.
    The residual is updated in place, so the graph's launches chain (each
    adds x once more), which changes the values but not the work."""
    from paper_2606_02963_amd import api
    from paper_2606_02963_amd.synth import FINALIZE_BATCHES, NORM_H, make_norm_inputs

    reps = 50
    H = NORM_H
    dev = torch.device("cuda", 0)
    bf = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)  # noqa: E731
    sweep = {}
    for T in FINALIZE_BATCHES:
        x, r, w = (bf(a) for a in make_norm_inputs(T))
        out = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        api.add_rmsnorm(x, r, w, out=out)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                api.add_rmsnorm(x, r, w, out=out)
        settle(g.replay, min(args.warmup_seconds, 0.3), torch)
        ms = time_steps(g.replay, max(args.steps // 5, 5), max(args.warmup // 5, 2), torch) / reps
        nbytes = 4 * T * H * 2 + H * 2
        sweep[T] = {"us": round(ms * 1e3, 3), "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1), "bytes": nbytes}
    T = FINALIZE_BATCHES[-1]
    head = sweep[T]
    roof = {"bound": "hbm", "achieved": head["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(head["gbs"] / PEAK_HBM_GBS, 4), "traffic": None,
            "algorithmic_bytes_per_launch": head["bytes"]}
    result = {
        "metric": "fused add + RMSNorm effective HBM GB/s (paper Table I batch sweep)", "value": head["gbs"],
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(head["us"] / 1e3, 6), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded: x ~ N(0,1), residual ~ N(0,4), weight ~ U(0.5,1.5); see "
                "paper_2606_02963_amd/synth.py)",
        "config": {"workload": f"residual add + RMSNorm, x/residual[{T}, {H}] bf16, eps 1e-5",
                   "T": T, "H": H, "launches_per_graph": reps},
        "roofline": roof, "sweep": {str(t): v for t, v in sweep.items()}}
    if not args.no_cpu_baseline:
        from oracle import bf16_decode, ref_add_rmsnorm
        x, r, w = (bf16_decode(a) for a in make_norm_inputs(T))
        t0, n = time.perf_counter(), 0
        while time.perf_counter() - t0 < 1.0:
            ref_add_rmsnorm(x, r, w, 1e-5)
            n += 1
        sec = (time.perf_counter() - t0) / n
        result["cpu_baseline"] = {"value": round(head["bytes"] / sec / 1e9, 3), "unit": "GB/s",
                                  "cores": 1, "kind": "oracle",
                                  "sample": f"the whole T={T} step, {n} repetitions in ~1 s",
                                  "seconds": round(sec, 6)}
    return result


def bench_rope_kv(args, torch, np):
    """QKV bias + RoPE + paged KV-cache update over the batch sizes of paper
    Table I (gpt-oss-20b attention sizes: 64 query and 8 key/value heads of
    64, base 150000, 64-token blocks), timed like the finalize: launches
    captured back to back in one HIP graph. Every launch rewrites the same
    cache rows with the same values. The headline line is T = 128."""
    from paper_2606_02963_amd import api
    from paper_2606_02963_amd.synth import FINALIZE_BATCHES, RopeSpec, make_rope_inputs

    reps = 50
    dev = torch.device("cuda", 0)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)  # noqa: E731
    sweep = {}
    for T in FINALIZE_BATCHES:
        spec = RopeSpec(T)
        inp = make_rope_inputs(spec)
        qkv, bias, cache = bf(inp["qkv"]), bf(inp["bias"]), bf(inp["cache"])
        pos = torch.from_numpy(inp["positions"]).to(dev)
        table = torch.from_numpy(inp["block_table"]).to(dev)
        q = torch.empty((T, spec.n_q, spec.D), dtype=torch.bfloat16, device=dev)

        def step():
            api.bias_rope_kv_update(qkv, bias, pos, table, cache, spec.n_q, spec.n_kv, spec.D, spec.base,
                                    q_out=q)

        step()
        torch.cuda.synchronize()
        eager_q, eager_c = q.clone(), cache.clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                step()
        g.replay()
        torch.cuda.synchronize()
        if not (torch.equal(q, eager_q) and torch.equal(cache, eager_c)):
            raise RuntimeError("graph replay of bias_rope_kv_update differs from the eager launch")
        settle(g.replay, min(args.warmup_seconds, 0.3), torch)
        ms = time_steps(g.replay, max(args.steps // 5, 5), max(args.warmup // 5, 2), torch) / reps
        nbytes = spec.bytes()
        sweep[T] = {"us": round(ms * 1e3, 3), "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1), "bytes": nbytes}
    T = FINALIZE_BATCHES[-1]
    spec = RopeSpec(T)
    head = sweep[T]
    roof = {"bound": "hbm", "achieved": head["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(head["gbs"] / PEAK_HBM_GBS, 4), "traffic": None,
            "algorithmic_bytes_per_launch": head["bytes"]}
    result = {
        "metric": "bias + RoPE + KV-cache update effective HBM GB/s (paper Table I batch sweep)",
        "value": head["gbs"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(head["us"] / 1e3, 6), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded: qkv ~ N(0,1), bias ~ U(-0.1,0.1), positions ~ U{0..8191}; see "
                "paper_2606_02963_amd/synth.py)",
        "config": {"workload": f"QKV bias + RoPE + paged KV write, qkv[{T}, {spec.width}] bf16, "
                               f"{spec.n_q} q / {spec.n_kv} kv heads x {spec.D}, base {spec.base:g}, "
                               f"{spec.block_size}-token blocks",
                   "T": T, "launches_per_graph": reps},
        "roofline": roof, "sweep": {str(t): v for t, v in sweep.items()}}
    if not args.no_cpu_baseline:
        from oracle import bf16_decode, ref_bias_rope_kv_update
        inp = make_rope_inputs(spec)
        args64 = (bf16_decode(inp["qkv"]), bf16_decode(inp["bias"]), inp["positions"], inp["block_table"],
                  bf16_decode(inp["cache"]), spec.n_q, spec.n_kv, spec.D, spec.block_size, spec.base)
        t0, n = time.perf_counter(), 0
        while time.perf_counter() - t0 < 1.0:
            ref_bias_rope_kv_update(*args64)
            n += 1
        sec = (time.perf_counter() - t0) / n
        result["cpu_baseline"] = {"value": round(head["bytes"] / sec / 1e9, 3), "unit": "GB/s",
                                  "cores": 1, "kind": "oracle",
                                  "sample": f"the whole T={T} step, {n} repetitions in ~1 s",
                                  "seconds": round(sec, 6)}
    return result


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the library runs one GPU per process and has no multi-GPU path; --gpus must be 1",
                          "n_gpus": args.gpus}))
        print("bench.py: no multi-GPU path is implemented (the step runs on one GPU); use --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_02963_amd import _lib

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    _lib.lib()   # fail loudly if the HIP library is missing
    if args.workload in MOE_WORKLOADS:
        result = bench_moe(args, torch, np)
    elif args.workload == "moe_finalize":
        result = bench_finalize(args, torch, np)
    elif args.workload == "add_rmsnorm":
        result = bench_add_rmsnorm(args, torch, np)
    elif args.workload == "rope_kv":
        result = bench_rope_kv(args, torch, np)
    else:
        result = bench_fgemm(args, torch, np)
    if args.copy_calibration_mb > 0:
        n = args.copy_calibration_mb << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
