#!/usr/bin/env python3
"""Benchmark of the fused GEMM + tail library on one MI355X.

Default workload (the largest single-GPU configuration): one MoE expert-FFN
step of a gpt-oss-20b-like layer, T = 4096 tokens, hidden 2880, 32 experts,
top-4, bf16 weights ~ N(0, 0.02), clamped SwiGLU: routing, permutation, the
grouped gate/up GEMM with the SwiGLU epilogue, the grouped down GEMM with the
routing weight, and the finalize, all on the device with inputs resident in
HBM. Other workloads: the dense fused GEMM + tail configurations, the e4m3
MoE variants, the decode step, and the Table I kernels.

Timing: W untimed warmup steps (after about a second of untimed work so
that clocks settle), then seven repeats, each timing a multiple of K steps
with HIP events on the stream the library launches on, bracketed by device
synchronisation, and lasting at least --min-repeat-seconds; ``value`` and
``ms_per_step`` are the median over the repeats (their coefficient of
variation is reported beside it). The shader and memory clocks are sampled
from sysfs during the repeats. A separate pass of K steps traces every
launch with HIP events (fg_trace_begin) to give each kernel's average
duration; ``roofline`` is that of the dominant kernel, ``step_roofline`` that
of the whole step. The unfused PyTorch sequence is timed the same way, and
the fp64 CPU oracle on a bounded sample whose outputs are also compared.

Prints ONE JSON line.

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
                       [--workload moe_prefill_bf16|moe_prefill_e4m3|moe_decode_bf16|moe_decode_e4m3|
                                   gelu_clamp|gelu_clamp_e4m3|lse|silu_gn|tiny_f32|scale_lse_mish|
                                   gn_swish_mul_swish|gn_lrelu_sum|swish_sum_gn|
                                   moe_finalize|add_rmsnorm|rope_kv]
"""

import argparse
import glob
import hashlib
import json
import math
import os
import re
import statistics
import subprocess
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X published dense peaks (no sparsity)
PEAK_BF16_TFLOPS = 2516.6
PEAK_FP8_TFLOPS = 5033.2
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
PEAK_SCLK_MHZ = 2400.0
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ["fg_tile.hpp", "fg_epilogue.hpp", "fgemm.hip"]
MOE_KERNEL_SOURCES = ["fg_tile.hpp", "fg_quant.hpp", "moe.hip", "quant.hip"]
REPEATS = 7


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--warmup-seconds", type=float, default=1.0,
                    help="extra untimed work first, so clocks settle before timing")
    ap.add_argument("--min-repeat-seconds", type=float, default=1.0,
                    help="each of the seven timed repeats runs whole multiples of --steps steps for at "
                         "least this long")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target oracle sample time")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after the measurement, run a plain device-to-device copy of this many MiB "
                         "(3 times); its HBM counters calibrate rocprofv3 FETCH_SIZE/WRITE_SIZE")
    ap.add_argument("--workload", default="moe_prefill_bf16",
                    choices=["moe_prefill_bf16", "moe_prefill_e4m3", "moe_decode_bf16", "moe_decode_e4m3",
                             "gelu_clamp", "gelu_clamp_e4m3", "lse", "silu_gn", "tiny_f32", "scale_lse_mish",
                             "gn_swish_mul_swish", "gn_lrelu_sum", "swish_sum_gn", "moe_finalize",
                             "add_rmsnorm", "rope_kv"],
                    help="moe_prefill_bf16 (default) is the headline workload; the others are the "
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


def time_block(fn, n, torch):
    """Milliseconds for n back-to-back steps: HIP events on the current
    stream (where the library launches), device synchronised before and
    after."""
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(n):
        fn()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop)


def timed_repeats(fn, steps, warmup, min_seconds, torch, repeats=REPEATS):
    """`warmup` untimed steps, then `repeats` timings, each of blocks × steps
    back-to-back steps where blocks is the smallest count that makes one
    repeat last at least `min_seconds`. Returns the median ms per step and
    the spread."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    probe = time_block(fn, steps, torch)
    blocks = max(1, math.ceil(min_seconds * 1e3 / max(probe, 1e-6)))
    per = [time_block(fn, steps * blocks, torch) / (steps * blocks) for _ in range(repeats)]
    med = statistics.median(per)
    return {"ms_per_step": med, "repeats": repeats, "steps_per_repeat": steps * blocks,
            "seconds_per_repeat": round(med * steps * blocks / 1e3, 3),
            "ms_per_step_each": [round(v, 5) for v in per],
            "cv": round(statistics.pstdev(per) / statistics.fmean(per), 5)}


class ClockSampler:
    """Samples the GPU's current shader (sclk) and memory (mclk) clock from
    sysfs (pp_dpm_sclk / pp_dpm_mclk, the level marked '*') every 50 ms
    while active. The device is found by the PCI address torch reports for
    device 0; with no readable file the summary says so."""

    def __init__(self, torch):
        self.paths = {}
        try:
            p = torch.cuda.get_device_properties(0)
            addr = f"{p.pci_domain_id:04x}:{p.pci_bus_id:02x}:{p.pci_device_id:02x}"
            cands = sorted(glob.glob(f"/sys/bus/pci/devices/{addr}.*"))
        except Exception:
            cands = []
        if not cands:
            cards = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
            cands = [os.path.dirname(cards[0])] if len(cards) == 1 else []
        for d in cands:
            for clk in ("sclk", "mclk"):
                f = os.path.join(d, f"pp_dpm_{clk}")
                if os.access(f, os.R_OK):
                    self.paths[clk] = f
            if self.paths:
                break
        self.samples = {k: [] for k in self.paths}
        self._stop = threading.Event()
        self._thread = None

    @staticmethod
    def _read(path):
        try:
            with open(path) as fh:
                for line in fh:
                    if "*" in line:
                        m = re.search(r"(\d+)\s*[Mm][Hh]z", line)
                        return int(m.group(1)) if m else None
        except OSError:
            return None
        return None

    def _run(self):
        while not self._stop.is_set():
            for k, f in self.paths.items():
                v = self._read(f)
                if v is not None:
                    self.samples[k].append(v)
            self._stop.wait(0.05)

    def __enter__(self):
        if self.paths:
            self._thread = threading.Thread(target=self._run, daemon=True)
            self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self._thread is not None:
            self._thread.join()

    def summary(self):
        out = {"source": self.paths.get("sclk", "unavailable (no readable pp_dpm_sclk)")}
        for k, v in self.samples.items():
            if v:
                out[f"{k}_mhz"] = {"median": statistics.median(v), "min": min(v), "max": max(v),
                                   "samples": len(v)}
        return out


def demangle(names):
    try:
        r = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True, timeout=10)
        out = r.stdout.splitlines()
        if r.returncode == 0 and len(out) == len(names):
            return out
    except (OSError, subprocess.SubprocessError):
        pass
    return list(names)


def trace_kernels(fn, steps, torch):
    """Run `steps` steps with the library's launch trace open and return,
    per kernel, the number of launches and the average and total time
    between the HIP events recorded around each launch."""
    from paper_2606_02963_amd import _lib
    torch.cuda.synchronize()
    _lib.fg_trace_begin(steps * 64)
    try:
        for _ in range(steps):
            fn()
    finally:
        n = _lib.fg_trace_end()
    torch.cuda.synchronize()
    rows = [_lib.fg_trace_read(i) for i in range(n)]
    names = demangle(sorted({name for _, name in rows}))
    pretty = dict(zip(sorted({name for _, name in rows}), names))
    per = {}
    for ms, name in rows:
        per.setdefault(pretty[name], []).append(ms)
    return {k: {"launches": len(v), "avg_us": round(1e3 * statistics.fmean(v), 2),
                "total_ms": round(sum(v), 4)} for k, v in per.items()}


def dominant(kernels):
    return max(kernels.items(), key=lambda kv: kv[1]["total_ms"])


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


def base_result(args, metric_value, tim, dtype, data, config, roofline):
    return {
        "metric": "fused GEMM+epilogue TFLOP/s (% of MI355X MFMA peak) vs unfused sequence",
        "value": round(metric_value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(tim["ms_per_step"], 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": data, "config": config,
        "roofline": roofline,
    }


def timing_record(tim, clk):
    t = dict(tim)
    t["ms_per_step"] = round(t["ms_per_step"], 5)
    t["clocks"] = clk.summary()
    sclk = t["clocks"].get("sclk_mhz", {}).get("median")
    if sclk:
        t["peak_scale_at_sampled_sclk"] = round(sclk / PEAK_SCLK_MHZ, 4)
    return t


def measure(fn, args, torch):
    """Settle, then the seven timed repeats with the clocks sampled, then the
    traced pass. Returns (timing, clock sampler, per-kernel trace)."""
    settle(fn, args.warmup_seconds, torch)
    with ClockSampler(torch) as clk:
        tim = timed_repeats(fn, args.steps, args.warmup, args.min_repeat_seconds, torch)
    kernels = trace_kernels(fn, args.steps, torch)
    return tim, clk, kernels


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

    tim, clk, kernels = measure(fused, args, torch)
    ms = tim["ms_per_step"]
    flops = spec.flops()
    tflops = flops / (ms * 1e-3) / 1e12
    peak = {"bf16": PEAK_BF16_TFLOPS, "e4m3": PEAK_FP8_TFLOPS, "f32": PEAK_FP32_TFLOPS}[spec.dtype]
    kname, kst = dominant(kernels)
    k_tflops = flops / (kst["avg_us"] * 1e-6) / 1e12
    name = f"fgemm_{spec.name}_{spec.M}x{spec.N}x{spec.K}"
    result = base_result(
        args, tflops, tim, spec.dtype,
        "synthetic (seeded: x ~ N(0,1), W, b ~ U(+-a); see paper_2606_02963_amd/synth.py)",
        {"workload": f"{spec.dtype} GEMM + {TAIL_TEXT[spec.name]} tail, x[{spec.M},{spec.K}] "
                     f"W[{spec.N},{spec.K}] -> {spec.out}"
                     f"[{spec.M}{'' if spec.reduction == 'lse' else ',' + str(spec.N)}]",
         "M": spec.M, "N": spec.N, "K": spec.K, "tile": f"{info['tile_m']}x{info['tile_n']}",
         "workgroups": info["workgroups"], "launches_per_step": info["launches"]},
        {"bound": "mfma", "kernel": kname, "achieved": round(k_tflops, 2), "peak": peak, "unit": "TFLOP/s",
         "frac": round(k_tflops / peak, 4), "traffic": measured_traffic(name),
         "avg_launch_us": kst["avg_us"], "algorithmic_flops_per_launch": flops,
         "algorithmic_bytes_per_launch": spec.bytes()})
    result["step_roofline"] = {"bound": "mfma", "achieved": round(tflops, 2), "peak": peak, "unit": "TFLOP/s",
                               "frac": round(tflops / peak, 4), "scope": "whole step (all launches)"}
    result["timing"] = timing_record(tim, clk)
    result["kernels"] = kernels

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
            tu = timed_repeats(unfused, args.steps, args.warmup, args.min_repeat_seconds, torch)
            tg = timed_repeats(vendor_mm, args.steps, args.warmup, args.min_repeat_seconds, torch)
        except RuntimeError as e:         # a torch build without row-wise fp8 scaling
            result["unfused"] = {"ms": None, "error": str(e).splitlines()[0][:200]}
        else:
            ms_u, ms_g = tu["ms_per_step"], tg["ms_per_step"]
            result["unfused"] = {"ms": round(ms_u, 5), "cv": tu["cv"],
                                 "tflops": round(flops / (ms_u * 1e-3) / 1e12, 2),
                                 "sequence": ("torch._scaled_mm (vendor fp8 GEMM, row-wise scales)"
                                              if spec.dtype == "e4m3" else "torch.mm (vendor BLAS)")
                                 + " then one eager kernel per tail op"}
            result["gemm_only"] = {"ms": round(ms_g, 5), "cv": tg["cv"],
                                   "tflops": round(flops / (ms_g * 1e-3) / 1e12, 2)}
            result["speedup_vs_unfused"] = round(ms_u / ms, 3)

    if not args.no_cpu_baseline:
        torch.cuda.synchronize()
        cpu = cpu_oracle_fgemm(spec, inp, args.cpu_seconds, out, np)
        result["cpu_baseline"], rep = cpu
        result["parity_sample"] = {"rel_err": rep.rel_err, "tol": rep.tol, "ok": bool(rep.ok),
                                   "rows_compared": int(cpu[0]["rows"])}
    return result


def cpu_oracle_fgemm(spec, inp, budget_s, out, np):
    """Time the fp64 oracle on a growing sample of rows until ~budget_s (or
    all rows), and compare every row it computed with the GPU output."""
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
    rows, t_total, flops_total, n_rows, refs = 8, 0.0, 0.0, 0, []
    while t_total < budget_s and n_rows < spec.M:
        r = min(rows, spec.M - n_rows)
        sel = slice(n_rows, n_rows + r)
        t0 = time.perf_counter()
        ref = ref_fgemm(x64[sel], W64, b, spec.ops, spec.reduction, spec.gn_groups, spec.gn_eps,
                        inp.get("gamma"), inp.get("beta"), spec.post_ops)
        t_total += time.perf_counter() - t0
        refs.append(ref)
        flops_total += 2.0 * r * spec.N * spec.K
        n_rows += r
        rows *= 2
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    rep = compare(got[:n_rows], np.concatenate(refs), {"f32": "f32", "bf16": "bf16", "e4m3": "e4m3"}[spec.dtype])
    return ({"value": flops_total / t_total / 1e12, "unit": "TFLOP/s", "cores": int(threads),
             "kind": "oracle",
             "sample": f"{n_rows} of {spec.M} output rows (all {spec.N} columns, K={spec.K}), "
                       f"fp64 numpy matmul + tail, {t_total:.1f} s",
             "seconds": round(t_total, 2), "rows": n_rows}, rep)


def grouped_epi(kernel_name):
    """0 for the gate/up grouped GEMM, 1 for the down GEMM, None otherwise."""
    m = re.search(r"grouped_kernel<fg::Tile<[^>]*>,\s*([01])(?:,\s*(?:true|false))?>\(", kernel_name) or \
        re.search(r"grouped_kernel.*Li([01])E(?:Lb[01]E)?EEvNS_11GroupedArgsE", kernel_name)
    return int(m.group(1)) if m else None


def moe_kernel_work(spec, epi, active, S):
    """Algorithmic FLOP and bytes of one launch of a grouped GEMM: the
    weights of the experts that receive a slot read once, the activation
    rows read once, the output written once."""
    es = 1 if spec.w_dtype == "e4m3" else 2
    H, I = spec.H, spec.I
    if epi == 0:
        flops = 2.0 * S * H * 2 * I
        nbytes = active * 2 * I * H * es + spec.T * H * es + S * I * 2
        if es == 1:
            nbytes += active * 2 * I * 4 + spec.T * 4
    else:
        flops = 2.0 * S * I * H
        nbytes = active * H * I * es + S * I * es + S * H * 4
        if es == 1:
            nbytes += active * H * 4 + S * 4
    return flops, nbytes


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
    bufs = api.moe_ffn(x, lg, wgu, wd, sgu, sd, top_k=spec.k)

    def fused():
        api.moe_ffn(x, lg, wgu, wd, sgu, sd, top_k=spec.k, buffers=bufs)

    tim, clk, kernels = measure(fused, args, torch)
    ms = tim["ms_per_step"]
    counts = np.diff(bufs.offsets.cpu().numpy())
    active = int(np.sum(counts > 0))
    S = spec.T * spec.k
    flops = spec.flops()
    nbytes = spec.bytes(active)
    tflops = flops / (ms * 1e-3) / 1e12
    gbs = nbytes / (ms * 1e-3) / 1e9
    decode = spec.T <= 256
    peak_c = PEAK_BF16_TFLOPS if spec.w_dtype == "bf16" else PEAK_FP8_TFLOPS
    kname, kst = dominant(kernels)
    epi = grouped_epi(kname)
    if epi is None:
        raise RuntimeError(f"the dominant kernel of the MoE step is not a grouped GEMM: {kname}")
    k_flops, k_bytes = moe_kernel_work(spec, epi, active, S)
    sec = kst["avg_us"] * 1e-6
    common = {"kernel": kname, "avg_launch_us": kst["avg_us"], "algorithmic_flops_per_launch": k_flops,
              "algorithmic_bytes_per_launch": k_bytes,
              "traffic": measured_traffic(f"{spec.name}_{'gateup' if epi == 0 else 'down'}", MOE_KERNEL_SOURCES)}
    if decode:
        roof = {"bound": "hbm", "achieved": round(k_bytes / sec / 1e9, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(k_bytes / sec / 1e9 / PEAK_HBM_GBS, 4), **common}
        step_roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs / PEAK_HBM_GBS, 4)}
    else:
        roof = {"bound": "mfma", "achieved": round(k_flops / sec / 1e12, 2), "peak": peak_c, "unit": "TFLOP/s",
                "frac": round(k_flops / sec / 1e12 / peak_c, 4), **common}
        step_roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": peak_c, "unit": "TFLOP/s",
                     "frac": round(tflops / peak_c, 4)}
    step_roof.update({"scope": "whole step (all launches)", "algorithmic_flops": flops,
                      "algorithmic_bytes": nbytes, "active_experts": active,
                      "traffic": measured_traffic(spec.name, MOE_KERNEL_SOURCES)})
    result = base_result(
        args, tflops, tim, "e4m3" if spec.w_dtype == "e4m3" else "bf16",
        "synthetic (seeded: logits, x ~ N(0,1); W ~ N(0,0.02); see paper_2606_02963_amd/synth.py)",
        {"workload": f"MoE expert FFN step T={spec.T} H={spec.H} I={spec.I} E={spec.E} top-{spec.k} "
                     f"{spec.w_dtype} weights, clamped SwiGLU",
         "T": spec.T, "H": spec.H, "I": spec.I, "E": spec.E, "top_k": spec.k}, roof)
    result["step_roofline"] = step_roof
    result["hbm_gbs"] = round(gbs, 1)
    result["timing"] = timing_record(tim, clk)
    result["kernels"] = kernels
    if not args.no_cpu_baseline:
        torch.cuda.synchronize()
        cpu, rep, over, n_el = cpu_oracle_moe(spec, act, w, bufs.out, nbytes, decode, np, torch)
        result["cpu_baseline"] = cpu
        # every element within the tolerance after the full bound of legitimate
        # deviations, the normwise error within it, and at most 1e-4 of the
        # elements beyond it after the narrow bound (fp32-accurate h)
        result["parity_sample"] = {"rel_err": rep.rel_err, "normwise": rep.normwise, "tol": rep.tol,
                                   "beyond_tol_narrow_bound": over, "elements": n_el,
                                   "ok": bool(rep.ok and rep.normwise <= rep.tol and over <= 1e-4 * n_el),
                                   "tokens_compared": cpu["tokens"]}
    del w

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
            tu = timed_repeats(unfused, args.steps, args.warmup, args.min_repeat_seconds, torch)
        except RuntimeError as e:         # a torch build without row-wise fp8 scaling
            result["unfused"] = {"ms": None, "error": str(e).splitlines()[0][:200]}
        else:
            ms_u = tu["ms_per_step"]
            result["unfused"] = {"ms": round(ms_u, 5), "cv": tu["cv"],
                                 "tflops": round(flops / (ms_u * 1e-3) / 1e12, 2),
                                 "hbm_gbs": round(nbytes / (ms_u * 1e-3) / 1e9, 1),
                                 "sequence": "eager torch: topk, softmax, stable argsort, per-expert "
                                             + ("row quantisation + torch._scaled_mm (fp8) + elementwise "
                                                "clamped SwiGLU + row quantisation + torch._scaled_mm"
                                                if f8 else "torch.mm + elementwise clamped SwiGLU + torch.mm")
                                             + ", weighted scatter, slot sum"}
            result["speedup_vs_unfused"] = round(ms_u / ms, 3)
    return result


def cpu_oracle_moe(spec, act, w, out, step_bytes, decode, np, torch):
    """Time the fp64 oracle's MoE step on the host: the whole step at decode
    size (T = 64), the first 64 tokens of the prefill batch otherwise, and
    compare every token it computed with the GPU output. The oracle decodes
    each expert's weights to fp64 as part of its work."""
    from threadpoolctl import threadpool_info
    from oracle import bf16_decode, compare, e4m3_decode, ref_moe
    from oracle.compare import count_above

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
    over = count_above(got, ref["out"], "e4m3" if f8 else "bf16", slack=ref["out_bound_narrow"])
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
             "seconds": round(sec, 2), "tokens": int(n)}, rep, over, int(got.size))


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
        ms = timed_repeats(g.replay, max(args.steps // 5, 2), max(args.warmup // 5, 2), min(args.min_repeat_seconds, 0.25), torch)["ms_per_step"] / reps
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
        ms = timed_repeats(g.replay, max(args.steps // 5, 2), max(args.warmup // 5, 2), min(args.min_repeat_seconds, 0.25), torch)["ms_per_step"] / reps
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
        ms = timed_repeats(g.replay, max(args.steps // 5, 2), max(args.warmup // 5, 2), min(args.min_repeat_seconds, 0.25), torch)["ms_per_step"] / reps
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
