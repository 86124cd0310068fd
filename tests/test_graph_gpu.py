"""HIP-graph capture of the library's launches.

No entry point records a memset or synchronises, and the split-K arrival
counters carry an epoch that a replayed launch reuses (the last arrival
resets the count under the same epoch). Each case runs eagerly, is captured
into a graph and replayed several times; between replays the program does its
own eager work on the same workspace (which leaves counters of another epoch
behind) and synchronises; every replay must reproduce the eager result bit for
bit (the kernels are deterministic)."""

import numpy as np
import pytest
import torch

from paper_2606_02963_amd import api
from paper_2606_02963_amd.synth import FGEMM_SPECS, MoeSpec, make_fgemm_inputs, make_moe_activations, \
    make_moe_weights
from tests.gpu_helpers import dev_bf16, dev_f32, log, require_gpu

pytestmark = pytest.mark.gpu

REPLAYS = 3


def _fgemm_case(spec):
    inp = make_fgemm_inputs(spec, 7)
    x, W, b = dev_bf16(inp["x"]), dev_bf16(inp["W"]), dev_f32(inp["b"])
    g = dev_f32(inp["gamma"]) if "gamma" in inp else None
    be = dev_f32(inp["beta"]) if "beta" in inp else None
    plan = api.get_plan(spec.M, spec.N, spec.K, "bf16", spec.out, True, spec.ops, spec.reduction,
                        spec.gn_groups, spec.gn_eps, spec.post_ops)
    ws = torch.empty(max(plan.workspace_bytes(), 16), dtype=torch.uint8, device="cuda")
    shape = (spec.M,) if spec.reduction == "lse" else (spec.M, spec.N)
    dt = torch.float32 if spec.out == "f32" else torch.bfloat16

    def run(out):
        api.linear_epilogue(x, W, b, spec.ops, spec.reduction, spec.gn_groups, spec.gn_eps, g, be,
                            out_dtype=spec.out, out=out, workspace=ws, post_ops=spec.post_ops)

    return plan, run, lambda: torch.empty(shape, dtype=dt, device="cuda")


@pytest.mark.parametrize("spec", [
    FGEMM_SPECS["bf16_gelu_clamp"].scaled(M=1000, N=2056, K=4104),   # split-K over 4 slices
    FGEMM_SPECS["bf16_scale_lse_mish"].scaled(M=300, N=1000, K=264),  # two launches, post op
    FGEMM_SPECS["bf16_silu_gn"].scaled(M=2048, N=4096, K=128),
], ids=lambda s: s.name)
def test_fgemm_graph_replays_match_eager(spec):
    require_gpu()
    plan, run, alloc = _fgemm_case(spec)
    log(f"[graph] {spec.name} {plan.info()}")
    eager = alloc()
    run(eager)
    torch.cuda.synchronize()
    out_g = alloc()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(out_g)
    scratch = alloc()
    for r in range(REPLAYS):
        out_g.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, eager), f"replay {r} differs from the eager result"
        run(scratch)                 # eager work on the same workspace, another epoch
        torch.cuda.synchronize()
        assert torch.equal(scratch, eager)


def test_moe_step_graph_replays_match_eager():
    require_gpu()
    spec = MoeSpec("graph_decode", T=37, H=192, I=128, E=8, k=4)
    act, w = make_moe_activations(spec, 3), make_moe_weights(spec, 3)
    x, lg = dev_bf16(act["x"]), dev_f32(act["logits"])
    wgu, wd = dev_bf16(w["w_gate_up"]), dev_bf16(w["w_down"])
    bufs = api.moe_ffn(x, lg, wgu, wd, None, None, top_k=spec.k)
    torch.cuda.synchronize()
    eager = {k: getattr(bufs, k).clone() for k in ("out", "topk_idx", "topk_w", "perm", "offsets")}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        api.moe_ffn(x, lg, wgu, wd, None, None, top_k=spec.k, buffers=bufs)
    for r in range(REPLAYS):
        bufs.out.zero_()
        bufs.perm.fill_(-1)
        g.replay()
        torch.cuda.synchronize()
        for k, v in eager.items():
            assert torch.equal(getattr(bufs, k), v), f"replay {r}: {k} differs from the eager result"
        other = api.moe_ffn(x, lg, wgu, wd, None, None, top_k=spec.k)   # eager work in between
        torch.cuda.synchronize()
        assert torch.equal(other.out, eager["out"])
