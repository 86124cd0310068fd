"""The allocation-free MoE entry point (moe_grouped_ffn_noalloc) against the
workspace entry point (moe_grouped_ffn), through the C ABI.

Both run the same kernels on the same inputs, so every output must agree
bit for bit: token outputs, top-k indices and weights, the permutation and
the expert offsets. Each case makes two calls in a row on the static
scratch, the second with fewer tokens (and the other row-tile size), so
that anything a call depends on from the scratch's previous contents would
show up. The smaller call is also checked against the fp64 oracle."""

import numpy as np
import pytest
import torch

from oracle import bf16_decode, e4m3_decode, ref_moe
from paper_2606_02963_amd import _lib as L
from paper_2606_02963_amd import api
from paper_2606_02963_amd.synth import MoeSpec, make_moe_activations, make_moe_weights
from tests.gpu_helpers import check_moe_outputs, dev_bf16, dev_f32, dev_u8, host64, log, require_gpu

pytestmark = pytest.mark.gpu


def _noalloc(desc, x, lg, wgu, wd, sgu, sd):
    T, k, E, H = desc.T, desc.top_k, desc.E, desc.H
    dev = x.device
    out = torch.full((T, H), float("nan"), dtype=torch.bfloat16, device=dev)
    idx = torch.full((T, k), -1, dtype=torch.int32, device=dev)
    w = torch.full((T, k), float("nan"), dtype=torch.float32, device=dev)
    perm = torch.full((T * k,), -1, dtype=torch.int32, device=dev)
    offs = torch.full((E + 1,), -1, dtype=torch.int32, device=dev)
    p = lambda t: t.data_ptr() if t is not None else None  # noqa: E731
    L.moe_grouped_ffn_noalloc(desc, p(x), p(lg), p(wgu), p(wd), p(sgu), p(sd), p(out), p(idx), p(w), p(perm),
                              p(offs), torch.cuda.current_stream().cuda_stream)
    return out, idx, w, perm, offs


@pytest.mark.parametrize("w_dtype,T1,T2", [("bf16", 300, 40), ("e4m3", 256, 9)])
def test_noalloc_matches_workspace_entry_point(w_dtype, T1, T2):
    require_gpu()
    base = MoeSpec(f"noalloc_{w_dtype}", T=T1, H=2880, I=2880, E=8, k=4, w_dtype=w_dtype)
    w = make_moe_weights(base, 31)
    if w_dtype == "bf16":
        wgu, wd, sgu, sd = dev_bf16(w["w_gate_up"]), dev_bf16(w["w_down"]), None, None
    else:
        wgu, wd = dev_u8(w["w_gate_up"]), dev_u8(w["w_down"])
        sgu, sd = dev_f32(w["s_gate_up"]), dev_f32(w["s_down"])
    for T in (T1, T2):
        spec = MoeSpec(base.name, T=T, H=base.H, I=base.I, E=base.E, k=base.k, w_dtype=w_dtype)
        log(f"[noalloc] {w_dtype} T={T} H={spec.H} I={spec.I} E={spec.E} k={spec.k}")
        act = make_moe_activations(spec, 32 + T)
        x, lg = dev_bf16(act["x"]), dev_f32(act["logits"])
        desc = L.moe_desc(T, spec.H, spec.I, spec.E, spec.k, w_dtype)
        assert L.moe_workspace_bytes(desc) <= L.moe_noalloc_scratch_bytes()
        ref_run = api.moe_ffn(x, lg, wgu, wd, sgu, sd, top_k=spec.k)
        got = _noalloc(desc, x, lg, wgu, wd, sgu, sd)
        torch.cuda.synchronize()
        assert torch.equal(got[0].view(torch.int16), ref_run.out.view(torch.int16)), "token outputs differ"
        assert torch.equal(got[1], ref_run.topk_idx)
        assert torch.equal(got[2].view(torch.int32), ref_run.topk_w.view(torch.int32))
        assert torch.equal(got[3], ref_run.perm)
        assert torch.equal(got[4], ref_run.offsets)
    # the second (smaller) call against the oracle as well
    f8 = w_dtype == "e4m3"
    if f8:
        W = lambda e: (e4m3_decode(w["w_gate_up"][e]) * w["s_gate_up"][e][:, None].astype(np.float64),  # noqa: E731
                       e4m3_decode(w["w_down"][e]) * w["s_down"][e][:, None].astype(np.float64))
    else:
        W = lambda e: (bf16_decode(w["w_gate_up"][e]), bf16_decode(w["w_down"][e]))  # noqa: E731
    ref = ref_moe(bf16_decode(act["x"]), act["logits"].astype(np.float64), W, spec.k,
                  storage="e4m3" if f8 else "bf16", act_quant=f8, with_bound=True)
    check_moe_outputs(host64(got[0]), ref, "e4m3" if f8 else "bf16")


def test_noalloc_graph_replays_match_eager():
    """The callers this entry point is for include code under HIP graph
    capture: a captured step, replayed with other calls on the same static
    scratch in between, must reproduce the eager result bit for bit."""
    require_gpu()
    spec = MoeSpec("noalloc_graph", T=37, H=192, I=128, E=8, k=4)
    other = MoeSpec("noalloc_graph_other", T=21, H=192, I=128, E=8, k=4)
    w = make_moe_weights(spec, 41)
    wgu, wd = dev_bf16(w["w_gate_up"]), dev_bf16(w["w_down"])
    act, act2 = make_moe_activations(spec, 42), make_moe_activations(other, 43)
    x, lg = dev_bf16(act["x"]), dev_f32(act["logits"])
    x2, lg2 = dev_bf16(act2["x"]), dev_f32(act2["logits"])
    desc = L.moe_desc(spec.T, spec.H, spec.I, spec.E, spec.k, "bf16")
    desc2 = L.moe_desc(other.T, other.H, other.I, other.E, other.k, "bf16")
    eager = _noalloc(desc, x, lg, wgu, wd, None, None)           # also looks up the scratch address
    eager2 = _noalloc(desc2, x2, lg2, wgu, wd, None, None)
    torch.cuda.synchronize()
    bufs = [torch.empty_like(t) for t in eager]
    p = lambda t: t.data_ptr()  # noqa: E731
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        L.moe_grouped_ffn_noalloc(desc, p(x), p(lg), p(wgu), p(wd), None, None, *[p(b) for b in bufs],
                                  torch.cuda.current_stream().cuda_stream)
    for r in range(3):
        for b in bufs:
            b.zero_()
        g.replay()
        torch.cuda.synchronize()
        for name, got, want in zip(("out", "topk_idx", "topk_w", "perm", "offsets"), bufs, eager):
            assert torch.equal(got.view(torch.int8), want.view(torch.int8)), f"replay {r}: {name} differs"
        between = _noalloc(desc2, x2, lg2, wgu, wd, None, None)   # another call on the same scratch
        torch.cuda.synchronize()
        assert torch.equal(between[0].view(torch.int16), eager2[0].view(torch.int16))
