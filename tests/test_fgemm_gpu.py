"""GPU parity of the fused GEMM + tail against the fp64 oracle.

Every case runs the HIP kernels through the C ABI on seeded inputs and
compares element by element with ``oracle.ref_fgemm`` under the RMS-floored
relative error: ≤ 1e-4 for fp32 inputs, ≤ 1e-2 for bf16 inputs. Sizes span
several tiles with ragged M, N and K tails and cover every bf16 tile
configuration (128×128, 256×128, 256×256, and 256×256 with K split over
slices) with each tail; the full-size workloads are checked on every output
element."""

import numpy as np
import pytest
import torch

from oracle import bf16_decode, compare, e4m3_decode, ref_fgemm
from paper_2606_02963_amd import api
from paper_2606_02963_amd import _lib as L
from paper_2606_02963_amd.synth import FGEMM_SPECS, FgemmSpec, make_fgemm_inputs
from tests.gpu_helpers import dev_bf16, dev_f32, dev_u8, host64, log, require_gpu

pytestmark = pytest.mark.gpu


def _device_inputs(spec, inp):
    if spec.dtype == "f32":
        x, W = dev_f32(inp["x"]), dev_f32(inp["W"])
        x64, W64 = inp["x"].astype(np.float64), inp["W"].astype(np.float64)
    elif spec.dtype == "e4m3":
        # the oracle reads the exact values the fp8 MFMA multiplies: decoded
        # codes times the per-row scales
        x, W = dev_u8(inp["x"]), dev_u8(inp["W"])
        x64 = e4m3_decode(inp["x"]) * inp["x_scale"].astype(np.float64)[:, None]
        W64 = e4m3_decode(inp["W"]) * inp["w_scale"].astype(np.float64)[:, None]
    else:
        x, W = dev_bf16(inp["x"]), dev_bf16(inp["W"])
        x64, W64 = bf16_decode(inp["x"]), bf16_decode(inp["W"])
    b = dev_f32(inp["b"])
    g = dev_f32(inp["gamma"]) if "gamma" in inp else None
    be = dev_f32(inp["beta"]) if "beta" in inp else None
    return (x, W, b, g, be), (x64, W64)


def run_spec(spec, seed=0, rows=None, inp=None, with_bias=True):
    require_gpu()
    log(f"[fgemm] {spec.name} M={spec.M} N={spec.N} K={spec.K} seed={seed}")
    inp = inp if inp is not None else make_fgemm_inputs(spec, seed)
    (x, W, b, g, be), (x64, W64) = _device_inputs(spec, inp)
    sx = dev_f32(inp["x_scale"]) if spec.dtype == "e4m3" else None
    sw = dev_f32(inp["w_scale"]) if spec.dtype == "e4m3" else None
    y = api.linear_epilogue(x, W, b if with_bias else None, spec.ops, spec.reduction, spec.gn_groups,
                            spec.gn_eps, g, be, out_dtype=spec.out, post_ops=spec.post_ops,
                            x_scale=sx, w_scale=sw)
    torch.cuda.synchronize()
    got = host64(y)
    sel = slice(None) if rows is None else np.asarray(rows)
    ref = ref_fgemm(x64[sel], W64, inp["b"].astype(np.float64) if with_bias else None, spec.ops,
                    spec.reduction, spec.gn_groups, spec.gn_eps,
                    inp.get("gamma"), inp.get("beta"), spec.post_ops)
    rep = compare(got[sel], ref, {"f32": "f32", "bf16": "bf16", "e4m3": "e4m3"}[spec.dtype])
    log(f"    {rep}")
    assert rep.ok, f"{spec.name}: {rep}"
    return y


C1, C2, C3, C4 = (FGEMM_SPECS[k] for k in ("tiny_f32_relu_x2", "bf16_gelu_clamp", "bf16_lse", "bf16_silu_gn"))

SMALL = [
    # the smallest shapes each input type and reduction admits: one row, one
    # 16-byte chunk of K (a partial stage only), one output chunk; LSE over
    # a single column; one GroupNorm group of 8 channels (the second launch)
    FgemmSpec("min_bf16", 1, 8, 8, "bf16", 0.1, (("gelu_tanh",),)),
    FgemmSpec("min_f32", 1, 4, 4, "f32", 0.2, (("relu",),)),
    FgemmSpec("min_e4m3", 1, 8, 16, "e4m3", 0.1, (("silu",),), out_dtype="bf16"),
    FgemmSpec("min_lse_one_column", 3, 1, 8, "bf16", 0.1, (("add", -0.25),), "lse"),
    FgemmSpec("min_gn_one_group", 2, 8, 8, "bf16", 0.1, (), "groupnorm", 1, 1e-5),
    C1,                                               # the fp32 workload at full size
    C1.scaled(M=77, N=200, K=36, name="f32_ragged"),  # K tail (36 % 32), ragged M, N
    C2.scaled(M=300, N=520, K=264),                   # 128×128 tiles, ragged, K tail
    C2.scaled(M=2000, N=4104, K=136),                 # 256×256 tiles, ragged, K tail
    C2.scaled(M=4000, N=4000, K=200),                 # 256×256 tiles filling the chip, ragged
    C2.scaled(M=3900, N=4000, K=200),                 # last row tile of 60 rows: its lower waves idle
    C2.scaled(M=1000, N=2056, K=4104),                # split-K over 4 slices, ragged, K tail
    C2.scaled(M=512, N=1024, K=8192),                 # split-K over 4 slices, 8 tiles
    C3.scaled(M=300, N=1000, K=264),                  # LSE across 8 N tiles, ragged N
    C3.scaled(M=70, N=100, K=64),                     # LSE inside one partial tile
    C3.scaled(M=2048, N=4096, K=128),                 # LSE with 256×128 tiles
    C3.scaled(M=4000, N=4000, K=200),                 # LSE with 256×256 tiles, ragged N
    C3.scaled(M=3900, N=4000, K=200),                 # LSE, last row tile of 60 rows (idle waves)
    C3.scaled(M=1000, N=2056, K=4104),                # LSE after a split-K gather
    C4.scaled(M=300, N=512, K=264),                   # GroupNorm, 4 groups of 128
    FgemmSpec("gn64_ragged", 133, 320, 72, "bf16", 1 / 64, (("silu",),), "groupnorm", 5, 1e-5),
    C4.scaled(M=2048, N=4096, K=128),                 # GroupNorm with 256×128 tiles
    C4.scaled(M=4000, N=4096, K=200),                 # GroupNorm with 256×256 tiles
    C4.scaled(M=3900, N=4096, K=200),                 # GroupNorm, last row tile of 60 rows (idle waves)
    C4.scaled(M=1000, N=2048, K=4104),                # GroupNorm after a split-K gather
    FgemmSpec("f32_gn_lse_chain", 96, 256, 64, "f32", 0.2, (("gelu_tanh",), ("scale", 1.5)), "lse"),
    FgemmSpec("f32_gn", 96, 256, 64, "f32", 0.2, (("silu",),), "groupnorm", 2, 1e-5),
    FgemmSpec("bf16_all_ops", 130, 264, 200, "bf16", 0.1,
              (("scale", 0.75), ("add", 0.1), ("gelu_tanh",), ("silu",), ("relu",),
               ("clamp", -0.5, 0.25), ("scale", -2.0), ("add", 0.5))),
    FgemmSpec("bf16_f32out", 130, 264, 200, "bf16", 0.1, (("gelu_tanh",),), out_dtype="f32"),
]


@pytest.mark.parametrize("spec", SMALL, ids=lambda s: s.name)
def test_parity_small(spec):
    run_spec(spec)


@pytest.mark.parametrize("spec", SMALL, ids=lambda s: s.name)
def test_parity_small_other_seed(spec):
    run_spec(spec, seed=1)


# Row LogSumExp at small M (the 16 / 64 / 256-row shapes of the one-launch
# comparison, N = 8192, K = 4096, split-K), ragged rows and columns, one
# partial n-tile, and a post op.
LSE_SMALL_M = [
    C3.scaled(M=16, N=8192, K=4096),
    C3.scaled(M=64, N=8192, K=4096),
    C3.scaled(M=256, N=8192, K=4096),
    C3.scaled(M=5, N=1000, K=264),
    C3.scaled(M=33, N=96, K=64),
    FGEMM_SPECS["bf16_scale_lse_mish"].scaled(M=250, N=1000, K=264),
]


@pytest.mark.parametrize("spec", LSE_SMALL_M, ids=lambda s: s.name)
def test_parity_lse_small_m(spec):
    run_spec(spec)


# GroupNorm over every kind of group width: 16 and 32 channels inside one
# wave, 64 inside one wave on the 256×256 tile too, 256 channels on the
# 256×256 tile (across its four wave columns), and groups no tile holds in
# registers — wider than the tile (512, 2048), or not whole 16-column
# fragments (24, 96) — through the second launch, with post ops, e4m3 and
# fp32 inputs and fp32 output.
_SILU = (("silu",),)
GN_WIDTHS = [
    FgemmSpec("gn16", 300, 512, 264, "bf16", 1 / 16, _SILU, "groupnorm", 32, 1e-5),
    FgemmSpec("gn32", 200, 1024, 136, "bf16", 1 / 16, _SILU, "groupnorm", 32, 1e-5),
    FgemmSpec("gn64_huge", 4000, 4096, 200, "bf16", 1 / 16, _SILU, "groupnorm", 64, 1e-5),
    FgemmSpec("gn256", 512, 2048, 256, "bf16", 1 / 16, _SILU, "groupnorm", 8, 1e-5),
    FgemmSpec("gn512_two_pass", 300, 4096, 264, "bf16", 1 / 16, _SILU, "groupnorm", 8, 1e-5,
              post_ops=(("leaky_relu", 0.01), ("scale", 2.0))),
    FgemmSpec("gn2048_two_pass", 130, 4096, 128, "bf16", 1 / 16, _SILU, "groupnorm", 2, 1e-5),
    FgemmSpec("gn24_two_pass", 130, 480, 64, "bf16", 1 / 8, _SILU, "groupnorm", 20, 1e-5),
    FgemmSpec("gn96_two_pass", 77, 384, 72, "bf16", 1 / 8, _SILU, "groupnorm", 4, 1e-5, out_dtype="f32"),
    FgemmSpec("gn256_e4m3_two_pass", 256, 2048, 256, "e4m3", 1 / 16, _SILU, "groupnorm", 8, 1e-5),
    FgemmSpec("gn16_f32", 96, 256, 64, "f32", 0.2, _SILU, "groupnorm", 16, 1e-5),
    FgemmSpec("gn512_f32_two_pass", 96, 1024, 64, "f32", 0.2, _SILU, "groupnorm", 2, 1e-5),
]


@pytest.mark.parametrize("spec", GN_WIDTHS, ids=lambda s: s.name)
def test_parity_groupnorm_widths(spec):
    gw = spec.N // spec.gn_groups
    plan = api.get_plan(spec.M, spec.N, spec.K, spec.dtype, spec.out, True, spec.ops, "groupnorm",
                        spec.gn_groups, spec.gn_eps, spec.post_ops)
    log(f"[gn] width {gw}: {plan.info()}")
    assert plan.info()["launches"] == (2 if "two_pass" in spec.name else 1)
    run_spec(spec)


# Table III tail chains: Mish, LeakyReLU and elementwise ops after the
# reduction, on every tile configuration and after a split-K gather.
T3 = [FGEMM_SPECS[k] for k in ("bf16_scale_lse_mish", "bf16_gn_swish_mul_swish", "bf16_gn_lrelu_sum",
                               "bf16_swish_sum_gn")]
TABLE3 = []
for _s in T3:
    TABLE3 += [
        _s.scaled(M=300, N=512, K=264),        # 128×128 tiles, ragged M, K tail
        _s.scaled(M=2048, N=4096, K=128),      # 256×128 tiles
        _s.scaled(M=4000, N=4096, K=200),      # 256×256 tiles, ragged M
        _s.scaled(M=1000, N=2048, K=4104),     # split-K gather, K tail
    ]
TABLE3 += [
    # the LSE chain with a ragged N inside the last tile
    T3[0].scaled(M=300, N=1000, K=264),
    # Mish and LeakyReLU as ordinary ops before a plain store, and large
    # arguments (weights ×16 push |z| past Mish's exponent clamp at 20)
    FgemmSpec("bf16_mish_lrelu", 130, 264, 200, "bf16", 0.1, (("mish",), ("leaky_relu", 0.2))),
    FgemmSpec("bf16_mish_large", 130, 264, 512, "bf16", 1.6, (("mish",),)),
    FgemmSpec("f32_lse_mish", 96, 256, 64, "f32", 0.2, (("scale", 2.0),), "lse", post_ops=(("mish",),)),
    FgemmSpec("f32_gn_lrelu", 96, 256, 64, "f32", 0.2, (), "groupnorm", 2, 1e-5,
              post_ops=(("leaky_relu", 0.01), ("scale", 2.0))),
    # the longest post chains (8 ops) after each reduction, the GroupNorm one
    # also in the second launch (groups of 96 channels)
    FgemmSpec("bf16_lse_post8", 130, 1000, 200, "bf16", 0.1, (("add", -0.25),), "lse",
              post_ops=(("scale", 0.5), ("add", 0.1), ("mish",), ("leaky_relu", 0.1), ("silu",),
                        ("gelu_tanh",), ("clamp", -1.0, 2.0), ("relu",))),
    FgemmSpec("bf16_gn_post8", 130, 512, 200, "bf16", 0.1, (("silu",),), "groupnorm", 4, 1e-5,
              post_ops=(("scale", 0.5), ("add", 0.1), ("mish",), ("leaky_relu", 0.1), ("silu",),
                        ("gelu_tanh",), ("clamp", -1.0, 2.0), ("relu",))),
    FgemmSpec("bf16_gn96_post8", 130, 576, 200, "bf16", 0.1, (("silu",),), "groupnorm", 6, 1e-5,
              post_ops=(("scale", 0.5), ("add", 0.1), ("mish",), ("leaky_relu", 0.1), ("silu",),
                        ("gelu_tanh",), ("clamp", -1.0, 2.0), ("relu",))),
]


@pytest.mark.parametrize("spec", TABLE3, ids=lambda s: s.name)
def test_parity_table3_chains(spec):
    run_spec(spec)


# W8A8 (e4m3 codes, per-row fp32 scales): both e4m3 tiles, ragged M, N and
# K tails (K = 272: two full 128-byte stages and a 16-byte tail), every
# reduction, fp32 output.
E8 = FGEMM_SPECS["e4m3_gelu_clamp"]
E4M3 = [
    E8.scaled(M=300, N=520, K=272),                    # 128×128 tiles, ragged, K tail
    E8.scaled(M=1000, N=4104, K=1040),                 # 256×128 tiles, ragged, K tail
    E8.scaled(M=2048, N=4096, K=512),                  # 256×128 tiles, full
    FgemmSpec("e4m3_lse_mish", 300, 1000, 272, "e4m3", 1 / 16, (("scale", 2.0),), "lse",
              post_ops=(("mish",),)),
    FgemmSpec("e4m3_silu_gn", 520, 4096, 256, "e4m3", 1 / 16, (("silu",),), "groupnorm", 32, 1e-5),
    FgemmSpec("e4m3_f32out", 130, 264, 208, "e4m3", 0.1, (("gelu_tanh",),), out_dtype="f32"),
]


@pytest.mark.parametrize("spec", E4M3, ids=lambda s: s.name)
def test_parity_e4m3(spec):
    run_spec(spec)


def test_parity_e4m3_full_size():
    run_spec(E8)


def test_e4m3_plan_needs_scales():
    require_gpu()
    spec = E8.scaled(M=64, N=128, K=64)
    inp = make_fgemm_inputs(spec, 2)
    x, W = dev_u8(inp["x"]), dev_u8(inp["W"])
    plan = api.get_plan(spec.M, spec.N, spec.K, "e4m3", "bf16", False)
    out = torch.empty((spec.M, spec.N), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(L.FgError) as ei:
        L.fgemm_run(plan, x.data_ptr(), W.data_ptr(), None, None, None, out.data_ptr(), None, 0, None)
    assert ei.value.status == L.FG_ERR_INVALID_ARG
    with pytest.raises(ValueError):
        api.linear_epilogue(x, W, None, ())


@pytest.mark.parametrize("spec", T3, ids=lambda s: s.name)
def test_parity_table3_full_size(spec):
    run_spec(spec)


@pytest.mark.parametrize("spec", [C2, C3, C4], ids=lambda s: s.name)
def test_parity_full_size(spec):
    # every output element of the benchmark workload, in the launch
    # configuration the benchmark times
    run_spec(spec)


@pytest.mark.parametrize("M,K", [(300, 256), (1000, 1024), (256, 4096)])
def test_identity_weight_empty_tail_is_bit_exact(M, K):
    """W = I (N = K) with no tail ops: each output is one product x·1 plus the
    bias, so the result must be bf16(x + b) exactly. x and b are chosen so
    that x + b is exact in fp32 (both on a 2^-13 grid with magnitudes below
    16), hence the single rounding to bf16 has one correct answer. Covers
    the 128×128, 256×128 and 256×256 / split-K tiles."""
    require_gpu()
    rng = np.random.default_rng(40 + M)
    xv = rng.standard_normal((M, K)).astype(np.float32)
    xv = np.where(np.abs(xv) < 2.0 ** -6, 0.0, xv).astype(np.float32)
    xb = torch.from_numpy(xv).to(torch.bfloat16)
    bv = (rng.integers(-2 ** 13, 2 ** 13, K) / 2.0 ** 13).astype(np.float32)
    bv = np.where(np.abs(bv) < 2.0 ** -6, 0.0, bv).astype(np.float32)
    eye = torch.eye(K, dtype=torch.bfloat16)
    plan = api.get_plan(M, K, K, "bf16", "bf16", True, ())
    log(f"[fgemm] identity M={M} K={K} {plan.info()}")
    y = api.linear_epilogue(xb.cuda(), eye.cuda(), dev_f32(bv), ())
    torch.cuda.synchronize()
    x64 = xb.double().numpy()
    want = x64 + bv.astype(np.float64)
    assert np.array_equal(want.astype(np.float32).astype(np.float64), want)     # x + b exact in fp32
    want_bits = torch.from_numpy(want.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy()
    assert np.array_equal(y.cpu().view(torch.int16).numpy(), want_bits)


@pytest.mark.parametrize("K", [128, 2880])
def test_e4m3_contraction_noise_within_the_moe_parity_neighbourhood(K):
    """The e4m3 MFMA does not sum its 128-wide dot products as IEEE fp32. Its
    error per output element must stay within the accumulation noise that the
    W8A8 MoE parity neighbourhood allows for (oracle.moe.f8_contraction_noise,
    from the oracle's exact values): one MFMA per dot product (K = 128) and
    the MoE contraction length (2880). No bias and no tail, fp32 output."""
    from oracle.moe import f8_contraction_noise
    require_gpu()
    spec = FgemmSpec(f"e4m3_dot_K{K}", 512, 1024, K, "e4m3", 0.05, (), out_dtype="f32")
    log(f"[fgemm] {spec.name} M={spec.M} N={spec.N} K={spec.K}")
    inp = make_fgemm_inputs(spec, 7)
    (x, W, _, _, _), (x64, W64) = _device_inputs(spec, inp)
    y = api.linear_epilogue(x, W, None, (), out_dtype="f32", x_scale=dev_f32(inp["x_scale"]),
                            w_scale=dev_f32(inp["w_scale"]))
    torch.cuda.synchronize()
    exact = ref_fgemm(x64, W64, None, ())
    rel = np.abs(host64(y) - exact) / f8_contraction_noise(x64, W64)
    log(f"    error / allowed noise: median {np.median(rel):.3g}, max {rel.max():.3g}")
    assert rel.max() <= 1.0


def test_identity_weight_gives_tail_of_x_plus_b():
    K = 256
    spec = FgemmSpec("identity", 64, K, K, "bf16", 1 / 16, (("scale", 0.5), ("gelu_tanh",), ("clamp", -1.0, 1.0)))
    inp = make_fgemm_inputs(spec, 3)
    eye = torch.eye(K, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    inp["W"] = eye
    y = run_spec(spec, inp=inp)
    # single nonzero product per output: identical to the tail of x + b evaluated in fp32 on the host
    u = (torch.from_numpy(bf16_decode(inp["x"])).float() + torch.from_numpy(inp["b"])) * 0.5
    ref = torch.clamp(torch.nn.functional.gelu(u, approximate="tanh"), -1, 1)
    assert compare(host64(y), ref.double().numpy(), "bf16").ok


def test_zero_weight_and_zero_k():
    spec = FgemmSpec("zeroW", 40, 128, 64, "bf16", 0.5, (("relu",), ("scale", 2.0)))
    inp = make_fgemm_inputs(spec, 4)
    inp["W"] = np.zeros_like(inp["W"])
    y = run_spec(spec, inp=inp)
    want = np.maximum(inp["b"].astype(np.float64), 0) * 2
    assert np.array_equal(host64(y), np.tile(bf16_decode(
        torch.from_numpy(want.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)),
        (40, 1)))
    # K = 0: z = b exactly
    x = torch.empty((5, 0), dtype=torch.bfloat16, device="cuda")
    W = torch.empty((128, 0), dtype=torch.bfloat16, device="cuda")
    b = dev_f32(inp["b"])
    y0 = api.linear_epilogue(x, W, b, ())
    torch.cuda.synchronize()
    assert torch.equal(y0.float().cpu(), b.to(torch.bfloat16).float().cpu().expand(5, 128))


def test_empty_m_enqueues_nothing():
    require_gpu()
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    W = torch.ones((128, 64), dtype=torch.bfloat16, device="cuda")
    y = api.linear_epilogue(x, W, None, (("relu",),))
    torch.cuda.synchronize()
    assert y.shape == (0, 128)


def test_repeat_runs_are_bit_identical_and_stream_aware():
    require_gpu()
    spec = C3.scaled(M=512, N=2048, K=512)
    inp = make_fgemm_inputs(spec, 5)
    (x, W, b, _, _), _ = _device_inputs(spec, inp)
    y1 = api.linear_epilogue(x, W, b, spec.ops, "lse")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y2 = api.linear_epilogue(x, W, b, spec.ops, "lse")
    s.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


def test_run_errors_on_device():
    require_gpu()
    x = torch.ones((8, 64), dtype=torch.bfloat16, device="cuda")
    W = torch.ones((128, 64), dtype=torch.bfloat16, device="cuda")
    plan = api.get_plan(8, 128, 64, "bf16", "f32", False, (), "lse")
    out = torch.empty(8, device="cuda")
    with pytest.raises(L.FgError) as ei:
        L.fgemm_run(plan, x.data_ptr(), W.data_ptr(), None, None, None, out.data_ptr(), None, 0,
                    torch.cuda.current_stream().cuda_stream)
    assert ei.value.status == L.FG_ERR_WORKSPACE


def test_split_k_ignores_workspace_contents_and_repeats_bit_identically():
    """The split-K arrival counters work from any initial value: a workspace
    full of random bytes gives the same, correct result, run after run."""
    require_gpu()
    spec = C2.scaled(M=1000, N=2056, K=4104)
    plan = api.get_plan(spec.M, spec.N, spec.K, "bf16", "bf16", True, spec.ops)
    assert plan.info()["k_slices"] == 4
    inp = make_fgemm_inputs(spec, 5)
    (x, W, b, _, _), (x64, W64) = _device_inputs(spec, inp)
    ws = torch.randint(0, 256, (plan.workspace_bytes(),), dtype=torch.uint8, device="cuda")
    outs = []
    for _ in range(3):
        outs.append(api.linear_epilogue(x, W, b, spec.ops, workspace=ws))
        ws[:512].random_(0, 256)              # scramble the counter words between runs
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    rows = np.array([0, 1, 255, 256, 511, 767, 998, 999])
    ref = ref_fgemm(x64[rows], W64, inp["b"].astype(np.float64), spec.ops)
    rep = compare(host64(outs[0])[rows], ref, "bf16")
    log(f"    {rep}")
    assert rep.ok, rep


def test_x_and_y_past_4_gib():
    """Maximum sizes along M: x and y each span more than 2^32 bytes
    (540 000 rows of 4096 bf16), so tile base offsets and output row offsets
    beyond 32 bits are exercised. x repeats a seeded 64-row block on the
    device; each sampled output row is checked against the oracle row of its
    block row (an output row depends only on its own input row)."""
    require_gpu()
    R, M = 64, 540_000
    spec = C2.scaled(M=R, N=4096, K=4096)
    inp = make_fgemm_inputs(spec, 11)
    (blk, W, b, _, _), (x64, W64) = _device_inputs(spec, inp)
    x = blk.repeat((M + R - 1) // R, 1)[:M]
    assert x.is_contiguous() and x.numel() * 2 > 2 ** 32
    log(f"[fgemm] offsets past 4 GiB M={M} N={spec.N} K={spec.K} "
        f"{api.get_plan(M, spec.N, spec.K, 'bf16', 'bf16', True, spec.ops).info()}")
    y = api.linear_epilogue(x, W, b, spec.ops)
    torch.cuda.synchronize()
    assert y.numel() * 2 > 2 ** 32
    first_past = 2 ** 32 // (spec.K * 2)            # first row whose offset needs 33 bits
    rows = np.array([0, 1, R - 1, 262_143, first_past - 1, first_past, first_past + 1, 530_001, M - 1])
    got = host64(y[torch.from_numpy(rows).cuda()])
    ref = ref_fgemm(x64, W64, inp["b"].astype(np.float64), spec.ops)[rows % R]
    rep = compare(got, ref, "bf16")
    log(f"    {rep}")
    assert rep.ok, rep
    del x, y


@pytest.mark.parametrize("M,N,K", [(16, 16, 1 << 21), (40, 24, (1 << 21) - 8)])
def test_k_at_the_row_limit(M, N, K):
    """Maximum K: rows of 4 MiB (bf16 K = 2^21, the plan's limit), and one
    8-element chunk short of it (a partial last stage), through split-K."""
    spec = FgemmSpec(f"rowlimit_{K}", M, N, K, "bf16", 1 / 1024.0, C2.ops)
    assert api.get_plan(M, N, K, "bf16", "bf16", True, spec.ops).info()["k_slices"] > 1
    run_spec(spec, seed=12)
