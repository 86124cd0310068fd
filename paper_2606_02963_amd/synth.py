"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke run.

This module holds no arithmetic of the method: it only draws random numbers
and stores them in the formats the library consumes (fp32, bf16 bit patterns,
or e4m3 weight codes with per-row fp32 scales, which stand in for a quantised
checkpoint). Both the HIP path and the CPU oracle read what it produces; the
oracle decodes the stored bits itself.

The workloads stand in for those of paper §IV: the KernelBench Level-2
"GEMM + tail-ops" problems run on Intel Arc B580 (§IV-B, Table III: Swish,
Scale, LogSumExp, GroupNorm tails) and the gpt-oss-20b MoE decode path on
B200 (§IV-A). Neither the benchmark suite nor the model is used; these are
seeded draws with the shapes and value distributions listed below.

Draw order per config: one ``numpy.random.default_rng(seed)`` (PCG64) stream
in the order x, W, b, γ, β; MoE: router logits, then tokens from that
stream, and each expert's weights from its own stream
``default_rng([seed, 1000 + e])`` (W_gate_up first, then W_down) so a single
expert can be regenerated without the others. N(0, σ) means standard
deviation σ. U(−a, a) is drawn in fp32 as (2u − 1)·a with u ~ U[0, 1).
bf16 values are the RNE roundings of the fp32 draws.
"""

from dataclasses import dataclass, field
import math

import numpy as np
import torch


# --------------------------------------------------------------------------
# storage helpers (format conversion only)

def to_bf16_bits(a):
    """fp32 numpy array -> uint16 bf16 bit patterns (RNE, via torch's cast)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def rows_to_e4m3(w):
    """Store an fp32 weight matrix [n, k] as e4m3fn codes with one fp32 scale
    per row: s = amax/448 (1 for a zero row), code = e4m3(w/s) (RNE,
    saturated). This is the offline weight format a quantised checkpoint
    would ship; it happens once, before any timed work."""
    w = torch.from_numpy(np.ascontiguousarray(w, dtype=np.float32))
    amax = w.abs().amax(dim=1, keepdim=True)
    s = torch.where(amax > 0, amax / 448.0, torch.ones_like(amax))
    q = (w / s).clamp_(-448.0, 448.0).to(torch.float8_e4m3fn)
    return q.view(torch.uint8).numpy(), s[:, 0].numpy().astype(np.float32)


def _uniform(rng, shape, a):
    return ((rng.random(shape, dtype=np.float32) * np.float32(2.0) - np.float32(1.0))
            * np.float32(a)).astype(np.float32)


def _normal(rng, shape, std):
    return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


# --------------------------------------------------------------------------
# fused GEMM + tail workloads

@dataclass(frozen=True)
class FgemmSpec:
    name: str
    M: int
    N: int
    K: int
    dtype: str                    # "f32", "bf16" or "e4m3" (x, W); out dtype follows
    w_bound: float                # W, b ~ U(-w_bound, w_bound)
    ops: tuple                    # ((kind, a, b), ...) applied after +b
    reduction: str = None         # None | "lse" | "groupnorm"
    gn_groups: int = 0
    gn_eps: float = 1e-5
    out_dtype: str = None         # default: f32 for f32/LSE, else bf16
    post_ops: tuple = ()          # ops applied to the reduction's result

    @property
    def out(self):
        if self.out_dtype:
            return self.out_dtype
        return "f32" if (self.dtype == "f32" or self.reduction == "lse") else "bf16"

    def flops(self):
        return 2.0 * self.M * self.N * self.K

    def bytes(self):
        """Algorithmic bytes: each input read once, the output written once."""
        e = {"f32": 4, "bf16": 2, "e4m3": 1}[self.dtype]
        b = (self.M * self.K + self.N * self.K) * e + self.N * 4
        if self.dtype == "e4m3":
            b += (self.M + self.N) * 4            # per-row scales
        if self.reduction == "groupnorm":
            b += 2 * self.N * 4
        o = 4 if self.out == "f32" else 2
        b += (self.M if self.reduction == "lse" else self.M * self.N) * o
        return b

    def scaled(self, M=None, N=None, K=None, name=None):
        """Same tail and distributions at another shape (parity-test sizes)."""
        N2 = N or self.N
        groups = self.gn_groups
        if self.reduction == "groupnorm":
            groups = N2 // (self.N // self.gn_groups)
        return FgemmSpec(name or f"{self.name}@{M or self.M}x{N2}x{K or self.K}",
                         M or self.M, N2, K or self.K, self.dtype,
                         self.w_bound, self.ops, self.reduction, groups,
                         self.gn_eps, self.out_dtype, self.post_ops)


FGEMM_SPECS = {
    # ReLU then ×2 on a tiny fp32 linear; x ~ N(0,1), W, b ~ U(±1/16)
    "tiny_f32_relu_x2": FgemmSpec("tiny_f32_relu_x2", 128, 256, 256, "f32", 1 / 16,
                                  (("relu",), ("scale", 2.0))),
    # clamp(GELU_tanh((x·Wᵀ + b)·0.5), −1, 1); W, b ~ U(±1/√8192)
    "bf16_gelu_clamp": FgemmSpec("bf16_gelu_clamp", 1024, 8192, 8192, "bf16",
                                 1 / math.sqrt(8192),
                                 (("scale", 0.5), ("gelu_tanh",), ("clamp", -1.0, 1.0))),
    # LSE over 8192 columns of x·Wᵀ + b − 0.25; W, b ~ U(±1/64)
    "bf16_lse": FgemmSpec("bf16_lse", 4096, 8192, 4096, "bf16", 1 / 64,
                          (("add", -0.25),), "lse"),
    # GroupNorm(32 × 128, eps 1e-5)(SiLU(x·Wᵀ + b)); γ ~ U(0.5,1.5), β ~ N(0,0.1)
    "bf16_silu_gn": FgemmSpec("bf16_silu_gn", 2048, 4096, 4096, "bf16", 1 / 64,
                              (("silu",),), "groupnorm", 32, 1e-5),
    # the GELU/clamp workload in the W8A8 form: x and W stored as e4m3 codes
    # with one fp32 scale per row (the format of the MoE fp8 variant)
    "e4m3_gelu_clamp": FgemmSpec("e4m3_gelu_clamp", 1024, 8192, 8192, "e4m3",
                                 1 / math.sqrt(8192),
                                 (("scale", 0.5), ("gelu_tanh",), ("clamp", -1.0, 1.0)), out_dtype="bf16"),
    # The four tail chains of paper Table III. Their problem shapes are not
    # in the paper; they take the shapes of the LSE and GroupNorm workloads
    # above. "Mul" is read as a scalar multiply, "Sum" as adding a constant
    # (Swish → Sum → GN) or the tensor to itself, x + x = 2x (GN → LReLU →
    # Sum); the LeakyReLU slope is 0.01.
    "bf16_scale_lse_mish": FgemmSpec("bf16_scale_lse_mish", 4096, 8192, 4096, "bf16", 1 / 64,
                                     (("scale", 2.0),), "lse", post_ops=(("mish",),)),
    "bf16_gn_swish_mul_swish": FgemmSpec("bf16_gn_swish_mul_swish", 2048, 4096, 4096, "bf16", 1 / 64,
                                         (), "groupnorm", 32, 1e-5,
                                         post_ops=(("silu",), ("scale", 1.5), ("silu",))),
    "bf16_gn_lrelu_sum": FgemmSpec("bf16_gn_lrelu_sum", 2048, 4096, 4096, "bf16", 1 / 64,
                                   (), "groupnorm", 32, 1e-5,
                                   post_ops=(("leaky_relu", 0.01), ("scale", 2.0))),
    "bf16_swish_sum_gn": FgemmSpec("bf16_swish_sum_gn", 2048, 4096, 4096, "bf16", 1 / 64,
                                   (("silu",), ("add", 0.25)), "groupnorm", 32, 1e-5),
}


def make_fgemm_inputs(spec, seed=0):
    """Draw x, W, b (and γ, β for GroupNorm) for ``spec``.

    Returns a dict of numpy arrays in storage form: x [M,K] and W [N,K] as
    fp32 (dtype f32), uint16 bf16 bits (dtype bf16) or uint8 e4m3 codes with
    fp32 per-row scales x_scale [M] and w_scale [N] (dtype e4m3); b, gamma,
    beta fp32."""
    rng = np.random.default_rng(seed)
    x = _normal(rng, (spec.M, spec.K), 1.0)
    W = _uniform(rng, (spec.N, spec.K), spec.w_bound)
    b = _uniform(rng, (spec.N,), spec.w_bound)
    out = {"b": b}
    if spec.dtype == "f32":
        out["x"], out["W"] = x, W
    elif spec.dtype == "e4m3":
        out["x"], out["x_scale"] = rows_to_e4m3(x)
        out["W"], out["w_scale"] = rows_to_e4m3(W)
    else:
        out["x"], out["W"] = to_bf16_bits(x), to_bf16_bits(W)
    if spec.reduction == "groupnorm":
        out["gamma"] = (np.float32(0.5) + rng.random(spec.N, dtype=np.float32)).astype(np.float32)
        out["beta"] = _normal(rng, (spec.N,), 0.1)
    return out


# --------------------------------------------------------------------------
# MoE expert FFN workloads (gpt-oss-20b-like geometry)

@dataclass(frozen=True)
class MoeSpec:
    name: str
    T: int
    H: int = 2880
    I: int = 2880
    E: int = 32
    k: int = 4
    w_dtype: str = "bf16"         # "bf16" or "e4m3"
    w_std: float = 0.02
    alpha: float = 1.702
    limit: float = 7.0
    x_std: float = 1.0

    def flops(self):
        return 2.0 * self.T * self.k * (self.H * 2 * self.I + self.I * self.H)

    def weight_bytes_per_expert(self):
        e = 1 if self.w_dtype == "e4m3" else 2
        b = (2 * self.I * self.H + self.H * self.I) * e
        if self.w_dtype == "e4m3":
            b += (2 * self.I + self.H) * 4
        return b

    def bytes(self, active_experts):
        """Algorithmic bytes: tokens and logits read once, the weights of the
        experts that receive at least one slot read once, output written once."""
        return (self.T * self.H * 2 + self.T * self.E * 4
                + active_experts * self.weight_bytes_per_expert()
                + self.T * self.H * 2)


MOE_SPECS = {
    "moe_prefill_bf16": MoeSpec("moe_prefill_bf16", 4096),
    "moe_decode_bf16": MoeSpec("moe_decode_bf16", 64),
    "moe_prefill_e4m3": MoeSpec("moe_prefill_e4m3", 4096, w_dtype="e4m3"),
    "moe_decode_e4m3": MoeSpec("moe_decode_e4m3", 64, w_dtype="e4m3"),
}


def make_moe_activations(spec, seed=0):
    """Router logits [T,E] fp32 ~ N(0,1) and tokens [T,H] bf16 bits ~ N(0, x_std)."""
    rng = np.random.default_rng(seed)
    logits = _normal(rng, (spec.T, spec.E), 1.0)
    x = to_bf16_bits(_normal(rng, (spec.T, spec.H), spec.x_std))
    return {"logits": logits, "x": x}


def make_moe_expert(spec, e, seed=0):
    """Weights of expert ``e``: W_gate_up [2I,H] (rows 0..I-1 gate, I..2I-1 up)
    and W_down [H,I], ~ N(0, w_std). bf16: uint16 bits. e4m3: uint8 codes plus
    fp32 per-row scales ``s_gate_up`` [2I] and ``s_down`` [H]."""
    rng = np.random.default_rng([seed, 1000 + e])
    wgu = _normal(rng, (2 * spec.I, spec.H), spec.w_std)
    wd = _normal(rng, (spec.H, spec.I), spec.w_std)
    if spec.w_dtype == "bf16":
        return {"w_gate_up": to_bf16_bits(wgu), "w_down": to_bf16_bits(wd)}
    qgu, sgu = rows_to_e4m3(wgu)
    qd, sd = rows_to_e4m3(wd)
    return {"w_gate_up": qgu, "s_gate_up": sgu, "w_down": qd, "s_down": sd}


def make_moe_weights(spec, seed=0):
    """All experts stacked: w_gate_up [E,2I,H], w_down [E,H,I] (+ scales)."""
    parts = [make_moe_expert(spec, e, seed) for e in range(spec.E)]
    return {key: np.stack([p[key] for p in parts]) for key in parts[0]}


# --------------------------------------------------------------------------
# MoE finalize (the standalone kernel of paper §IV-A, Table I): batch sizes
# 1 .. 128 of the gpt-oss-20b decode path, top-4, H = 2880.

FINALIZE_BATCHES = (1, 4, 8, 16, 32, 64, 128)
FINALIZE_H = 2880
FINALIZE_K = 4


def make_finalize_inputs(T, H=FINALIZE_H, k=FINALIZE_K, seed=0, exact=False):
    """Routing-weighted slot outputs y_slot [T·k, H] as bf16 bits.

    Default: N(0, 0.25), the scale of a weighted expert output. With
    ``exact``, every value is ±(1 + u/128)·2^e with u in 0..127 and e in
    −4..4 (each exactly a bf16 value), so that a sum of up to eight of them
    needs at most 19 significant bits and is exact in fp32."""
    rng = np.random.default_rng([seed, 2000 + T])
    if not exact:
        return to_bf16_bits(_normal(rng, (T * k, H), 0.25))
    u = rng.integers(0, 128, (T * k, H))
    e = rng.integers(-4, 5, (T * k, H))
    sign = np.where(rng.random((T * k, H)) < 0.5, -1.0, 1.0)
    return to_bf16_bits((sign * (1.0 + u / 128.0) * np.exp2(e)).astype(np.float32))


# --------------------------------------------------------------------------
# Fused residual add + RMSNorm (paper §IV-A, Table I): the same batch sizes,
# hidden size 2880.

NORM_H = 2880


def make_norm_inputs(T, H=NORM_H, seed=0):
    """x [T, H] ~ N(0, 1) (a layer output), residual [T, H] ~ N(0, 4) (the
    residual stream) and weight [H] ~ U(0.5, 1.5), as bf16 bits."""
    rng = np.random.default_rng([seed, 3000 + T])
    x = to_bf16_bits(_normal(rng, (T, H), 1.0))
    r = to_bf16_bits(_normal(rng, (T, H), 4.0))
    w = to_bf16_bits((rng.random(H, dtype=np.float32) + np.float32(0.5)).astype(np.float32))
    return x, r, w


# --------------------------------------------------------------------------
# QKV bias + rotary embedding + KV-cache update (paper §IV-A, Table I): the
# same batch sizes. The attention geometry is not in the paper; these are
# gpt-oss-20b's published attention sizes (64 query heads and 8 key/value
# heads of 64 values, rotary base 150000), with a paged cache of 64-token
# blocks.

@dataclass(frozen=True)
class RopeSpec:
    T: int
    n_q: int = 64
    n_kv: int = 8
    D: int = 64
    block_size: int = 64
    base: float = 150000.0
    interleaved: bool = False
    max_pos: int = 8192            # positions ~ U{0 .. max_pos − 1}

    @property
    def width(self):
        return (self.n_q + 2 * self.n_kv) * self.D

    @property
    def max_blocks(self):
        return (self.max_pos + self.block_size - 1) // self.block_size

    @property
    def num_blocks(self):
        return 2 * self.T + 16

    def bytes(self):
        """Algorithmic bytes of one step: qkv and bias read, q and the new K/V
        cache rows written (bf16), positions and the used block-table entries
        read."""
        return (self.T * self.width + self.width + self.T * self.n_q * self.D
                + 2 * self.T * self.n_kv * self.D) * 2 + self.T * 8


def make_rope_inputs(spec, seed=0):
    """qkv [T, width] ~ N(0, 1) and bias [width] ~ U(−0.1, 0.1) as bf16 bits,
    positions [T] int32 ~ U{0 .. max_pos − 1}, block_table [T, max_blocks]
    int32 and the cache's prior contents [num_blocks, 2, n_kv, block_size, D]
    ~ N(0, 1) bf16 bits. Each token's current block is a distinct block id;
    the other table entries hold ids of blocks no token of the step writes,
    so a wrong table lookup lands in a block that must stay unchanged."""
    rng = np.random.default_rng([seed, 4000 + spec.T])
    qkv = to_bf16_bits(_normal(rng, (spec.T, spec.width), 1.0))
    bias = to_bf16_bits(_uniform(rng, (spec.width,), 0.1))
    pos = rng.integers(0, spec.max_pos, spec.T).astype(np.int32)
    perm = rng.permutation(spec.num_blocks).astype(np.int32)
    current, others = perm[:spec.T], perm[spec.T:]
    table = others[rng.integers(0, others.size, (spec.T, spec.max_blocks))].astype(np.int32)
    table[np.arange(spec.T), pos // spec.block_size] = current
    cache = to_bf16_bits(_normal(rng, (spec.num_blocks, 2, spec.n_kv, spec.block_size, spec.D), 1.0))
    return {"qkv": qkv, "bias": bias, "positions": pos, "block_table": table, "cache": cache}
