"""fp64 oracle for the fused GEMM + tail: y = tail(x·Wᵀ + b).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Paper §IV-B describes what the generated GEMM + tail-ops kernels do: the
post-GEMM sequence (pointwise activations, scaling, normalisation,
LogSumExp; Table III names Swish = SiLU, Scale, LSE, GroupNorm) is applied to
the matmul result, which is read once and written once, with fp32
accumulation and post-processing. Fusion only reschedules these operations,
so the oracle is their plain definition, composed in the order given:

  1. z = x·Wᵀ (+ b)                    — one fp64 matmul (library dgemm)
  2. each elementwise op, in order     — SCALE, ADD, RELU, GELU_TANH, SILU,
                                         CLAMP, MISH, LEAKY_RELU
  3. an optional terminal reduction    — row LogSumExp (one value per row) or
                                         GroupNorm over contiguous channel groups
  4. elementwise ops after the reduction, in order (per element after
     GroupNorm, per row value after LogSumExp): Table III chains such as
     GroupNorm → LeakyReLU → Sum, GroupNorm → Swish → Mul → Swish, and
     LogSumExp → Mish

Definitions used (standard forms; the paper names the ops, not formulas):
  GELU_TANH(u) = ½·u·(1 + tanh(√(2/π)·(u + 0.044715·u³)))   (Hendrycks & Gimpel, tanh form)
  SILU(u)      = u / (1 + e^(−u))                              (Swish with β = 1)
  CLAMP(u)     = min(max(u, lo), hi)
  MISH(u)      = u·tanh(ln(1 + e^u))                            (Misra 2019)
  LEAKY_RELU(u)= u for u ≥ 0, a·u otherwise                     (slope a)
  LSE(row)     = M + ln Σ_n e^(z_n − M),  M = max_n z_n
  GroupNorm    : groups are contiguous channel blocks of N/G channels; per
                 row and group, μ = mean, σ² = mean((z − μ)²) (biased);
                 y = (z − μ)/√(σ² + eps)·γ[n] + β[n]
Every value is fp64 and nothing is rounded: the comparison upcasts the GPU
result instead.
"""

import math

import numpy as np

OPS = ("scale", "add", "relu", "gelu_tanh", "silu", "clamp", "mish", "leaky_relu")

_SQRT_2_OVER_PI = math.sqrt(2.0 / math.pi)


def _gelu_tanh(u):
    return 0.5 * u * (1.0 + np.tanh(_SQRT_2_OVER_PI * (u + 0.044715 * u ** 3)))


def _silu(u):
    # u·σ(u) written so that neither branch overflows: σ(u) = 1/(1+e^-u) for
    # u ≥ 0 and e^u/(1+e^u) for u < 0 (the same function)
    out = np.empty_like(u)
    pos = u >= 0
    out[pos] = u[pos] / (1.0 + np.exp(-u[pos]))
    eu = np.exp(u[~pos])
    out[~pos] = u[~pos] * eu / (1.0 + eu)
    return out


def _mish(u):
    # softplus = ln(1 + e^u) = logaddexp(0, u), which overflows for no u
    return u * np.tanh(np.logaddexp(0.0, u))


def apply_op(z, op):
    """Apply one elementwise tail op, given as (kind, a, b), in fp64."""
    kind, a, b = (tuple(op) + (0.0, 0.0))[:3]
    if kind == "scale":
        return z * a
    if kind == "add":
        return z + a
    if kind == "relu":
        return np.maximum(z, 0.0)
    if kind == "gelu_tanh":
        return _gelu_tanh(z)
    if kind == "silu":
        return _silu(z)
    if kind == "clamp":
        return np.minimum(np.maximum(z, a), b)
    if kind == "mish":
        return _mish(z)
    if kind == "leaky_relu":
        return np.where(z >= 0.0, z, a * z)
    raise ValueError(f"unknown op {kind!r}")


def row_logsumexp(z):
    """LSE over the last axis: M + ln Σ exp(z − M), with M the row max."""
    m = np.max(z, axis=-1, keepdims=True)
    return (m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True)))[..., 0]


def group_norm(z, groups, eps, gamma, beta):
    """GroupNorm of [M, N] over ``groups`` contiguous channel blocks."""
    M, N = z.shape
    if N % groups:
        raise ValueError("N must be a multiple of the group count")
    zg = z.reshape(M, groups, N // groups)
    mu = zg.mean(axis=-1, keepdims=True)
    var = ((zg - mu) ** 2).mean(axis=-1, keepdims=True)
    y = ((zg - mu) / np.sqrt(var + eps)).reshape(M, N)
    return y * gamma[None, :] + beta[None, :]


def ref_fgemm(x, W, b=None, ops=(), reduction=None, gn_groups=None, gn_eps=1e-5,
              gamma=None, beta=None, post_ops=()):
    """Plain definition of the fused linear + tail, in fp64.

    x: [M, K], W: [N, K] (nn.Linear layout), b: [N] or None — all fp64 arrays
    holding the exact values the kernel reads (decoded bf16 / fp32).
    ops: sequence of (kind, a, b) applied in order after the bias.
    reduction: None, "lse" (returns [M]) or "groupnorm" (returns [M, N]).
    post_ops: (kind, a, b) ops applied in order to the reduction's result.
    """
    x = np.asarray(x, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    if x.ndim != 2 or W.ndim != 2 or x.shape[1] != W.shape[1]:
        raise ValueError("x must be [M,K] and W [N,K]")
    z = x @ W.T
    if b is not None:
        z = z + np.asarray(b, dtype=np.float64)[None, :]
    for op in ops:
        z = apply_op(z, op)
    if reduction is None:
        if post_ops:
            raise ValueError("post_ops need a reduction")
        return z
    if reduction == "lse":
        y = row_logsumexp(z)
    elif reduction == "groupnorm":
        y = group_norm(z, gn_groups, gn_eps,
                       np.asarray(gamma, dtype=np.float64),
                       np.asarray(beta, dtype=np.float64))
    else:
        raise ValueError(f"unknown reduction {reduction!r}")
    for op in post_ops:
        y = apply_op(y, op)
    return y
