"""Torch-facing wrappers over the C ABI.

PyTorch supplies device memory and the current stream; every step of the
computation runs in the library's HIP kernels. Inputs must already be CUDA
(HIP) tensors: there is no CPU path.
"""

import torch

from . import _lib

_TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}
_PLANS = {}


def _dt_name(t):
    if t.dtype == torch.float32:
        return "f32"
    if t.dtype == torch.bfloat16:
        return "bf16"
    if t.dtype in (torch.uint8, torch.float8_e4m3fn):
        return "e4m3"
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dev(t, name):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor (no CPU fallback)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def get_plan(M, N, K, in_dtype, out_dtype, has_bias, ops=(), reduction=None, gn_groups=0, gn_eps=1e-5,
             post_ops=()):
    """Cached fgemm plan for a problem description."""
    key = (M, N, K, in_dtype, out_dtype, bool(has_bias), tuple(tuple(o) for o in ops), reduction,
           gn_groups, float(gn_eps), tuple(tuple(o) for o in post_ops))
    p = _PLANS.get(key)
    if p is None:
        epi = _lib.make_epilogue(has_bias, ops, reduction, gn_groups, gn_eps, post_ops)
        p = _lib.fgemm_plan(M, N, K, in_dtype, out_dtype, epi)
        _PLANS[key] = p
    return p


def linear_epilogue(x, W, bias=None, ops=(), reduction=None, gn_groups=0, gn_eps=1e-5,
                    gamma=None, beta=None, out_dtype=None, out=None, workspace=None, stream=None,
                    post_ops=(), x_scale=None, w_scale=None):
    """y = tail(x·Wᵀ + b) in one fused launch (two for a row LogSumExp).

    x [M, K] and W [N, K] (f32 or bf16, same dtype; or e4m3 codes as uint8
    with per-row fp32 scales x_scale [M] and w_scale [N]), bias/gamma/beta
    fp32 [N]. ops: ((kind, a, b), ...) with kinds scale, add, relu,
    gelu_tanh, silu, clamp, mish, leaky_relu. reduction: None, "lse"
    (returns fp32 [M]) or "groupnorm". post_ops: ops of the same kinds
    applied to the reduction's result."""
    M, K = x.shape
    N, K2 = W.shape
    if K2 != K or x.dtype != W.dtype:
        raise ValueError("x must be [M,K] and W [N,K] of one dtype")
    in_dt = _dt_name(x)
    if in_dt == "e4m3" and (x_scale is None or w_scale is None):
        raise ValueError("e4m3 inputs need x_scale [M] and w_scale [N]")
    if out_dtype is None:
        out_dtype = "f32" if (in_dt == "f32" or reduction == "lse") else "bf16"
    plan = get_plan(M, N, K, in_dt, out_dtype, bias is not None, ops, reduction, gn_groups, gn_eps,
                    post_ops)
    if out is None:
        shape = (M,) if reduction == "lse" else (M, N)
        out = torch.empty(shape, dtype=_TORCH_DT[out_dtype], device=x.device)
    ws_bytes = plan.workspace_bytes()
    if ws_bytes and workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=x.device)
    _lib.fgemm_run_scaled(plan, _dev(x, "x"), _dev(W, "W"), _dev(x_scale, "x_scale"), _dev(w_scale, "w_scale"),
                          _dev(bias, "bias"), _dev(gamma, "gamma"), _dev(beta, "beta"), _dev(out, "out"),
                          _dev(workspace, "workspace"), ws_bytes, _stream(stream))
    return out


class MoeBuffers:
    """Outputs and workspace of one moe_grouped_ffn problem size."""

    def __init__(self, desc, device):
        T, k, E, H = desc.T, desc.top_k, desc.E, desc.H
        self.out = torch.empty((T, H), dtype=torch.bfloat16, device=device)
        self.topk_idx = torch.empty((T, k), dtype=torch.int32, device=device)
        self.topk_w = torch.empty((T, k), dtype=torch.float32, device=device)
        self.perm = torch.empty((T * k,), dtype=torch.int32, device=device)
        self.offsets = torch.empty((E + 1,), dtype=torch.int32, device=device)
        self.ws_bytes = _lib.moe_workspace_bytes(desc)
        self.workspace = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device=device)


def moe_ffn(tokens, router_logits, w_gateup, w_down, s_gateup=None, s_down=None, top_k=4,
            alpha=1.702, limit=7.0, interleaved=False, buffers=None, stream=None):
    """One MoE expert-FFN step. tokens [T,H] bf16, router_logits [T,E] fp32,
    w_gateup [E,2I,H] and w_down [E,H,I] bf16 (or uint8 e4m3 codes with fp32
    per-row scales s_gateup [E,2I], s_down [E,H]). Returns MoeBuffers."""
    T, H = tokens.shape
    E = router_logits.shape[1]
    I = w_down.shape[2]
    w_dt = "e4m3" if w_gateup.dtype in (torch.uint8, torch.float8_e4m3fn) else "bf16"
    desc = _lib.moe_desc(T, H, I, E, top_k, w_dt, alpha, limit, interleaved)
    if buffers is None:
        buffers = MoeBuffers(desc, tokens.device)
    b = buffers
    _lib.moe_grouped_ffn(desc, _dev(tokens, "tokens"), _dev(router_logits, "router_logits"),
                         _dev(w_gateup, "w_gateup"), _dev(w_down, "w_down"), _dev(s_gateup, "s_gateup"),
                         _dev(s_down, "s_down"), _dev(b.out, "out"), _dev(b.topk_idx, "topk_idx"),
                         _dev(b.topk_w, "topk_w"), _dev(b.perm, "perm"), _dev(b.offsets, "offsets"),
                         _dev(b.workspace, "workspace"), b.ws_bytes, _stream(stream))
    return b


def quantize_rows_e4m3(x, stream=None):
    """Per-row e4m3 quantisation of a bf16 [rows, cols] tensor: (codes uint8, scales fp32)."""
    rows, cols = x.shape
    q = torch.empty((rows, cols), dtype=torch.uint8, device=x.device)
    s = torch.empty((rows,), dtype=torch.float32, device=x.device)
    _lib.fg_quantize_rows_e4m3(_dev(x, "x"), rows, cols, _dev(q, "q"), _dev(s, "s"), _stream(stream))
    return q, s


def moe_finalize(y_slot, top_k, out=None, stream=None):
    """MoE finalize: y_slot [T·top_k, H] bf16 (routing-weighted slot outputs,
    row t·top_k + j) → out [T, H] bf16 = Σ_j y_slot[t·top_k + j], fp32 sum."""
    S, H = y_slot.shape
    if y_slot.dtype != torch.bfloat16:
        raise TypeError("y_slot must be bf16")
    if S % top_k != 0:
        raise ValueError("y_slot rows must be a multiple of top_k")
    T = S // top_k
    if out is None:
        out = torch.empty((T, H), dtype=torch.bfloat16, device=y_slot.device)
    _lib.moe_finalize(_dev(y_slot, "y_slot"), _dev(out, "out"), T, H, top_k, _stream(stream))
    return out


def add_rmsnorm(x, residual, weight, eps=1e-5, out=None, stream=None):
    """Fused residual add + RMSNorm on bf16 [T, H] rows: residual is updated
    in place to x + residual and out = RMSNorm(x + residual)·weight."""
    T, H = x.shape
    for name, t in (("x", x), ("residual", residual), ("weight", weight)):
        if t.dtype != torch.bfloat16:
            raise TypeError(f"{name} must be bf16")
    if out is None:
        out = torch.empty((T, H), dtype=torch.bfloat16, device=x.device)
    _lib.add_rmsnorm(_dev(x, "x"), _dev(residual, "residual"), _dev(weight, "weight"), _dev(out, "out"),
                     T, H, eps, _stream(stream))
    return out


def bias_rope_kv_update(qkv, bias, positions, block_table, kv_cache, n_q, n_kv, head_dim, rope_base,
                        interleaved=False, q_out=None, stream=None):
    """QKV bias + rotary embedding + paged KV-cache write of one decode step.

    qkv [T, (n_q + 2·n_kv)·head_dim] bf16, bias [(n_q + 2·n_kv)·head_dim] bf16
    or None, positions [T] int32, block_table [T, max_blocks] int32, kv_cache
    [num_blocks, 2, n_kv, block_size, head_dim] bf16 (written in place at each
    token's row). Returns q_out [T, n_q, head_dim] bf16."""
    T = qkv.shape[0]
    for name, t in (("qkv", qkv), ("kv_cache", kv_cache)) + ((("bias", bias),) if bias is not None else ()):
        if t.dtype != torch.bfloat16:
            raise TypeError(f"{name} must be bf16")
    for name, t in (("positions", positions), ("block_table", block_table)):
        if t.dtype != torch.int32:
            raise TypeError(f"{name} must be int32")
    if kv_cache.dim() != 5 or kv_cache.shape[1] != 2 or kv_cache.shape[2] != n_kv or kv_cache.shape[4] != head_dim:
        raise ValueError("kv_cache must be [num_blocks, 2, n_kv, block_size, head_dim]")
    if qkv.shape[1] != (n_q + 2 * n_kv) * head_dim or positions.shape != (T,) or block_table.shape[0] != T:
        raise ValueError("qkv, positions and block_table shapes do not match")
    if q_out is None:
        q_out = torch.empty((T, n_q, head_dim), dtype=torch.bfloat16, device=qkv.device)
    d = _lib.rope_desc(T, n_q, n_kv, head_dim, kv_cache.shape[3], block_table.shape[1], kv_cache.shape[0],
                       rope_base, interleaved)
    _lib.bias_rope_kv_update(d, _dev(qkv, "qkv"), _dev(bias, "bias"), _dev(positions, "positions"),
                             _dev(block_table, "block_table"), _dev(q_out, "q_out"), _dev(kv_cache, "kv_cache"),
                             _stream(stream))
    return q_out
