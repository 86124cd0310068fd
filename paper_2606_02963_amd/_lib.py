"""ctypes binding of ``include/fgemm.h`` (argument marshalling only).

The names mirror the C entry points. Pointers are passed as Python ints
(device addresses, e.g. ``tensor.data_ptr()``); the stream is a hipStream_t
as an int (``torch.cuda.current_stream().cuda_stream``) or None. A status
other than FG_OK raises :class:`FgError` carrying ``fg_status_str`` and
``fg_last_error``. Loading fails loudly if the library has not been built:
there is no fallback path.
"""

import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libfgemm.so")

FG_OK, FG_ERR_INVALID_ARG, FG_ERR_UNSUPPORTED, FG_ERR_ALIGNMENT, FG_ERR_WORKSPACE, FG_ERR_HIP = range(6)
FG_F32, FG_BF16, FG_E4M3 = 0, 1, 2
DTYPES = {"f32": FG_F32, "bf16": FG_BF16, "e4m3": FG_E4M3}
OP_KINDS = {"scale": 0, "add": 1, "relu": 2, "gelu_tanh": 3, "silu": 4, "clamp": 5, "mish": 6,
            "leaky_relu": 7}
REDUCTIONS = {None: 0, "lse": 1, "groupnorm": 2}
FG_MAX_OPS = 8


class FgOp(C.Structure):
    _fields_ = [("kind", C.c_int32), ("a", C.c_float), ("b", C.c_float)]


class FgEpilogue(C.Structure):
    _fields_ = [("has_bias", C.c_int32), ("n_ops", C.c_int32), ("ops", FgOp * FG_MAX_OPS),
                ("reduction", C.c_int32), ("gn_groups", C.c_int32), ("gn_eps", C.c_float),
                ("n_post_ops", C.c_int32), ("post_ops", FgOp * FG_MAX_OPS)]


class MoeDesc(C.Structure):
    _fields_ = [("T", C.c_int64), ("H", C.c_int64), ("I", C.c_int64), ("E", C.c_int32),
                ("top_k", C.c_int32), ("w_dtype", C.c_int32), ("swiglu_alpha", C.c_float),
                ("swiglu_limit", C.c_float), ("gateup_interleaved", C.c_int32)]


class RopeDesc(C.Structure):
    _fields_ = [("T", C.c_int64), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("block_size", C.c_int32), ("max_blocks", C.c_int32),
                ("num_blocks", C.c_int64), ("rope_base", C.c_float), ("interleaved", C.c_int32)]


class FgError(RuntimeError):
    def __init__(self, status, func, detail):
        self.status = status
        super().__init__(f"{func}: {status_str(status)}" + (f" — {detail}" if detail else ""))


_lib = None


def lib():
    """The loaded library (raises if it was never built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"HIP library {LIB_PATH} is not built; run `python -m paper_2606_02963_amd.build` "
                "(or __graft_entry__.build()) first")
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
        L.fgemm_plan.argtypes = [C.POINTER(vp), i64, i64, i64, i32, i32, C.POINTER(FgEpilogue)]
        L.fgemm_plan.restype = i32
        L.fgemm_workspace_bytes.argtypes = [vp]
        L.fgemm_workspace_bytes.restype = sz
        L.fgemm_run.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.fgemm_run.restype = i32
        L.fgemm_run_scaled.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.fgemm_run_scaled.restype = i32
        L.fgemm_destroy.argtypes = [vp]
        L.fgemm_destroy.restype = None
        L.fgemm_plan_info.argtypes = [vp, C.POINTER(i32), C.POINTER(i32), C.POINTER(i64), C.POINTER(i32),
                                      C.POINTER(i32)]
        L.fgemm_plan_info.restype = i32
        L.moe_workspace_bytes.argtypes = [C.POINTER(MoeDesc)]
        L.moe_workspace_bytes.restype = sz
        L.moe_grouped_ffn.argtypes = [C.POINTER(MoeDesc)] + [vp] * 12 + [sz, vp]
        L.moe_grouped_ffn.restype = i32
        L.moe_grouped_ffn_noalloc.argtypes = [C.POINTER(MoeDesc)] + [vp] * 12
        L.moe_grouped_ffn_noalloc.restype = i32
        L.moe_noalloc_scratch_bytes.argtypes = []
        L.moe_noalloc_scratch_bytes.restype = sz
        L.moe_finalize.argtypes = [vp, vp, i64, i64, i32, vp]
        L.moe_finalize.restype = i32
        L.add_rmsnorm.argtypes = [vp, vp, vp, vp, i64, i64, C.c_float, vp]
        L.add_rmsnorm.restype = i32
        L.bias_rope_kv_update.argtypes = [C.POINTER(RopeDesc), vp, vp, vp, vp, vp, vp, vp]
        L.bias_rope_kv_update.restype = i32
        L.fg_quantize_rows_e4m3.argtypes = [vp, i64, i64, vp, vp, vp]
        L.fg_quantize_rows_e4m3.restype = i32
        L.fg_trace_begin.argtypes = [i32]
        L.fg_trace_begin.restype = i32
        L.fg_trace_end.argtypes = []
        L.fg_trace_end.restype = i32
        L.fg_trace_read.argtypes = [i32, C.POINTER(C.c_float), C.POINTER(C.c_char_p)]
        L.fg_trace_read.restype = i32
        L.fg_status_str.argtypes = [i32]
        L.fg_status_str.restype = C.c_char_p
        L.fg_last_error.argtypes = []
        L.fg_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def status_str(st):
    return lib().fg_status_str(st).decode()


def last_error():
    return lib().fg_last_error().decode()


def _check(st, func):
    if st != FG_OK:
        raise FgError(st, func, last_error())


def _fill_ops(dst, ops):
    for i, op in enumerate(ops):
        kind, a, b = (tuple(op) + (0.0, 0.0))[:3]
        dst[i].kind = OP_KINDS[kind] if isinstance(kind, str) else int(kind)
        dst[i].a = a
        dst[i].b = b


def make_epilogue(has_bias=False, ops=(), reduction=None, gn_groups=0, gn_eps=1e-5, post_ops=()):
    """Build an FgEpilogue from ((kind, a, b), ...) tuples as used by the oracle.
    post_ops are applied to the reduction's result."""
    if len(ops) > FG_MAX_OPS or len(post_ops) > FG_MAX_OPS:
        raise ValueError(f"at most {FG_MAX_OPS} ops per chain")
    e = FgEpilogue()
    e.has_bias = 1 if has_bias else 0
    e.n_ops = len(ops)
    _fill_ops(e.ops, ops)
    e.reduction = REDUCTIONS[reduction] if not isinstance(reduction, int) else reduction
    e.gn_groups = gn_groups
    e.gn_eps = gn_eps
    e.n_post_ops = len(post_ops)
    _fill_ops(e.post_ops, post_ops)
    return e


class Plan:
    """Owns an fg_plan handle (released on close/garbage collection)."""

    def __init__(self, handle):
        self._h = handle

    @property
    def handle(self):
        if not self._h:
            raise ValueError("plan already destroyed")
        return self._h

    def workspace_bytes(self):
        return fgemm_workspace_bytes(self)

    def info(self):
        tm, tn, wg, nl, ks = C.c_int32(), C.c_int32(), C.c_int64(), C.c_int32(), C.c_int32()
        _check(lib().fgemm_plan_info(self.handle, C.byref(tm), C.byref(tn), C.byref(wg), C.byref(nl),
                                     C.byref(ks)), "fgemm_plan_info")
        return {"tile_m": tm.value, "tile_n": tn.value, "workgroups": wg.value, "launches": nl.value,
                "k_slices": ks.value}

    def close(self):
        if self._h:
            lib().fgemm_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def fgemm_plan(M, N, K, in_dtype, out_dtype, epi):
    h = C.c_void_p()
    st = lib().fgemm_plan(C.byref(h), int(M), int(N), int(K), DTYPES.get(in_dtype, in_dtype),
                          DTYPES.get(out_dtype, out_dtype), C.byref(epi) if epi is not None else None)
    _check(st, "fgemm_plan")
    return Plan(h.value)


def fgemm_workspace_bytes(plan):
    return lib().fgemm_workspace_bytes(plan.handle if plan is not None else None)


def fgemm_run(plan, A, W, bias, gamma, beta, out, workspace, ws_bytes, stream=None):
    st = lib().fgemm_run(plan.handle, A, W, bias, gamma, beta, out, workspace, ws_bytes, stream)
    _check(st, "fgemm_run")


def fgemm_run_scaled(plan, A, W, a_scale, w_scale, bias, gamma, beta, out, workspace, ws_bytes, stream=None):
    """fgemm_run with per-row scales of x and W (required for e4m3 plans)."""
    st = lib().fgemm_run_scaled(plan.handle, A, W, a_scale, w_scale, bias, gamma, beta, out, workspace,
                                ws_bytes, stream)
    _check(st, "fgemm_run_scaled")


def moe_desc(T, H, I, E, top_k, w_dtype="bf16", alpha=1.702, limit=7.0, interleaved=False):
    d = MoeDesc()
    d.T, d.H, d.I, d.E, d.top_k = int(T), int(H), int(I), int(E), int(top_k)
    d.w_dtype = DTYPES.get(w_dtype, w_dtype)
    d.swiglu_alpha, d.swiglu_limit = alpha, limit
    d.gateup_interleaved = 1 if interleaved else 0
    return d


def moe_workspace_bytes(desc):
    return lib().moe_workspace_bytes(C.byref(desc))


def moe_grouped_ffn(desc, tokens, router_logits, w_gateup, w_down, s_gateup, s_down, out,
                    topk_idx, topk_w, perm, expert_offsets, workspace, ws_bytes, stream=None):
    st = lib().moe_grouped_ffn(C.byref(desc), tokens, router_logits, w_gateup, w_down, s_gateup,
                               s_down, out, topk_idx, topk_w, perm, expert_offsets, workspace,
                               ws_bytes, stream)
    _check(st, "moe_grouped_ffn")


def moe_grouped_ffn_noalloc(desc, tokens, router_logits, w_gateup, w_down, s_gateup, s_down, out,
                            topk_idx, topk_w, perm, expert_offsets, stream=None):
    """moe_grouped_ffn with the library's static per-GPU scratch as workspace."""
    st = lib().moe_grouped_ffn_noalloc(C.byref(desc), tokens, router_logits, w_gateup, w_down, s_gateup,
                                       s_down, out, topk_idx, topk_w, perm, expert_offsets, stream)
    _check(st, "moe_grouped_ffn_noalloc")


def moe_noalloc_scratch_bytes():
    return lib().moe_noalloc_scratch_bytes()


def fg_quantize_rows_e4m3(x, rows, cols, q, s, stream=None):
    _check(lib().fg_quantize_rows_e4m3(x, int(rows), int(cols), q, s, stream), "fg_quantize_rows_e4m3")


def fg_trace_begin(capacity):
    _check(lib().fg_trace_begin(int(capacity)), "fg_trace_begin")


def fg_trace_end():
    return lib().fg_trace_end()


def fg_trace_read(i):
    """(milliseconds between the two events of traced launch i, kernel name)."""
    ms, name = C.c_float(), C.c_char_p()
    _check(lib().fg_trace_read(int(i), C.byref(ms), C.byref(name)), "fg_trace_read")
    return ms.value, (name.value or b"").decode(errors="replace")


def moe_finalize(y_slot, out, T, H, top_k, stream=None):
    """out[t] = Σ_j y_slot[t·top_k + j] (bf16, fp32 sum in ascending j)."""
    _check(lib().moe_finalize(y_slot, out, T, H, top_k, stream), "moe_finalize")


def add_rmsnorm(x, residual, weight, out, T, H, eps, stream=None):
    """residual <- bf16(x + residual); out = bf16(RMSNorm(x + residual) * weight)."""
    _check(lib().add_rmsnorm(x, residual, weight, out, T, H, eps, stream), "add_rmsnorm")


def rope_desc(T, n_q, n_kv, D, block_size, max_blocks, num_blocks, base, interleaved=False):
    d = RopeDesc()
    d.T, d.n_q_heads, d.n_kv_heads, d.head_dim = int(T), int(n_q), int(n_kv), int(D)
    d.block_size, d.max_blocks, d.num_blocks = int(block_size), int(max_blocks), int(num_blocks)
    d.rope_base = base
    d.interleaved = 1 if interleaved else 0
    return d


def bias_rope_kv_update(desc, qkv, bias, positions, block_table, q_out, kv_cache, stream=None):
    """q_out = RoPE(q + b); kv_cache rows at each token's position = (RoPE(k + b), v + b)."""
    _check(lib().bias_rope_kv_update(C.byref(desc) if desc is not None else None, qkv, bias, positions,
                                     block_table, q_out, kv_cache, stream), "bias_rope_kv_update")
