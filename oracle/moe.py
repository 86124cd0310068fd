"""fp64 oracle for the MoE expert FFN step (route → permute → grouped FFN →
finalize).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Paper §IV-A optimises the decode-path kernels of the gpt-oss-20b MoE model on
B200, among them "MoE finalize" (Table I): the routing-weighted sum of each
token's top-k expert outputs, returned to token order. §V names the joint
optimisation of the whole MoE-MLP block as the next step. The expert MLP of
that model is a clamped SwiGLU: the gate is clamped above at ``limit``, the up
projection to [−limit, limit], glu = gate·σ(α·gate) and the output is
(up + 1)·glu, with α = 1.702 and limit = 7.

The oracle takes the block's steps in order, each as its plain definition:

  route     top-k of the E router logits per token, ordered by value
            descending with ties to the lower expert index; routing weights
            are the softmax over the k selected logits
  permute   slot p = t·k + j carries expert idx[t, j]; counts[e] is the
            histogram, offsets the exclusive prefix sum (length E + 1) and
            perm lists the slot ids sorted by (expert, slot id) — a stable
            sort, which makes it unique
  expert e  X = x[perm[r] // k] for the rows r of expert e;
            G = X·W_gu[e]ᵀ, gate | up = the two halves of G (or its even /
            odd columns when interleaved); h = clamped SwiGLU(gate, up);
            h is stored in the method's declared intermediate format,
            modelled here: bf16 RNE; in the W8A8 variant the bf16 h is
            then quantised per row to e4m3 with an fp32 scale;
            y_slot[rows] = h·W_d[e]ᵀ
  finalize  out[t] = Σ_j w[t, j]·y_slot[t·k + j], j ascending: the
            routing-weighted sum, kept exact (fp64) until the single output
            rounding, which the comparison applies to nothing (the oracle
            output is returned unrounded)

fp8 (W8A8) variant: weights are stored as e4m3 codes with one fp32 scale per
output row (decoded before they reach this oracle); activations (x per
token, and the bf16-stored h per slot row) are quantised online with
s = amax/448 and code = RNE_sat(v / s). Those quantisation decisions are
taken in fp32 on the stored (bf16) values, the precision the kernel takes
them in, so both sides pick the same code for the same stored value.

Several results are correct where h lies within the arithmetic noise of a
storage rounding boundary (the kernel evaluates h in another rounding order,
and in the W8A8 variant on an fp8 dot product that is not summed as IEEE
fp32). ``ref_moe(..., with_bound=True)`` returns, per output element, the
largest change that taking any such decision the other way can cause
(``storage_bound``, with the fp8 contraction noise of ``f8_contraction_noise``
carried through ``swiglu_noise``), and the same for h within fp32 evaluation
noise only (``out_bound_narrow``); the outputs themselves do not depend on
either.
"""

import numpy as np

from .codecs import (E4M3_MAX, bf16_decode, bf16_encode_rne, e4m3_decode,
                     e4m3_encode_rne_sat, f32_round)


def ref_route(logits, k):
    """Top-k experts per token (descending, ties → lower index) and the
    softmax over the selected logits (fp64)."""
    logits = np.asarray(logits, dtype=np.float64)
    T, E = logits.shape
    idx = np.empty((T, k), dtype=np.int32)
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-logits[t, e], e))
        idx[t] = order[:k]
    sel = np.take_along_axis(logits, idx.astype(np.int64), axis=1)
    ex = np.exp(sel - sel.max(axis=1, keepdims=True))
    w = ex / ex.sum(axis=1, keepdims=True)
    return idx, w


def ref_permute(idx, E):
    """Expert histogram, exclusive offsets and the stable slot permutation."""
    idx = np.asarray(idx)
    T, k = idx.shape
    flat = idx.reshape(-1)
    counts = np.array([int(np.sum(flat == e)) for e in range(E)], dtype=np.int32)
    offsets = np.zeros(E + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    perm = np.array(sorted(range(T * k), key=lambda p: (int(flat[p]), p)), dtype=np.int32)
    return counts, offsets, perm


def ref_swiglu_clamped(gate, up, alpha=1.702, limit=7.0):
    """Clamped SwiGLU: (clip(up, −L, L) + 1) · g·σ(α·g), g = min(gate, L)."""
    g = np.minimum(gate, limit)
    u = np.clip(up, -limit, limit)
    # for very negative α·g the exponential overflows to +inf and σ is 0,
    # its exact limit; the overflow is expected, not an error
    with np.errstate(over="ignore"):
        sig = 1.0 / (1.0 + np.exp(-alpha * g))
    return (u + 1.0) * (g * sig)


def ref_quant_rows_e4m3(v):
    """Per-row e4m3 quantisation, decisions in fp32.

    s = fp32(amax_row)/448 rounded to fp32 (a zero row gets s = 1);
    code = RNE_sat_e4m3(fp32(fp32(v)/s)). Returns (codes uint8, s fp64)."""
    v32 = f32_round(v)
    amax = np.max(np.abs(v32), axis=-1, keepdims=True)
    s = f32_round(amax / E4M3_MAX)
    s = np.where(amax == 0.0, 1.0, s)
    q = e4m3_encode_rne_sat(f32_round(v32 / s))
    return q, s[..., 0]


def _dequant_rows(codes, s):
    return e4m3_decode(codes) * np.asarray(s, dtype=np.float64)[..., None]


def _dequant_with_scale(b, s):
    """e4m3 code of fp32(b/s) (RNE, saturated) decoded and rescaled, per row scale s."""
    s = np.asarray(s, dtype=np.float64)[..., None]
    return e4m3_decode(e4m3_encode_rne_sat(f32_round(f32_round(b) / s))) * s


def _bf16(v):
    return bf16_decode(bf16_encode_rne(v))


def store_h(h, storage):
    """The declared storage of the intermediate h (the down GEMM's operand):
    "bf16" rounds to bf16 (RNE); "e4m3" rounds to bf16 and then quantises
    each row to e4m3 codes with an fp32 scale (decoded back to values);
    "none" keeps h exact."""
    if storage == "none":
        return h
    hb = bf16_decode(bf16_encode_rne(h))
    if storage == "bf16":
        return hb
    if storage == "e4m3":
        q, s = ref_quant_rows_e4m3(hb)
        return _dequant_rows(q, s)
    raise ValueError(f"unknown storage {storage!r}")


# Relative and row-absolute size of the neighbourhood of a storage rounding
# boundary inside which a kernel that evaluates h in fp32 (a different
# rounding order than this fp64 oracle) may legitimately take the other
# rounding decision. Both are far above fp32 evaluation error of h and far
# below any tolerance.
FRAGILE_REL = 2.0 ** -16
FRAGILE_ABS = 2.0 ** -20

# Accumulation noise of one 128-wide e4m3 × e4m3 dot product on the matrix
# cores, as a fraction of its Σ|x_i·w_i|. gfx950's f8f6f4 MFMA does not sum
# the dot product as IEEE fp32: products far below the largest one lose
# low-order bits. Measured: at most 2.4e-5 of Σ|products| on Gaussian data
# (150 000 dot products), up to 2.6e-4 when one product dominates the other
# 127. A contraction over K runs K/128 such dot products (128 consecutive
# K-values each) and adds their results in fp32; with sign-mixed data their
# errors are independent, so the noise of the whole contraction is taken as
# F8_DOT_NOISE · √(Σ_c S_c²), S_c = Σ|x_i·w_i| over dot product c (see
# f8_contraction_noise). The value is 2.5× the Gaussian-data maximum (the
# synthetic workloads are Gaussian), not a worst-case bound.
F8_DOT_NOISE = 2.0 ** -14
F8_DOT_K = 128


def f8_contraction_noise(X, W):
    """Noise bound of the e4m3 contraction X·Wᵀ per output element (X [n, K],
    W [m, K], exact values): F8_DOT_NOISE · √(Σ_c S_c²) over the K/128 dot
    products of 128 consecutive K-values (a partial last one included)."""
    aX = np.abs(np.asarray(X, dtype=np.float64))
    aW = np.abs(np.asarray(W, dtype=np.float64))
    ss = np.zeros((aX.shape[0], aW.shape[0]))
    for c0 in range(0, aX.shape[1], F8_DOT_K):
        s_c = aX[:, c0:c0 + F8_DOT_K] @ aW[:, c0:c0 + F8_DOT_K].T
        ss += s_c * s_c
    return F8_DOT_NOISE * np.sqrt(ss)


def storage_deviation(h, storage, noise=None):
    """Largest change of the stored value of each element of h (per row for
    the per-row-scaled e4m3 storage) over the rounding decisions that are
    within FRAGILE_REL·|h| + FRAGILE_ABS·max|h_row| (+ noise, a per-element
    absolute bound on how far a kernel's h may lie from the exact one) of a
    boundary. Zero for every element whose stored value is robust. Returns
    (stored, deviation), stored being store_h(h, storage)."""
    h = np.asarray(h, dtype=np.float64)
    stored = store_h(h, storage)
    if storage == "none":
        return stored, np.zeros_like(h)
    pert = FRAGILE_REL * np.abs(h) + FRAGILE_ABS * np.max(np.abs(h), axis=-1, keepdims=True)
    if noise is not None:
        pert = pert + np.asarray(noise, dtype=np.float64)
    b_ref, b_lo, b_hi = _bf16(h), _bf16(h - pert), _bf16(h + pert)
    if storage == "bf16":
        return stored, np.maximum(np.abs(b_lo - b_ref), np.abs(b_hi - b_ref))
    # the e4m3 decision of a bf16 value under a given scale is taken in fp32
    # on both sides, so only the bf16 decisions (of each element, and of the
    # row maximum, which sets the scale) can go either way
    bs = (b_ref, b_lo, b_hi)
    scales = [ref_quant_rows_e4m3(b)[1] for b in bs]
    dev = np.zeros_like(h)
    # rows whose scale is fragile: every combination of element and scale decisions
    rows = np.flatnonzero((scales[1] != scales[0]) | (scales[2] != scales[0]))
    for b in bs:
        for sc in scales:
            dev[rows] = np.maximum(dev[rows], np.abs(_dequant_with_scale(b[rows], sc[rows]) - stored[rows]))
    # the other rows keep their scale: only elements whose bf16 value may differ can move
    keep = np.ones(h.shape[0], dtype=bool)
    keep[rows] = False
    for b in (b_lo, b_hi):
        r, c = np.nonzero((b != b_ref) & keep[:, None])
        sc = scales[0][r]
        moved = e4m3_decode(e4m3_encode_rne_sat(f32_round(f32_round(b[r, c]) / sc))) * sc
        dev[r, c] = np.maximum(dev[r, c], np.abs(moved - stored[r, c]))
    return stored, dev


def storage_bound(h, storage, W_d, noise=None):
    """(stored h)·W_dᵀ and, per element of it, the largest change that taking
    any storage decisions of h within the neighbourhood of a boundary the
    other way can cause (the neighbourhood as in storage_deviation; each
    element may take the bf16 value of h − pert, h or h + pert). For e4m3
    storage the row scale follows the row maximum of whichever values are
    taken, so its candidates are the scales of every candidate magnitude at
    or above the smallest maximum any choice gives. Under a candidate scale
    s′ the rescaling of the whole row, (h(s′) − stored)·W_dᵀ, is taken with
    its signs and only the element decisions are bounded in absolute value;
    the largest over the candidates is kept. bf16 storage: deviation·|W_d|ᵀ."""
    h = np.asarray(h, dtype=np.float64)
    W_d = np.asarray(W_d, dtype=np.float64)
    stored, dev = storage_deviation(h, storage, noise)
    out = stored @ W_d.T
    if storage != "e4m3":
        return out, dev @ np.abs(W_d).T
    pert = FRAGILE_REL * np.abs(h) + FRAGILE_ABS * np.max(np.abs(h), axis=-1, keepdims=True)
    if noise is not None:
        pert = pert + np.asarray(noise, dtype=np.float64)
    bs = (_bf16(h), _bf16(h - pert), _bf16(h + pert))
    mag = np.stack([np.abs(b) for b in bs])                       # 3 × rows × I
    floor = mag.min(axis=0).max(axis=-1, keepdims=True)            # smallest maximum any choice gives
    # an element that may hold the maximum has at most the three values
    # above: its neighbourhood spans at most two bf16 steps
    top = mag.max(axis=0) >= floor
    steps = np.abs(bf16_encode_rne(bs[2]).astype(np.int64) - bf16_encode_rne(bs[1]).astype(np.int64))
    if np.any(top & ((steps > 2) | (np.sign(bs[1]) * np.sign(bs[2]) < 0))):
        raise ValueError("storage_bound: a neighbourhood of a row maximum spans more than two bf16 steps")
    cand = np.where(mag >= floor, mag, -1.0).transpose(1, 0, 2).reshape(h.shape[0], -1)
    cand = -np.sort(-cand, axis=-1)                                 # candidates first, descending
    n_c = np.array([np.unique(c[c >= 0]).size for c in cand])
    width = int(n_c.max())
    amax = np.empty((h.shape[0], width))
    for r in range(h.shape[0]):
        u = np.unique(cand[r][cand[r] >= 0])
        amax[r] = np.concatenate([u, np.full(width - u.size, u[0])])
    scales = np.where(amax == 0.0, 1.0, f32_round(amax / E4M3_MAX))
    # rows with one candidate scale: element decisions only (scale of the stored row)
    s_ref = ref_quant_rows_e4m3(bs[0])[1]
    flips = np.zeros_like(h)
    for b in bs[1:]:
        flips = np.maximum(flips, np.abs(_dequant_with_scale(b, s_ref) - stored))
    bound = flips @ np.abs(W_d).T
    rows = np.flatnonzero(np.any(scales != scales[:, :1], axis=-1) | (scales[:, 0] != s_ref))
    if rows.size:
        best = np.zeros((rows.size, W_d.shape[0]))
        for c in range(width):
            sc = scales[rows, c]
            base = _dequant_with_scale(bs[0][rows], sc)
            fl = np.zeros_like(base)
            for b in bs[1:]:
                fl = np.maximum(fl, np.abs(_dequant_with_scale(b[rows], sc) - base))
            best = np.maximum(best, np.abs((base - stored[rows]) @ W_d.T) + fl @ np.abs(W_d).T)
        bound[rows] = best
    return out, bound


def swiglu_noise(gate, up, d_gate, d_up, alpha=1.702, limit=7.0):
    """Largest change of the clamped SwiGLU when gate and up move by at most
    d_gate and d_up: the four corners of that box. The function is monotone
    in the clamped up value and smooth in gate, so over intervals this small
    its extremes lie at the corners."""
    h0 = ref_swiglu_clamped(gate, up, alpha, limit)
    n = np.zeros_like(h0)
    for sg in (-1.0, 1.0):
        for su in (-1.0, 1.0):
            n = np.maximum(n, np.abs(ref_swiglu_clamped(gate + sg * d_gate, up + su * d_up, alpha, limit) - h0))
    return n


def _split_gate_up(G, I, interleaved):
    if interleaved:
        return G[:, 0::2], G[:, 1::2]
    return G[:, :I], G[:, I:]


def ref_moe_finalize(y_slot, k):
    """The MoE finalize step (§IV-A, the "MoE finalize" kernel of Table I), as
    the method declares it: y_slot [T·k, H] holds each token's k routed slot
    outputs, already multiplied by their routing weights, row t·k + j for
    slot j of token t; out[t] = Σ_j y_slot[t·k + j] over j = 0 .. k−1, in
    ascending j. Exact in fp64 for the decoded bf16 inputs of the tests."""
    y = np.asarray(y_slot, dtype=np.float64)
    if y.shape[0] % k != 0:
        raise ValueError("rows of y_slot must be a multiple of k")
    T = y.shape[0] // k
    out = np.zeros((T, y.shape[1]), dtype=np.float64)
    for j in range(k):
        out += y[j::k]
    return out


def ref_expert_rows(X, W_gu, W_d, storage="bf16", act_quant=False, alpha=1.702,
                    limit=7.0, interleaved=False, with_bound=False):
    """One expert's FFN over rows X [n, H] → y [n, H] (unweighted), fp64.

    storage: the declared format of the intermediate h — "bf16" (RNE),
    "e4m3" (bf16 RNE, then per-row e4m3 with an fp32 scale) or "none".
    act_quant: quantise X per row to e4m3 first (the W8A8 variant)."""
    X = np.asarray(X, dtype=np.float64)
    I = W_d.shape[1]
    if act_quant:
        q, s = ref_quant_rows_e4m3(X)
        X = _dequant_rows(q, s)
    G = X @ np.asarray(W_gu, dtype=np.float64).T
    gate, up = _split_gate_up(G, I, interleaved)
    h = ref_swiglu_clamped(gate, up, alpha, limit)
    W_d = np.asarray(W_d, dtype=np.float64)
    if with_bound:
        noise = None
        if act_quant:
            # the e4m3 contraction's accumulation noise, per element of G
            dG = f8_contraction_noise(X, W_gu)
            d_gate, d_up = _split_gate_up(dG, I, interleaved)
            noise = swiglu_noise(gate, up, d_gate, d_up, alpha, limit)
        out, bound = storage_bound(h, storage, W_d, noise)
        narrow = bound if noise is None else storage_bound(h, storage, W_d, None)[1]
        return out, bound, narrow
    return store_h(h, storage) @ W_d.T


def ref_moe(x, logits, weights, k, storage="bf16", act_quant=False, alpha=1.702,
            limit=7.0, interleaved=False, tokens=None, with_bound=False):
    """The MoE expert FFN step, fp64.

    x: [T, H] fp64 (decoded bf16 tokens); logits: [T, E] (fp32 values);
    weights: callable e -> (W_gu [2I, H], W_d [H, I]) fp64 (decoded, scales
    applied), or a pair of arrays [E, 2I, H], [E, H, I].
    tokens: optional subset of token ids whose outputs to compute (a token's
    output depends only on its own row and its own routing).
    with_bound: also return "out_bound", per output element the largest
    change any storage-rounding decision of h within the fragile
    neighbourhood of a boundary (see storage_bound; with act_quant it
    includes the e4m3 contraction's accumulation noise, F8_DOT_NOISE) can
    cause; a kernel that evaluates h in another rounding order may take
    those decisions either way, and every such result is correct. And
    "out_bound_narrow", the same without the accumulation noise (h within
    fp32 evaluation noise of the exact value), which only the rare
    decisions that noise moves may exceed.
    Returns a dict: out [T or len(tokens), H], idx, w, counts, offsets, perm
    (and out_bound).
    """
    x = np.asarray(x, dtype=np.float64)
    T, H = x.shape
    E = np.asarray(logits).shape[1]
    if not callable(weights):
        Wgu_all, Wd_all = weights
        weights = lambda e: (Wgu_all[e], Wd_all[e])  # noqa: E731
    idx, w = ref_route(logits, k)
    counts, offsets, perm = ref_permute(idx, E)
    tok = np.arange(T) if tokens is None else np.asarray(tokens, dtype=np.int64)
    # compact slot buffer: row c·k + j holds slot (tok[c], j)
    row_of_token = np.full(T, -1, dtype=np.int64)
    row_of_token[tok] = np.arange(tok.size)
    y_slot = np.zeros((tok.size * k, H), dtype=np.float64)
    b_slot = np.zeros((tok.size * k, H), dtype=np.float64) if with_bound else None
    n_slot = np.zeros((tok.size * k, H), dtype=np.float64) if with_bound else None
    for e in range(E):
        slots = perm[offsets[e]:offsets[e + 1]].astype(np.int64)
        slots = slots[row_of_token[slots // k] >= 0]
        if slots.size == 0:
            continue
        W_gu, W_d = weights(e)
        dst = row_of_token[slots // k] * k + slots % k
        if with_bound:
            y, yb, yn = ref_expert_rows(x[slots // k], W_gu, W_d, storage, act_quant, alpha,
                                        limit, interleaved, with_bound=True)
            b_slot[dst] = yb
            n_slot[dst] = yn
        else:
            y = ref_expert_rows(x[slots // k], W_gu, W_d, storage, act_quant, alpha,
                                limit, interleaved)
        y_slot[dst] = y
    # finalize: the routing-weighted sum of each token's k slot outputs,
    # j ascending, exact until the output
    out = np.zeros((tok.size, H), dtype=np.float64)
    bound = np.zeros((tok.size, H), dtype=np.float64) if with_bound else None
    narrow = np.zeros((tok.size, H), dtype=np.float64) if with_bound else None
    for j in range(k):
        out += w[tok, j][:, None] * y_slot[j::k]
        if with_bound:
            bound += w[tok, j][:, None] * b_slot[j::k]
            narrow += w[tok, j][:, None] * n_slot[j::k]
    res = {"out": out, "idx": idx, "w": w, "counts": counts, "offsets": offsets, "perm": perm}
    if with_bound:
        res["out_bound"] = bound
        res["out_bound_narrow"] = narrow
    return res
