"""fp64 oracle for the fused QKV bias + rotary embedding + KV-cache update of
the gpt-oss-20b decode path (paper §IV-A, "Bias + RoPE + KV update" in
Table I).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper names the kernel and its batch sweep only; the operation is the
standard attention pre-processing of one decode step. Each of the T tokens is
the newest token of its own sequence and sits at position ``pos[t]``:

  1. s = qkv[t] + bias                    — the QKV projection's bias
  2. split s into n_q query heads, n_kv key heads and n_kv value heads of
     head_dim D each, in that order
  3. rotate every query and key head by its position (rotary position
     embedding, Su et al., "RoFormer"): the head's D values form D/2 pairs
     (a_i, b_i); pair i is read as the complex number a_i + j·b_i and
     multiplied by e^(j·pos·θ_i), θ_i = base^(−2i/D), i.e.
         a' = a·cos(pos·θ_i) − b·sin(pos·θ_i)
         b' = a·sin(pos·θ_i) + b·cos(pos·θ_i)
     Pairs are (i, i + D/2) in the half-split layout (GPT-NeoX style) and
     (2i, 2i + 1) in the interleaved layout (the RoFormer paper's own).
     Value heads are not rotated.
  4. the rotated query heads are the output q; the rotated key heads and the
     value heads are written into a paged KV cache at the token's position:
     block = block_table[t, pos // block_size], row pos % block_size, cache
     layout [num_blocks, 2 (key, value), n_kv, block_size, D]. A token whose
     position lies outside its block table, or whose block id lies outside
     the cache, writes nothing to the cache.

Everything is fp64 on the exact stored values (bf16 decoded); the angles are
fp64 products pos·θ_i, and nothing is rounded.
"""

import numpy as np


def rope_pairs(D, interleaved):
    """Index arrays (a, b) of the D/2 rotated pairs of one head."""
    if D % 2:
        raise ValueError("head_dim must be even")
    i = np.arange(D // 2)
    if interleaved:
        return 2 * i, 2 * i + 1
    return i, i + D // 2


def rope_freqs(D, base):
    """θ_i = base^(−2i/D), i = 0 .. D/2 − 1."""
    return np.power(float(base), -2.0 * np.arange(D // 2) / D)


def ref_rope(x, pos, base, interleaved=False):
    """Rotate the last axis (one head of D values) of x[..., D] by the
    positions pos (shape x.shape[:-1], broadcastable)."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    a, b = rope_pairs(D, interleaved)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * rope_freqs(D, base)
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    out[..., a] = x[..., a] * c - x[..., b] * s
    out[..., b] = x[..., a] * s + x[..., b] * c
    return out


def ref_bias_rope_kv_update(qkv, bias, positions, block_table, cache, n_q, n_kv, D, block_size,
                            base, interleaved=False):
    """One decode step's QKV bias, RoPE and KV-cache write.

    qkv [T, (n_q + 2·n_kv)·D], bias [(n_q + 2·n_kv)·D] or None, positions
    [T] int, block_table [T, max_blocks] int, cache [num_blocks, 2, n_kv,
    block_size, D] — fp64 values of the stored inputs (the cache's contents
    before the step). Returns (q [T, n_q, D], cache_after, written) where
    written [num_blocks, 2, n_kv, block_size] marks the cache rows the step
    writes; every other row of cache_after equals the input cache."""
    qkv = np.asarray(qkv, dtype=np.float64)
    T = qkv.shape[0]
    if qkv.shape[1] != (n_q + 2 * n_kv) * D:
        raise ValueError("qkv row length must be (n_q + 2·n_kv)·D")
    s = qkv + (np.asarray(bias, dtype=np.float64)[None, :] if bias is not None else 0.0)
    q = s[:, :n_q * D].reshape(T, n_q, D)
    k = s[:, n_q * D:(n_q + n_kv) * D].reshape(T, n_kv, D)
    v = s[:, (n_q + n_kv) * D:].reshape(T, n_kv, D)
    pos = np.asarray(positions, dtype=np.int64)
    q_rot = ref_rope(q, pos[:, None], base, interleaved)
    k_rot = ref_rope(k, pos[:, None], base, interleaved)
    cache_after = np.array(cache, dtype=np.float64, copy=True)
    written = np.zeros(cache_after.shape[:4], dtype=bool)
    block_table = np.asarray(block_table, dtype=np.int64)
    max_blocks = block_table.shape[1]
    for t in range(T):
        p = int(pos[t])
        if p < 0 or p // block_size >= max_blocks:
            continue
        blk = int(block_table[t, p // block_size])
        if blk < 0 or blk >= cache_after.shape[0]:
            continue
        row = p % block_size
        cache_after[blk, 0, :, row, :] = k_rot[t]
        cache_after[blk, 1, :, row, :] = v[t]
        written[blk, :, :, row] = True
    return q_rot, cache_after, written
