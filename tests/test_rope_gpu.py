"""GPU parity of the QKV bias + RoPE + paged KV-cache update (paper §IV-A,
Table I) against the fp64 oracle.

Rotated query and key heads: each bf16 output lies within one bf16 spacing
of the exact rotated value, up to the fp32 noise of the rotation (4e-6 at
these magnitudes), and the rows pass the bf16 tolerance. Value heads: the
bias add is exact in fp32 wherever the host confirms it, and there the
stored value must be the RNE of the exact sum bit for bit. Every cache row
the step does not write keeps its prior bits. Covers the Table I batch sizes
with gpt-oss-20b's attention sizes, interleaved pairs, positions up to
131071 (angles of ~10^5 rad), no bias, other head sizes, more work items
than threads, out-of-range positions and block ids, and determinism."""

import numpy as np
import pytest
import torch

from oracle import bf16_decode, bf16_encode_rne, compare, ref_bias_rope_kv_update
from paper_2606_02963_amd import api
from paper_2606_02963_amd.synth import FINALIZE_BATCHES, RopeSpec, make_rope_inputs
from tests.gpu_helpers import dev_bf16, log, require_gpu

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _close_to_exact(got_bits, want, slack=4e-6):
    got = bf16_decode(got_bits)
    spacing = np.where(want != 0, np.exp2(np.floor(np.log2(np.abs(np.where(want != 0, want, 1.0)))) - 7), 0.0)
    return bool(np.all(np.abs(got - want) <= spacing + slack))


def run_case(spec, inp, with_bias=True):
    require_gpu()
    log(f"[rope] T={spec.T} n_q={spec.n_q} n_kv={spec.n_kv} D={spec.D} bs={spec.block_size} "
        f"interleaved={spec.interleaved} max_pos={spec.max_pos} bias={with_bias}")
    qkv, bias = dev_bf16(inp["qkv"]), dev_bf16(inp["bias"]) if with_bias else None
    pos = torch.from_numpy(inp["positions"]).cuda()
    table = torch.from_numpy(inp["block_table"]).cuda()
    cache = dev_bf16(inp["cache"])
    q = api.bias_rope_kv_update(qkv, bias, pos, table, cache, spec.n_q, spec.n_kv, spec.D, spec.base,
                                spec.interleaved)
    torch.cuda.synchronize()
    q_bits, cache_bits = _bits(q), _bits(cache)
    b64 = bf16_decode(inp["bias"]) if with_bias else None
    q_ref, cache_ref, written = ref_bias_rope_kv_update(
        bf16_decode(inp["qkv"]), b64, inp["positions"], inp["block_table"], bf16_decode(inp["cache"]),
        spec.n_q, spec.n_kv, spec.D, spec.block_size, spec.base, spec.interleaved)
    # rows the step does not write keep their bits
    assert np.array_equal(cache_bits[~written], inp["cache"][~written]), "an unwritten cache row changed"
    assert _close_to_exact(q_bits, q_ref), "a query output is off by more than one bf16 step"
    k_w = written[:, 0]
    assert _close_to_exact(cache_bits[:, 0][k_w], cache_ref[:, 0][k_w]), "a key is off by more than one bf16 step"
    # values: bit-exact where the fp32 bias add is exact
    v_got, v_ref = cache_bits[:, 1][written[:, 1]], cache_ref[:, 1][written[:, 1]]
    exact32 = v_ref.astype(np.float32).astype(np.float64) == v_ref
    assert exact32.mean() > 0.99
    assert np.array_equal(v_got[exact32], bf16_encode_rne(v_ref[exact32])), "a value differs from RNE(v + b)"
    assert _close_to_exact(v_got[~exact32], v_ref[~exact32])
    rep_q = compare(bf16_decode(q_bits), q_ref, "bf16")
    rep_k = compare(bf16_decode(cache_bits[:, 0][k_w]), cache_ref[:, 0][k_w], "bf16") if k_w.any() else None
    log(f"    q {rep_q}" + (f"; k {rep_k}" if rep_k else ""))
    assert rep_q.ok and (rep_k is None or rep_k.ok)
    return q_bits, cache_bits, written


@pytest.mark.parametrize("T", FINALIZE_BATCHES)
def test_rope_table_i_batches(T):
    spec = RopeSpec(T)
    run_case(spec, make_rope_inputs(spec, seed=1))


@pytest.mark.parametrize("spec", [
    RopeSpec(16, interleaved=True),
    RopeSpec(32, max_pos=131072),                              # angles up to ~1.3e5 rad
    RopeSpec(32, max_pos=131072, interleaved=True),
    RopeSpec(7, n_q=8, n_kv=2, D=128, block_size=16, base=10000.0),
    RopeSpec(5, n_q=3, n_kv=1, D=16, block_size=5, max_pos=97),  # odd sizes, block size 5
    RopeSpec(9, n_q=128, n_kv=16, D=128, block_size=32),        # 1408 items > 1024 threads
    RopeSpec(9, n_q=16, n_kv=4, D=256, block_size=8, interleaved=True),
    RopeSpec(1024),                                             # a prefill-sized batch of tokens
], ids=lambda s: f"T{s.T}_q{s.n_q}_kv{s.n_kv}_D{s.D}_bs{s.block_size}_p{s.max_pos}_il{int(s.interleaved)}")
def test_rope_geometries(spec):
    run_case(spec, make_rope_inputs(spec, seed=2))


def test_rope_without_bias():
    spec = RopeSpec(12)
    run_case(spec, make_rope_inputs(spec, seed=3), with_bias=False)


def test_rope_out_of_range_tokens_write_no_cache_row():
    spec = RopeSpec(8, max_pos=256)
    inp = make_rope_inputs(spec, seed=4)
    maxb = inp["block_table"].shape[1]
    inp["positions"][0] = maxb * spec.block_size                 # one past the table
    inp["positions"][1] = -3
    t2, t3 = 2, 3
    inp["block_table"][t2, inp["positions"][t2] // spec.block_size] = spec.num_blocks
    inp["block_table"][t3, inp["positions"][t3] // spec.block_size] = -1
    _, _, written = run_case(spec, inp)
    assert written[:, 0, 0].sum() == 4                          # tokens 4..7 only


def test_rope_empty_and_deterministic():
    require_gpu()
    spec = RopeSpec(0)
    q = api.bias_rope_kv_update(torch.empty((0, spec.width), dtype=torch.bfloat16, device="cuda"), None,
                                torch.empty(0, dtype=torch.int32, device="cuda"),
                                torch.empty((0, 4), dtype=torch.int32, device="cuda"),
                                torch.zeros((4, 2, spec.n_kv, spec.block_size, spec.D), dtype=torch.bfloat16,
                                            device="cuda"), spec.n_q, spec.n_kv, spec.D, spec.base)
    torch.cuda.synchronize()
    assert q.shape == (0, spec.n_q, spec.D)
    spec = RopeSpec(64)
    inp = make_rope_inputs(spec, seed=5)
    q1, c1, _ = run_case(spec, inp)
    q2, c2, _ = run_case(spec, inp)
    assert np.array_equal(q1, q2) and np.array_equal(c1, c2)
