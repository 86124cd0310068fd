"""Pins for the QKV bias + RoPE + KV-cache update oracle (``oracle.rope``).

Against an mpmath brute force of the definition in its complex form (pair i
as a + j·b times e^(j·pos·θ_i)); closed forms (position 0 is the identity,
pair 0 turns by pos radians because θ_0 = 1, the last pair's frequency is
base^(−(D−2)/D)); invariants of a rotation (each pair keeps its length,
rotations compose additively in the position, a query-key dot product depends
only on the position difference); torch's complex multiply in fp64; and the
cache placement rules (the written rows are exactly block_table[t, pos //
block_size] at row pos % block_size, nothing else changes, out-of-range
positions and block ids write nothing). Planted mistakes — sine sign, pair
layout, rotated values, bias after the rotation, a frequency exponent of i/D,
a block index or row off by one — each fail a pin."""

import math

import mpmath as mp
import numpy as np
import pytest
import torch

import oracle.rope as orp
from oracle.codecs import bf16_decode, bf16_encode_rne
from oracle.rope import ref_bias_rope_kv_update, ref_rope, rope_freqs, rope_pairs

mp.mp.dps = 50


def _bf16(a):
    return bf16_decode(bf16_encode_rne(np.asarray(a, dtype=np.float64)))


def _mp_rotate(x, pos, base, interleaved):
    """Brute force: complex multiply of each pair, 50 digits."""
    D = len(x)
    out = [None] * D
    for i in range(D // 2):
        ia, ib = (2 * i, 2 * i + 1) if interleaved else (i, i + D // 2)
        th = mp.power(mp.mpf(base), -mp.mpf(2 * i) / D)
        z = (mp.mpf(float(x[ia])) + 1j * mp.mpf(float(x[ib]))) * mp.expj(mp.mpf(int(pos)) * th)
        out[ia], out[ib] = z.real, z.imag
    return out


def _small_case(seed, T=3, n_q=2, n_kv=1, D=8, bs=4, max_pos=40, interleaved=False, nb=None):
    rng = np.random.default_rng(seed)
    W = (n_q + 2 * n_kv) * D
    qkv = _bf16(rng.standard_normal((T, W)))
    bias = _bf16(rng.uniform(-0.1, 0.1, W))
    pos = rng.integers(0, max_pos, T)
    maxb = (max_pos + bs - 1) // bs
    nb = nb or 2 * T + 3
    perm = rng.permutation(nb)
    table = perm[T:][rng.integers(0, nb - T, (T, maxb))]
    table[np.arange(T), pos // bs] = perm[:T]
    cache = _bf16(rng.standard_normal((nb, 2, n_kv, bs, D)))
    return dict(qkv=qkv, bias=bias, positions=pos, block_table=table, cache=cache, n_q=n_q, n_kv=n_kv,
                D=D, block_size=bs, interleaved=interleaved)


def _run(case, base=150000.0, fn=None):
    fn = fn or ref_bias_rope_kv_update
    c = dict(case)
    return fn(c.pop("qkv"), c.pop("bias"), c.pop("positions"), c.pop("block_table"), c.pop("cache"),
              c["n_q"], c["n_kv"], c["D"], c["block_size"], base, c["interleaved"])


@pytest.mark.parametrize("interleaved", [False, True])
def test_bruteforce_mpmath_whole_step(interleaved):
    case = _small_case(41, interleaved=interleaved)
    base = 10000.0
    q, cache, written = _run(case, base)
    n_q, n_kv, D, bs = case["n_q"], case["n_kv"], case["D"], case["block_size"]
    for t in range(case["qkv"].shape[0]):
        s = [mp.mpf(float(case["qkv"][t, i])) + mp.mpf(float(case["bias"][i])) for i in range(len(case["bias"]))]
        p = int(case["positions"][t])
        for h in range(n_q):
            want = _mp_rotate(s[h * D:(h + 1) * D], p, base, interleaved)
            for d in range(D):
                assert abs(q[t, h, d] - float(want[d])) <= 1e-15 * (1 + abs(float(want[d])))
        blk, row = int(case["block_table"][t, p // bs]), p % bs
        for h in range(n_kv):
            kw = _mp_rotate(s[(n_q + h) * D:(n_q + h + 1) * D], p, base, interleaved)
            for d in range(D):
                assert abs(cache[blk, 0, h, row, d] - float(kw[d])) <= 1e-15 * (1 + abs(float(kw[d])))
                assert cache[blk, 1, h, row, d] == float(s[(n_q + n_kv + h) * D + d])   # values: not rotated


def test_position_zero_is_identity_and_pair0_turns_by_pos_radians():
    rng = np.random.default_rng(42)
    x = rng.standard_normal((5, 16))
    np.testing.assert_array_equal(ref_rope(x, np.zeros(5), 150000.0), x)
    for interleaved in (False, True):
        a, b = rope_pairs(16, interleaved)
        for p in (1, 7, 1000):
            y = ref_rope(x, np.full(5, p), 150000.0, interleaved)
            c, s = math.cos(p), math.sin(p)
            np.testing.assert_allclose(y[:, a[0]], x[:, a[0]] * c - x[:, b[0]] * s, rtol=1e-14, atol=1e-14)
            np.testing.assert_allclose(y[:, b[0]], x[:, a[0]] * s + x[:, b[0]] * c, rtol=1e-14, atol=1e-14)
    th = rope_freqs(64, 150000.0)
    assert th[0] == 1.0
    assert abs(th[-1] - 150000.0 ** (-62 / 64)) <= 1e-16 * th[-1]
    assert np.all(np.diff(th) < 0)


def test_rotation_invariants():
    rng = np.random.default_rng(43)
    D = 64
    for interleaved in (False, True):
        a, b = rope_pairs(D, interleaved)
        assert sorted(np.concatenate([a, b]).tolist()) == list(range(D))     # pairs partition the head
        q, k = rng.standard_normal((2, 6, D))
        p, s = rng.integers(0, 5000, (2, 6))
        rq, rk = ref_rope(q, p, 150000.0, interleaved), ref_rope(k, s, 150000.0, interleaved)
        # each pair keeps its length
        np.testing.assert_allclose(rq[:, a] ** 2 + rq[:, b] ** 2, q[:, a] ** 2 + q[:, b] ** 2, rtol=1e-12)
        # composition: R(p2) R(p1) = R(p1 + p2)
        np.testing.assert_allclose(ref_rope(rq, s, 150000.0, interleaved),
                                   ref_rope(q, p + s, 150000.0, interleaved), rtol=1e-9, atol=1e-10)
        # q·k depends only on the position difference
        c = 1234
        d1 = np.sum(rq * rk, axis=1)
        d2 = np.sum(ref_rope(q, p + c, 150000.0, interleaved) * ref_rope(k, s + c, 150000.0, interleaved), axis=1)
        np.testing.assert_allclose(d1, d2, rtol=1e-9, atol=1e-9)


def test_matches_torch_complex_multiply():
    rng = np.random.default_rng(44)
    D, base = 64, 150000.0
    x = rng.standard_normal((7, D))
    p = rng.integers(0, 131072, 7)
    th = torch.pow(torch.tensor(base, dtype=torch.float64), -torch.arange(0, D, 2, dtype=torch.float64) / D)
    rot = torch.polar(torch.ones(7, D // 2, dtype=torch.float64), torch.from_numpy(p).double()[:, None] * th)
    xt = torch.from_numpy(x)
    # interleaved: adjacent pairs are the complex view of the head
    zi = torch.view_as_complex(xt.reshape(7, D // 2, 2).contiguous()) * rot
    np.testing.assert_allclose(ref_rope(x, p, base, True), torch.view_as_real(zi).reshape(7, D).numpy(),
                               rtol=1e-12, atol=1e-12)
    # half-split: first half real, second half imaginary
    zh = torch.complex(xt[:, :D // 2], xt[:, D // 2:]) * rot
    np.testing.assert_allclose(ref_rope(x, p, base, False), torch.cat([zh.real, zh.imag], 1).numpy(),
                               rtol=1e-12, atol=1e-12)


def test_cache_placement_and_out_of_range():
    case = _small_case(45, T=5, max_pos=37, nb=20)
    q, cache, written = _run(case)
    bs = case["block_size"]
    want = np.zeros_like(written)
    for t, p in enumerate(case["positions"]):
        want[case["block_table"][t, p // bs], :, :, p % bs] = True
    np.testing.assert_array_equal(written, want)
    np.testing.assert_array_equal(cache[~written], case["cache"][~written])
    # positions past the table, negative positions and bad block ids write nothing
    bad = dict(case)
    bad["positions"] = case["positions"].copy()
    bad["block_table"] = case["block_table"].copy()
    maxb = case["block_table"].shape[1]
    bad["positions"][0] = maxb * bs          # one past the table
    bad["positions"][1] = -1
    t2 = 2
    bad["block_table"][t2, bad["positions"][t2] // bs] = 20      # == num_blocks
    bad["block_table"][3, bad["positions"][3] // bs] = -5
    _, cache_b, written_b = _run(bad)
    assert written_b.sum() == written[case["block_table"][4, case["positions"][4] // bs]].sum()
    np.testing.assert_array_equal(cache_b[~written_b], case["cache"][~written_b])


def test_pins_catch_planted_mistakes(monkeypatch):
    good_rope, good_freqs, good_update = orp.ref_rope, orp.rope_freqs, orp.ref_bias_rope_kv_update

    def sin_sign(x, pos, base, interleaved=False):
        return good_rope(x, -np.asarray(pos), base, interleaved)

    def wrong_pairs(x, pos, base, interleaved=False):
        return good_rope(x, pos, base, not interleaved)

    def exponent_i_over_d(D, base):
        return np.power(float(base), -1.0 * np.arange(D // 2) / D)

    def rotate_values(qkv, bias, positions, block_table, cache, n_q, n_kv, D, bs, base, il=False):
        q, c, w = good_update(qkv, bias, positions, block_table, cache, n_q, n_kv, D, bs, base, il)
        c = c.copy()
        for t, p in enumerate(positions):
            if 0 <= p < block_table.shape[1] * bs:
                blk = block_table[t, p // bs]
                c[blk, 1, :, p % bs] = good_rope(c[blk, 1, :, p % bs], p, base, il)
        return q, c, w

    def bias_after(qkv, bias, positions, block_table, cache, n_q, n_kv, D, bs, base, il=False):
        q, c, w = good_update(qkv, None, positions, block_table, cache, n_q, n_kv, D, bs, base, il)
        return q + np.asarray(bias)[None, :n_q * D].reshape(1, n_q, D), c, w

    def block_off_by_one(qkv, bias, positions, block_table, cache, n_q, n_kv, D, bs, base, il=False):
        # rotate at pos but store through the next block-table entry
        q, c, w = good_update(qkv, bias, positions, block_table, cache, n_q, n_kv, D, bs, base, il)
        c2, w2 = np.array(cache, dtype=np.float64), np.zeros_like(w)
        for t, p in enumerate(positions):
            j = min(p // bs + 1, block_table.shape[1] - 1)
            blk, b2, r = block_table[t, p // bs], block_table[t, j], p % bs
            c2[b2, :, :, r] = c[blk, :, :, r]
            w2[b2, :, :, r] = True
        return q, c2, w2

    def row_off_by_one(qkv, bias, positions, block_table, cache, n_q, n_kv, D, bs, base, il=False):
        # rotate at pos but store at row pos % bs + 1 (within the same block)
        q, c, w = good_update(qkv, bias, positions, block_table, cache, n_q, n_kv, D, bs, base, il)
        c2, w2 = np.array(cache, dtype=np.float64), np.zeros_like(w)
        for t, p in enumerate(positions):
            blk, r = block_table[t, p // bs], p % bs
            c2[blk, :, :, (r + 1) % bs] = c[blk, :, :, r]
            w2[blk, :, :, (r + 1) % bs] = True
        return q, c2, w2

    pins = [
        lambda: test_bruteforce_mpmath_whole_step(False),
        lambda: test_bruteforce_mpmath_whole_step(True),
        test_position_zero_is_identity_and_pair0_turns_by_pos_radians,
        test_matches_torch_complex_multiply,
        test_cache_placement_and_out_of_range,
    ]
    mistakes = [("ref_rope", sin_sign), ("ref_rope", wrong_pairs), ("rope_freqs", exponent_i_over_d),
                ("ref_bias_rope_kv_update", rotate_values), ("ref_bias_rope_kv_update", bias_after),
                ("ref_bias_rope_kv_update", block_off_by_one), ("ref_bias_rope_kv_update", row_off_by_one)]
    for attr, bad in mistakes:
        with monkeypatch.context() as m:
            m.setattr(orp, attr, bad)
            # the pins reach the functions through these module-level names
            g = globals()
            saved = {n: g[n] for n in ("ref_rope", "rope_freqs", "ref_bias_rope_kv_update")}
            g[attr] = bad
            caught = False
            try:
                for pin in pins:
                    try:
                        pin()
                    except AssertionError:
                        caught = True
                        break
            finally:
                g.update(saved)
            assert caught, f"planted mistake {bad.__name__} in {attr} was not caught"
