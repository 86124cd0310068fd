"""Pins for the MoE oracle (``oracle.moe``).

Routing is checked against its defining property (every unselected expert
ranks below the last selected one under (value desc, index asc)) and closed
forms (arange and all-equal logits); the permutation against its definition
(a stable sort by expert); the clamped SwiGLU against its special values and
mpmath; the whole block against a token-order brute force in mpmath that
never builds the permutation, against the dense FFN it reduces to at E = 1,
k = 1, and against the identical-experts and zero-W_down closed forms. The
W8A8 composition (per-token and per-slot-row e4m3 quantisation, e4m3
weights with per-row scales) is pinned by a second token-order brute force
that rebuilds every storage rounding from the format definitions with exact
rationals, and planted mistakes in the dequantisation and in h's storage
must fail it. The fp8 activation quantiser is pinned by the e4m3 grid and by
its extreme code.
The standalone finalize is pinned by an mpmath brute force over (token,
column, slot), the k = 1 identity and an exactly cancelling slot pair."""

import math

import mpmath as mp
import numpy as np
import pytest

import oracle.moe as om
from oracle.codecs import bf16_decode, bf16_encode_rne, e4m3_decode
from oracle.fgemm import ref_fgemm
from oracle.moe import (ref_moe, ref_moe_finalize, ref_permute, ref_quant_rows_e4m3, ref_route,
                        ref_swiglu_clamped)
from paper_2606_02963_amd.synth import MoeSpec, make_moe_activations, make_moe_weights

mp.mp.dps = 50


def _check_route_property(logits, idx, w):
    T, E = logits.shape
    k = idx.shape[1]
    for t in range(T):
        sel = list(idx[t])
        assert len(set(sel)) == k
        keys = [(logits[t, e], -e) for e in sel]
        assert keys == sorted(keys, reverse=True)
        last = keys[-1]
        for e in range(E):
            if e not in sel:
                assert (logits[t, e], -e) < last
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=1e-15)
    assert np.all(np.diff(w, axis=1) <= 0)


def test_route_closed_forms():
    lg = np.tile(np.arange(32, dtype=np.float64), (3, 1))
    idx, w = ref_route(lg, 4)
    assert idx.tolist() == [[31, 30, 29, 28]] * 3
    e = np.exp([0.0, -1.0, -2.0, -3.0])
    np.testing.assert_allclose(w, np.tile(e / e.sum(), (3, 1)), rtol=1e-15)
    idx, w = ref_route(np.zeros((2, 32)), 4)
    assert idx.tolist() == [[0, 1, 2, 3]] * 2
    np.testing.assert_array_equal(w, 0.25)


def test_route_defining_property_with_ties():
    rng = np.random.default_rng(11)
    lg = np.round(rng.standard_normal((200, 32)) * 2) / 2      # many exact ties
    idx, w = ref_route(lg, 4)
    _check_route_property(lg, idx, w)
    lg = rng.standard_normal((300, 32)).astype(np.float32).astype(np.float64)
    idx, w = ref_route(lg, 4)
    _check_route_property(lg, idx, w)


def test_route_weights_mpmath():
    rng = np.random.default_rng(12)
    lg = rng.standard_normal((5, 8))
    idx, w = ref_route(lg, 3)
    for t in range(5):
        ex = [mp.exp(mp.mpf(float(lg[t, e]))) for e in idx[t]]
        s = mp.fsum(ex)
        np.testing.assert_allclose(w[t], [float(v / s) for v in ex], rtol=1e-15)


def test_permute_definition():
    rng = np.random.default_rng(13)
    idx = rng.integers(0, 8, size=(50, 4)).astype(np.int32)
    idx[:, 1] = (idx[:, 0] + 1) % 8        # keep experts distinct per token (not required)
    counts, offsets, perm = ref_permute(idx, 10)   # experts 8, 9 empty
    flat = idx.reshape(-1)
    assert sorted(perm.tolist()) == list(range(200))
    np.testing.assert_array_equal(counts, np.bincount(flat, minlength=10))
    assert offsets[0] == 0 and offsets[-1] == 200
    np.testing.assert_array_equal(np.diff(offsets), counts)
    assert counts[8] == 0 and offsets[8] == offsets[9] == offsets[10]
    for e in range(10):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e)
        assert np.all(np.diff(seg) > 0)       # stable: ascending slot id within an expert


def test_swiglu_special_values_and_mpmath():
    g = np.array([0.0, 1.0, 7.0, 8.0, 100.0, -3.0])
    u = np.array([5.0, -1.0, 2.0, 2.0, 9.0, -9.0])
    out = ref_swiglu_clamped(g, u)
    assert out[0] == 0.0 and out[1] == 0.0                     # gate 0 / up −1 give 0
    assert out[3] == out[2] and out[4] == ref_swiglu_clamped(np.array([7.0]), np.array([7.0]))[0]
    assert out[5] == ref_swiglu_clamped(np.array([-3.0]), np.array([-7.0]))[0]
    rng = np.random.default_rng(14)
    gg, uu = rng.standard_normal(50) * 6, rng.standard_normal(50) * 6
    got = ref_swiglu_clamped(gg, uu)
    for i in range(50):
        gm = min(mp.mpf(float(gg[i])), 7)
        um = min(max(mp.mpf(float(uu[i])), -7), 7)
        want = (um + 1) * gm / (1 + mp.exp(-mp.mpf("1.702") * gm))
        assert abs(got[i] - float(want)) <= 1e-14 * max(1.0, abs(float(want)))


def _mp_bruteforce_moe(x, lg, Wgu, Wd, k, alpha=1.702, limit=7.0):
    """Token-order evaluation in mpmath: no histogram, no permutation."""
    T, H = x.shape
    E = lg.shape[1]
    I = Wd.shape[2]
    out = np.zeros((T, H))
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-lg[t, e], e))[:k]
        ex = [mp.exp(mp.mpf(float(lg[t, e]))) for e in order]
        den = mp.fsum(ex)
        acc = [mp.mpf(0)] * H
        for j, e in enumerate(order):
            xs = [mp.mpf(float(v)) for v in x[t]]
            G = [mp.fsum(xs[c] * mp.mpf(float(Wgu[e, n, c])) for c in range(H)) for n in range(2 * I)]
            h = []
            for i in range(I):
                gm = min(G[i], limit)
                um = min(max(G[I + i], -limit), limit)
                hv = (um + 1) * gm / (1 + mp.exp(-mp.mpf(alpha) * gm))
                h.append(mp.mpf(float(bf16_decode(bf16_encode_rne(np.array([float(hv)])))[0])))
            for n in range(H):
                y = mp.fsum(h[i] * mp.mpf(float(Wd[e, n, i])) for i in range(I))
                acc[n] += ex[j] / den * y
        out[t] = [float(v) for v in acc]
    return out


def test_moe_bruteforce_token_order():
    rng = np.random.default_rng(15)
    T, H, I, E, k = 6, 4, 4, 4, 2
    x = bf16_decode(bf16_encode_rne(rng.standard_normal((T, H)) * 2))
    lg = rng.standard_normal((T, E)).astype(np.float32).astype(np.float64)
    lg[2, :] = 0.5                                  # a fully tied row
    Wgu = bf16_decode(bf16_encode_rne(rng.standard_normal((E, 2 * I, H))))
    Wd = bf16_decode(bf16_encode_rne(rng.standard_normal((E, H, I))))
    got = ref_moe(x, lg, (Wgu, Wd), k)["out"]
    want = _mp_bruteforce_moe(x, lg, Wgu, Wd, k)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    # the token subset path returns the same rows
    sub = ref_moe(x, lg, (Wgu, Wd), k, tokens=[4, 1])["out"]
    np.testing.assert_allclose(sub, got[[4, 1]], rtol=0, atol=0)


def test_moe_single_expert_is_dense_ffn():
    rng = np.random.default_rng(16)
    T, H, I = 9, 8, 6
    x = rng.standard_normal((T, H))
    Wgu = rng.standard_normal((1, 2 * I, H)) * 0.5
    Wd = rng.standard_normal((1, H, I)) * 0.5
    got = ref_moe(x, rng.standard_normal((T, 1)), (Wgu, Wd), 1, storage="none")["out"]
    G = ref_fgemm(x, Wgu[0])
    h = ref_swiglu_clamped(G[:, :I], G[:, I:])
    np.testing.assert_allclose(got, ref_fgemm(h, Wd[0]), rtol=1e-14, atol=1e-14)


def test_moe_identical_experts_and_zero_down():
    rng = np.random.default_rng(17)
    T, H, I, E = 7, 8, 4, 5
    x = rng.standard_normal((T, H))
    wgu1 = rng.standard_normal((2 * I, H))
    wd1 = rng.standard_normal((H, I))
    Wgu = np.stack([wgu1] * E)
    Wd = np.stack([wd1] * E)
    lg = rng.standard_normal((T, E))
    got = ref_moe(x, lg, (Wgu, Wd), 3, storage="none")["out"]
    G = x @ wgu1.T
    want = ref_swiglu_clamped(G[:, :I], G[:, I:]) @ wd1.T
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)
    z = ref_moe(x, lg, (Wgu, np.zeros_like(Wd)), 3)["out"]
    assert np.all(z == 0.0)


def test_interleaved_gate_up_is_a_row_permutation():
    rng = np.random.default_rng(18)
    T, H, I = 5, 8, 4
    x = rng.standard_normal((T, H))
    Wgu = rng.standard_normal((1, 2 * I, H))
    Wd = rng.standard_normal((1, H, I))
    lg = np.zeros((T, 1))
    a = ref_moe(x, lg, (Wgu, Wd), 1, storage="none")["out"]
    inter = np.empty_like(Wgu)
    inter[0, 0::2], inter[0, 1::2] = Wgu[0, :I], Wgu[0, I:]
    b = ref_moe(x, lg, (inter, Wd), 1, storage="none", interleaved=True)["out"]
    np.testing.assert_allclose(a, b, rtol=1e-15, atol=1e-15)


def test_quant_rows_e4m3():
    rng = np.random.default_rng(19)
    v = rng.standard_normal((20, 300)) * rng.random((20, 1)) * 10
    v[3] = 0.0
    q, s = ref_quant_rows_e4m3(v)
    d = e4m3_decode(q)
    assert s[3] == 1.0 and np.all(q[3] == 0)
    nz = np.arange(20) != 3
    # the row maximum lands on the largest code, ±448
    assert np.all(np.max(np.abs(d[nz]), 1) == 448.0)
    # every value is within half an e4m3 step (relative 2^-4 for normals, 2^-10·s below)
    err = np.abs(d * s[:, None] - v)
    bound = np.maximum(np.abs(v) * 2.0 ** -4, s[:, None] * 2.0 ** -10) * (1 + 1e-6)
    assert np.all(err <= bound)


def test_planted_mistakes_are_caught(monkeypatch):
    """Mistakes planted in the oracle on the CPU make a pin fail: unstable
    permutation order, ties broken to the higher index, and a dropped +1 on
    the up branch."""
    orig_perm = om.ref_permute

    def unstable_perm(idx, E):
        counts, offsets, perm = orig_perm(idx, E)
        out = perm.copy()
        for e in range(E):
            out[offsets[e]:offsets[e + 1]] = out[offsets[e]:offsets[e + 1]][::-1]
        return counts, offsets, out
    with pytest.raises(AssertionError):
        test_permute_definition_via(unstable_perm)

    def route_high_ties(logits, k):
        logits = np.asarray(logits, dtype=np.float64)
        T, E = logits.shape
        idx = np.array([sorted(range(E), key=lambda e: (-logits[t, e], -e))[:k] for t in range(T)], dtype=np.int32)
        sel = np.take_along_axis(logits, idx.astype(np.int64), 1)
        ex = np.exp(sel - sel.max(1, keepdims=True))
        return idx, ex / ex.sum(1, keepdims=True)
    with pytest.raises(AssertionError):
        lg = np.zeros((2, 32))
        idx, _ = route_high_ties(lg, 4)
        assert idx.tolist() == [[0, 1, 2, 3]] * 2

    def swiglu_no_plus_one(gate, up, alpha=1.702, limit=7.0):
        g = np.minimum(gate, limit)
        return np.clip(up, -limit, limit) * g / (1 + np.exp(-alpha * g))
    with monkeypatch.context() as m:
        m.setattr(om, "ref_swiglu_clamped", swiglu_no_plus_one)
        with pytest.raises(AssertionError):
            test_moe_bruteforce_token_order()


def test_permute_definition_via(fn=ref_permute):
    rng = np.random.default_rng(20)
    idx = rng.integers(0, 6, size=(40, 3)).astype(np.int32)
    counts, offsets, perm = fn(idx, 6)
    flat = idx.reshape(-1)
    for e in range(6):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e)
        assert np.all(np.diff(seg) > 0)


def test_synth_moe_shapes_small():
    spec = MoeSpec("t", T=8, H=64, I=64, E=4, k=2)
    a = make_moe_activations(spec, 0)
    w = make_moe_weights(spec, 0)
    assert a["x"].shape == (8, 64) and a["x"].dtype == np.uint16
    assert w["w_gate_up"].shape == (4, 128, 64) and w["w_down"].shape == (4, 64, 64)
    spec8 = MoeSpec("t8", T=8, H=64, I=64, E=4, k=2, w_dtype="e4m3")
    w8 = make_moe_weights(spec8, 0)
    assert w8["w_gate_up"].dtype == np.uint8 and w8["s_gate_up"].shape == (4, 128)
    # the stored codes reproduce the fp32 draws to e4m3 precision
    d = e4m3_decode(w8["w_gate_up"]) * w8["s_gate_up"][..., None]
    wf = bf16_decode(w["w_gate_up"])
    assert np.max(np.abs(d - wf)) <= 2.0 ** -4 * np.max(np.abs(wf)) + 1e-3
    assert math.isfinite(float(d.sum()))


def test_storage_deviation_bound():
    """The flip bound is zero away from rounding boundaries and covers the
    other rounding decision at a boundary (bf16 and bf16→e4m3 storage)."""
    from oracle.moe import storage_deviation, FRAGILE_REL
    # exactly representable values: no decision is fragile
    h = np.array([[1.0, 0.5, -2.0, 0.75]])
    for st in ("bf16", "e4m3"):
        stored, dev = storage_deviation(h, st)
        assert np.all(dev == 0.0)
    # an element right at a bf16 midpoint: both roundings are legitimate
    mid = 1.0 + 2.0 ** -8
    h = np.array([[mid * (1 + 1e-9), 0.3, 0.2]])
    stored, dev = storage_deviation(h, "bf16")
    other = 1.0 if stored[0, 0] != 1.0 else 1.0 + 2.0 ** -7
    assert dev[0, 0] >= abs(other - stored[0, 0]) and dev[0, 2] == 0.0
    # e4m3 with scale 1 (row max 448): 1.06640625 is the midpoint of the bf16 values
    # 1.0625 (an e4m3 tie, rounds to 1.0) and 1.0703125 (rounds to 1.125), so the
    # stored e4m3 value may legitimately be either 1.0 or 1.125
    h = np.array([[448.0, 1.06640625 * (1 + 1e-9), 3.0]])
    stored, dev = storage_deviation(h, "e4m3")
    assert stored[0, 1] == 1.125 and dev[0, 1] == 0.125 and dev[0, 2] == 0.0
    # a value at an e4m3 tie that bf16 keeps exactly: both sides decide alike
    h = np.array([[448.0, 1.0625 * (1 - 1e-9), 3.0]])
    stored, dev = storage_deviation(h, "e4m3")
    assert stored[0, 1] == 1.0 and dev[0, 1] == 0.0
    # the MoE bound is zero for storage "none" and non-negative otherwise
    rng = np.random.default_rng(21)
    x = rng.standard_normal((6, 8))
    Wgu = rng.standard_normal((2, 8, 8)) * 0.3
    Wd = rng.standard_normal((2, 8, 4)) * 0.3
    r = ref_moe(x, rng.standard_normal((6, 2)), (Wgu, Wd), 2, storage="none", with_bound=True)
    assert np.all(r["out_bound"] == 0.0)
    r2 = ref_moe(x, rng.standard_normal((6, 2)), (Wgu, Wd), 2, storage="e4m3", with_bound=True)
    assert np.all(r2["out_bound"] >= 0.0)
    r3 = ref_moe(x, rng.standard_normal((6, 2)), (Wgu, Wd), 2, storage="e4m3")
    assert r3["out"].shape == r2["out"].shape
    assert FRAGILE_REL < 1e-4


def test_storage_deviation_noise_and_swiglu_noise(monkeypatch):
    """A per-element noise widens the neighbourhood of a boundary; the SwiGLU
    noise is zero where both inputs sit in their clamped ranges and follows
    the derivative elsewhere; the W8A8 bound includes the e4m3 contraction's
    accumulation noise and only ever grows with it."""
    import oracle.moe as om
    # 2^-12 relative above a bf16 midpoint: robust without noise, fragile with it
    mid = 1.0 + 2.0 ** -8
    h = np.array([[mid * (1 + 2.0 ** -12), 0.3]])
    assert np.all(om.storage_deviation(h, "bf16")[1] == 0.0)
    dev = om.storage_deviation(h, "bf16", noise=np.array([[2.0 ** -11, 0.0]]))[1]
    assert dev[0, 0] == 2.0 ** -7 and dev[0, 1] == 0.0
    # SwiGLU noise: zero deltas → 0; gate above the limit and up beyond ±limit → 0
    g = np.array([0.5, -1.0, 9.0, 10.0])
    u = np.array([0.2, 1.5, 8.0, -9.0])
    assert np.all(om.swiglu_noise(g, u, 0 * g, 0 * u) == 0.0)
    n = om.swiglu_noise(g, u, np.full(4, 1e-3), np.full(4, 1e-3))
    assert n[2] == 0.0 and n[3] == 0.0
    # away from the clamps it matches |∂h/∂g|·dg + |∂h/∂u|·du to first order
    a, d = 1.702, 1e-6
    sig = lambda z: 1.0 / (1.0 + np.exp(-z))
    for gi, ui in ((0.5, 0.2), (-1.0, 1.5)):
        dh_dg = (ui + 1.0) * (sig(a * gi) + a * gi * sig(a * gi) * (1 - sig(a * gi)))
        dh_du = gi * sig(a * gi)
        lin = abs(dh_dg) * d + abs(dh_du) * d
        got = om.swiglu_noise(np.array([gi]), np.array([ui]), np.array([d]), np.array([d]))[0]
        assert got == pytest.approx(lin, rel=1e-4)
    # the contraction noise: one 128-wide dot product gives ε·Σ|x·w|; the dot
    # products of a longer contraction combine as a root sum of squares, a
    # partial last one included
    xs = np.random.default_rng(5).standard_normal((3, 300))
    ws = np.random.default_rng(6).standard_normal((4, 300))
    one = om.f8_contraction_noise(xs[:, :128], ws[:, :128])
    assert np.allclose(one, om.F8_DOT_NOISE * (np.abs(xs[:, :128]) @ np.abs(ws[:, :128]).T), rtol=1e-14)
    two = om.f8_contraction_noise(np.tile(xs[:, :128], 2), np.tile(ws[:, :128], 2))
    assert np.allclose(two, np.sqrt(2.0) * one, rtol=1e-14)
    full = om.f8_contraction_noise(xs, ws)
    parts = [np.abs(xs[:, a:b]) @ np.abs(ws[:, a:b]).T for a, b in ((0, 128), (128, 256), (256, 300))]
    assert np.allclose(full, om.F8_DOT_NOISE * np.sqrt(sum(p * p for p in parts)), rtol=1e-14)
    # the W8A8 bound: larger with the accumulation noise than without it
    spec, x, lg, w = _w8a8_case()
    with_noise = ref_moe(x, lg, _w8a8_weights64(w), spec.k, storage="e4m3", act_quant=True, with_bound=True)
    monkeypatch.setattr(om, "F8_DOT_NOISE", 0.0)
    without = ref_moe(x, lg, _w8a8_weights64(w), spec.k, storage="e4m3", act_quant=True, with_bound=True)
    assert np.all(with_noise["out_bound"] >= without["out_bound"])
    assert np.array_equal(with_noise["out"], without["out"])
    assert om.F8_DOT_NOISE == 0.0 and 2.0 ** -16 < 2.0 ** -14 < 1e-4


def test_storage_bound_covers_sampled_decisions():
    """Any h′ within the neighbourhood of h (a kernel's h with that error),
    stored as declared, moves the down projection by no more than
    storage_bound; the sample includes rows whose e4m3 scale moves and rows
    whose two largest values are both fragile."""
    rng = np.random.default_rng(31)
    h = rng.standard_normal((60, 64)) * 2.0
    h[::3, 1] = h[::3, 0] = np.max(np.abs(h[::3]), axis=1) * np.array([1.0, -1.0])[rng.integers(0, 2, 20)]
    W = rng.standard_normal((24, 64)) * 0.05
    noise = 1e-3 * np.abs(h)
    pert = om.FRAGILE_REL * np.abs(h) + om.FRAGILE_ABS * np.max(np.abs(h), axis=-1, keepdims=True) + noise
    for storage in ("bf16", "e4m3"):
        out, bound = om.storage_bound(h, storage, W, noise)
        assert np.allclose(out, om.store_h(h, storage) @ W.T, rtol=0, atol=0)
        moved_scale = 0
        for trial in range(300):
            u = rng.uniform(-1.0, 1.0, h.shape) if trial % 2 else rng.choice([-1.0, 1.0], h.shape)
            h2 = h + u * pert
            y2 = om.store_h(h2, storage) @ W.T
            assert np.all(np.abs(y2 - out) <= bound * (1 + 1e-12) + 1e-15), (storage, trial)
            if storage == "e4m3":
                moved_scale += int(np.sum(ref_quant_rows_e4m3(bf16_decode(bf16_encode_rne(h2)))[1]
                                          != ref_quant_rows_e4m3(bf16_decode(bf16_encode_rne(h)))[1]))
        if storage == "e4m3":
            assert moved_scale > 100
    # a neighbourhood wider than two bf16 steps at a row maximum is refused
    with pytest.raises(ValueError):
        om.storage_bound(h, "e4m3", W, 0.05 * np.abs(h))


def test_finalize_bruteforce_via(fn=ref_moe_finalize):
    """out[t, h] = Σ_j y_slot[t·k + j, h], summed one element at a time in
    mpmath, with slot rows of very different magnitudes."""
    rng = np.random.default_rng(23)
    T, H, k = 3, 5, 3
    y = bf16_decode(bf16_encode_rne(rng.standard_normal((T * k, H)) * np.exp2(rng.integers(-6, 7, (T * k, 1)))))
    got = fn(y, k)
    assert got.shape == (T, H)
    for t in range(T):
        for h in range(H):
            want = mp.fsum(mp.mpf(float(y[t * k + j, h])) for j in range(k))
            assert got[t, h] == float(want), (t, h)


def test_finalize_identity_and_cancellation():
    rng = np.random.default_rng(24)
    y = bf16_decode(bf16_encode_rne(rng.standard_normal((4, 16))))
    np.testing.assert_array_equal(ref_moe_finalize(y, 1), y)            # k = 1: each slot is its token
    pair = np.concatenate([y[:, None, :], -y[:, None, :]], axis=1).reshape(8, 16)
    np.testing.assert_array_equal(ref_moe_finalize(pair, 2), np.zeros((4, 16)))
    with pytest.raises(ValueError):
        ref_moe_finalize(y[:3], 2)


def test_finalize_planted_stride_mistake_is_caught():
    """Slots read with the token-major stride swapped (row j·T + t instead of
    t·k + j) fail the brute-force pin."""
    def wrong_stride(y_slot, k):
        y = np.asarray(y_slot, dtype=np.float64)
        T = y.shape[0] // k
        return sum(y[j * T:(j + 1) * T] for j in range(k))
    with pytest.raises(AssertionError):
        test_finalize_bruteforce_via(wrong_stride)



# ---------------------------------------------------------------------------
# W8A8 (e4m3) MoE path. The brute force below rebuilds every storage step from
# the format definitions with exact rationals, sharing nothing with
# ``oracle.codecs`` or ``oracle.moe``'s quantiser: OCP e4m3fn values
# (−1)^s·2^(e−7)·(1 + f/8), subnormals 2^−6·f/8, largest finite 448, rounded
# to nearest with ties to the even code and saturated; bf16 values rounded to
# 8 significant bits, ties to even; the per-row scale fp32(amax/448) (1 for a
# zero row) and the quotient fp32(v/s) taken in fp32 (numpy float32
# arithmetic is IEEE binary32 with correct rounding), the precision in which
# the method takes those decisions.

from fractions import Fraction

_E4M3_POS = [Fraction(c & 7, 8) * Fraction(2) ** -6 if (c >> 3) == 0
             else (1 + Fraction(c & 7, 8)) * Fraction(2) ** ((c >> 3) - 7) for c in range(0x7F)]
assert _E4M3_POS[-1] == 448


def _frac(v):
    if isinstance(v, mp.mpf):
        man, exp = v.man_exp                      # |mantissa| and exponent; the sign is separate
        return (-1 if v < 0 else 1) * Fraction(int(man)) * Fraction(2) ** int(exp)
    return Fraction(float(v))


def _e4m3_round(v):
    """Nearest e4m3fn value to v (exact rational), ties to the even code,
    magnitudes past 448 saturated."""
    a = abs(_frac(v))
    sign = -1 if _frac(v) < 0 else 1
    if a >= 448:
        return sign * Fraction(448)
    lo = max(c for c in range(0x7F) if _E4M3_POS[c] <= a)
    if _E4M3_POS[lo] == a:
        return sign * a
    hi = lo + 1
    dl, dh = a - _E4M3_POS[lo], _E4M3_POS[hi] - a
    c = lo if dl < dh else hi if dh < dl else (lo if lo % 2 == 0 else hi)
    return sign * _E4M3_POS[c]


def _bf16_round(v):
    """Nearest bf16 value (8 significant bits, ties to even) to v, normal range."""
    a = abs(_frac(v))
    if a == 0:
        return Fraction(0)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    ulp = Fraction(2) ** (e - 7)
    q = a / ulp
    n = q.numerator // q.denominator
    r = q - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return (-1 if _frac(v) < 0 else 1) * n * ulp


def _row_quant(vals):
    """Per-row e4m3 storage of exact values that are fp32-representable:
    s = fp32(amax/448) (1 for a zero row), value_i = e4m3(fp32(v_i/s))·s."""
    f32 = [np.float32(float(v)) for v in vals]
    assert all(Fraction(float(a)) == _frac(v) for a, v in zip(f32, vals))   # exact in fp32
    amax = max(abs(a) for a in f32)
    s = np.float32(1.0) if amax == 0 else np.float32(amax) / np.float32(448.0)
    return [_e4m3_round(np.float32(a) / s) * Fraction(float(s)) for a in f32]


def _mp(fr):
    fr = Fraction(fr)
    return mp.mpf(fr.numerator) / fr.denominator


def _e4m3_decode_def(code):
    code = int(code)
    v = _E4M3_POS[code & 0x7F]
    return -v if code & 0x80 else v


def _mp_bruteforce_moe_w8a8(x, lg, gu_codes, gu_s, d_codes, d_s, k, alpha=1.702, limit=7.0):
    T, H = x.shape
    E = lg.shape[1]
    I = d_codes.shape[2]
    Wgu = [[[_mp(_e4m3_decode_def(gu_codes[e, n, c]) * Fraction(float(gu_s[e, n]))) for c in range(H)]
            for n in range(2 * I)] for e in range(E)]
    Wd = [[[_mp(_e4m3_decode_def(d_codes[e, n, i]) * Fraction(float(d_s[e, n]))) for i in range(I)]
           for n in range(H)] for e in range(E)]
    out = np.zeros((T, H))
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-lg[t, e], e))[:k]
        ex = [mp.exp(mp.mpf(float(lg[t, e]))) for e in order]
        den = mp.fsum(ex)
        xq = [_mp(v) for v in _row_quant([float(v) for v in x[t]])]
        acc = [mp.mpf(0)] * H
        for j, e in enumerate(order):
            G = [mp.fsum(xq[c] * Wgu[e][n][c] for c in range(H)) for n in range(2 * I)]
            hb = []
            for i in range(I):
                g = min(G[i], limit)
                u = min(max(G[I + i], -limit), limit)
                hb.append(_bf16_round((u + 1) * g / (1 + mp.exp(-mp.mpf(alpha) * g))))
            hq = [_mp(v) for v in _row_quant(hb)]
            for n in range(H):
                acc[n] += ex[j] / den * mp.fsum(hq[i] * Wd[e][n][i] for i in range(I))
        out[t] = [float(v) for v in acc]
    return out


def _w8a8_case():
    spec = MoeSpec("w8a8_pin", T=3, H=64, I=64, E=2, k=2, w_dtype="e4m3", w_std=0.15)
    act, w = make_moe_activations(spec, 5), make_moe_weights(spec, 5)
    x = bf16_decode(act["x"])
    lg = act["logits"].astype(np.float64)
    return spec, x, lg, w


def _w8a8_weights64(w):
    return lambda e: (e4m3_decode(w["w_gate_up"][e]) * w["s_gate_up"][e][:, None].astype(np.float64),
                      e4m3_decode(w["w_down"][e]) * w["s_down"][e][:, None].astype(np.float64))


_W8A8_WANT = {}


def test_moe_w8a8_bruteforce_token_order():
    """The W8A8 composition (tokens quantised per row, bf16 h quantised per
    slot row, e4m3 weights with per-row scales) against the definition-level
    brute force, through both oracle paths (plain and with the flip bound).
    The weight scales and the activation scales are all far from 1."""
    spec, x, lg, w = _w8a8_case()
    assert np.all(np.abs(np.log2(w["s_gate_up"])) > 4) and np.all(np.abs(np.log2(w["s_down"])) > 4)
    if "want" not in _W8A8_WANT:
        _W8A8_WANT["want"] = _mp_bruteforce_moe_w8a8(x, lg, w["w_gate_up"], w["s_gate_up"], w["w_down"],
                                                     w["s_down"], spec.k)
    want = _W8A8_WANT["want"]
    for bound in (False, True):
        got = ref_moe(x, lg, _w8a8_weights64(w), spec.k, storage="e4m3", act_quant=True,
                      with_bound=bound)["out"]
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12 * np.max(np.abs(want)))


def test_moe_w8a8_planted_mistakes_are_caught(monkeypatch):
    """A division in place of the multiplication by the row scale when the
    e4m3 codes are decoded, and h quantised straight from its exact value
    without the bf16 storage step, each fail the W8A8 brute-force pin."""
    def dequant_divides(codes, s):
        return e4m3_decode(codes) / np.asarray(s, dtype=np.float64)[..., None]

    def store_h_without_bf16(h, storage):
        if storage == "e4m3":
            q, s = ref_quant_rows_e4m3(h)
            return om._dequant_rows(q, s)
        return orig_store(h, storage)
    orig_store = om.store_h
    for name, fake in (("_dequant_rows", dequant_divides), ("store_h", store_h_without_bf16)):
        with monkeypatch.context() as m:
            m.setattr(om, name, fake)
            with pytest.raises(AssertionError):
                test_moe_w8a8_bruteforce_token_order()
