"""Pins for the fused residual add + RMSNorm oracle (``oracle.norm``).

Against an mpmath brute force of the definition (sum, mean of squares, square
root, divide, scale), and closed forms: a constant row c gives
c/sqrt(c² + eps)·w; with eps = 0 and w = 1 the result is invariant under
scaling the row and every output row has RMS exactly 1; a zero row gives
zero. Planted mistakes (sum instead of mean, eps dropped, weight not applied,
residual not added) fail a pin."""

import mpmath as mp
import numpy as np
import pytest

import oracle.norm as on
from oracle.codecs import bf16_decode, bf16_encode_rne
from oracle.norm import ref_add_rmsnorm

mp.mp.dps = 50


def _bf16(a):
    return bf16_decode(bf16_encode_rne(np.asarray(a, dtype=np.float64)))


def test_add_rmsnorm_bruteforce_via(fn=ref_add_rmsnorm):
    rng = np.random.default_rng(31)
    T, H, eps = 3, 7, 1e-5
    x = _bf16(rng.standard_normal((T, H)))
    r = _bf16(rng.standard_normal((T, H)) * 4)
    w = _bf16(rng.uniform(0.5, 1.5, H))
    s, out = fn(x, r, w, eps)
    for t in range(T):
        st = [mp.mpf(float(x[t, h])) + mp.mpf(float(r[t, h])) for h in range(H)]
        rms = mp.sqrt(mp.fsum(v * v for v in st) / H + mp.mpf(eps))
        for h in range(H):
            assert s[t, h] == float(st[h])
            assert abs(out[t, h] - float(st[h] / rms * mp.mpf(float(w[h])))) <= 1e-15 * abs(out[t, h]) + 1e-300


def test_add_rmsnorm_closed_forms():
    H = 64
    w = _bf16(np.linspace(0.5, 2.0, H))
    for c, eps in ((3.0, 1e-5), (-0.25, 1e-6), (1e-3, 1e-5)):
        x = np.full((1, H), c / 2)
        _, out = ref_add_rmsnorm(x, x, w, eps)
        np.testing.assert_allclose(out[0], c / np.sqrt(c * c + eps) * w, rtol=1e-15)
    rng = np.random.default_rng(32)
    x, r = rng.standard_normal((4, H)), rng.standard_normal((4, H))
    _, o1 = ref_add_rmsnorm(x, r, np.ones(H), 0.0)
    _, o2 = ref_add_rmsnorm(8 * x, 8 * r, np.ones(H), 0.0)
    np.testing.assert_allclose(o1, o2, rtol=1e-14)
    np.testing.assert_allclose(np.sqrt(np.mean(o1 * o1, axis=1)), 1.0, rtol=1e-14)
    s, out = ref_add_rmsnorm(x, -x, w, 1e-5)
    assert not s.any() and not out.any()


def test_add_rmsnorm_planted_mistakes_are_caught(monkeypatch):
    def sum_not_mean(x, residual, weight, eps=1e-5):
        s = np.asarray(x, float) + np.asarray(residual, float)
        return s, s / np.sqrt(np.sum(s * s, axis=1, keepdims=True) + eps) * np.asarray(weight)[None, :]

    def no_eps(x, residual, weight, eps=1e-5):
        s = np.asarray(x, float) + np.asarray(residual, float)
        return s, s / np.sqrt(np.mean(s * s, axis=1, keepdims=True)) * np.asarray(weight)[None, :]

    def no_weight(x, residual, weight, eps=1e-5):
        s = np.asarray(x, float) + np.asarray(residual, float)
        return s, s / np.sqrt(np.mean(s * s, axis=1, keepdims=True) + eps)

    def no_residual(x, residual, weight, eps=1e-5):
        return ref_add_rmsnorm(x, np.zeros_like(np.asarray(x, float)), weight, eps)

    for bad in (sum_not_mean, no_weight, no_residual):
        with pytest.raises(AssertionError):
            test_add_rmsnorm_bruteforce_via(bad)
    # eps matters only for small rows: the closed form with c = 1e-3 catches it
    with monkeypatch.context() as m:
        m.setattr(on, "ref_add_rmsnorm", no_eps)
        with pytest.raises(AssertionError):
            H = 8
            w = np.ones(H)
            x = np.full((1, H), 0.5e-3)
            _, out = on.ref_add_rmsnorm(x, x, w, 1e-5)
            np.testing.assert_allclose(out[0], 1e-3 / np.sqrt(1e-6 + 1e-5) * w, rtol=1e-12)
