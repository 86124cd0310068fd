"""Pins for the fused GEMM + tail oracle (``oracle.fgemm``).

Each part is pinned by something other than itself: 50-digit mpmath brute
force on tiny shapes (bf16 inputs are dyadic rationals, so every product is
exact), closed forms (identity and zero weights, GELU(0) = 0, the odd-part
identities of GELU and SiLU, LSE of a constant row), invariants (LSE shift
and permutation invariance and its bounds, GroupNorm's per-group moments) and
library special cases (torch CPU float64 gelu / silu / group_norm /
logsumexp). ``test_pins_catch_planted_mistakes`` plants plausible mistakes in
the oracle and checks that a pin fails for each."""

import math

import mpmath as mp
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle.fgemm as of
from oracle.codecs import bf16_decode
from oracle.fgemm import ref_fgemm
from paper_2606_02963_amd.synth import FGEMM_SPECS, make_fgemm_inputs, to_bf16_bits

mp.mp.dps = 50


# ---------------------------------------------------------------- brute force

def _mp_gelu(u):
    return mp.mpf(0.5) * u * (1 + mp.tanh(mp.sqrt(2 / mp.pi) * (u + mp.mpf("0.044715") * u ** 3)))


def _mp_silu(u):
    return u / (1 + mp.exp(-u))


def _mp_apply(u, op):
    kind = op[0]
    if kind == "scale":
        return u * mp.mpf(op[1])
    if kind == "add":
        return u + mp.mpf(op[1])
    if kind == "relu":
        return u if u > 0 else mp.mpf(0)
    if kind == "gelu_tanh":
        return _mp_gelu(u)
    if kind == "silu":
        return _mp_silu(u)
    if kind == "clamp":
        return min(max(u, mp.mpf(op[1])), mp.mpf(op[2]))
    if kind == "mish":
        return u * mp.tanh(mp.log(1 + mp.exp(u)))
    if kind == "leaky_relu":
        return u if u >= 0 else mp.mpf(op[1]) * u
    raise ValueError(kind)


def _mp_fgemm(x, W, b, ops, reduction=None, groups=0, eps=1e-5, gamma=None, beta=None, post_ops=()):
    M, K = x.shape
    N = W.shape[0]
    z = [[mp.fsum(mp.mpf(float(x[m, k])) * mp.mpf(float(W[n, k])) for k in range(K))
          + mp.mpf(float(b[n])) for n in range(N)] for m in range(M)]
    for op in ops:
        z = [[_mp_apply(v, op) for v in row] for row in z]
    if reduction == "lse":
        out = [mp.log(mp.fsum(mp.exp(v) for v in row)) for row in z]
        for op in post_ops:
            out = [_mp_apply(v, op) for v in out]
        return out
    if reduction == "groupnorm":
        gs = N // groups
        out = []
        for row in z:
            r = []
            for g in range(groups):
                seg = row[g * gs:(g + 1) * gs]
                mu = mp.fsum(seg) / gs
                var = mp.fsum((v - mu) ** 2 for v in seg) / gs
                for i, v in enumerate(seg):
                    n = g * gs + i
                    y = ((v - mu) / mp.sqrt(var + mp.mpf(eps)) * mp.mpf(float(gamma[n]))
                         + mp.mpf(float(beta[n])))
                    for op in post_ops:
                        y = _mp_apply(y, op)
                    r.append(y)
            out.append(r)
        return out
    return z


def _tiny_bf16(M, N, K, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    x = bf16_decode(to_bf16_bits(rng.standard_normal((M, K)).astype(np.float32) * scale))
    W = bf16_decode(to_bf16_bits(rng.standard_normal((N, K)).astype(np.float32) * 0.3))
    b = rng.standard_normal(N).astype(np.float32).astype(np.float64) * 0.1
    return x, W, b


TAILS = [
    ((("relu",), ("scale", 2.0)), None),
    ((("scale", 0.5), ("gelu_tanh",), ("clamp", -1.0, 1.0)), None),
    ((("add", -0.25),), "lse"),
    ((("silu",),), "groupnorm"),
    ((("gelu_tanh",), ("silu",), ("scale", -1.5), ("add", 0.125)), None),
]


@pytest.mark.parametrize("ops,red", TAILS)
def test_bruteforce_mpmath(ops, red):
    x, W, b = _tiny_bf16(3, 8, 8, seed=len(ops))
    kw = {}
    if red == "groupnorm":
        rng = np.random.default_rng(9)
        kw = dict(gn_groups=2, gn_eps=1e-5, gamma=rng.random(8) + 0.5,
                  beta=rng.standard_normal(8) * 0.1)
    got = ref_fgemm(x, W, b, ops, red, **kw)
    want = _mp_fgemm(x, W, b, ops, red, kw.get("gn_groups", 0), 1e-5,
                     kw.get("gamma"), kw.get("beta"))
    want = np.array([[float(v) for v in r] for r in want]) if red != "lse" \
        else np.array([float(v) for v in want])
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-14)


# Table III tail patterns: elementwise ops before and after the reduction
POST_TAILS = [
    ((("scale", 0.5),), "lse", (("mish",),)),                                     # Scale → LSE → Mish
    ((), "groupnorm", (("silu",), ("scale", 1.5), ("silu",))),                    # GN → Swish → Mul → Swish
    ((), "groupnorm", (("leaky_relu", 0.01), ("scale", 2.0))),                    # GN → LReLU → Sum
    ((("silu",), ("add", 0.25)), "groupnorm", ()),                                # Swish → Sum → GN
    ((("mish",), ("leaky_relu", 0.2)), None, ()),
]


@pytest.mark.parametrize("ops,red,post", POST_TAILS)
def test_bruteforce_mpmath_post_ops(ops, red, post):
    x, W, b = _tiny_bf16(3, 8, 8, seed=11 + len(ops) + len(post), scale=2.0)
    kw = {}
    if red == "groupnorm":
        rng = np.random.default_rng(10)
        kw = dict(gn_groups=2, gn_eps=1e-5, gamma=rng.random(8) + 0.5, beta=rng.standard_normal(8) * 0.1)
    got = ref_fgemm(x, W, b, ops, red, post_ops=post, **kw)
    want = _mp_fgemm(x, W, b, ops, red, kw.get("gn_groups", 0), 1e-5, kw.get("gamma"), kw.get("beta"), post)
    want = np.array([[float(v) for v in r] for r in want]) if red != "lse" \
        else np.array([float(v) for v in want])
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-14)


def test_mish_and_leaky_relu_closed_forms_and_torch():
    u = torch.linspace(-30, 30, 6001, dtype=torch.float64)
    un = u.numpy()
    np.testing.assert_allclose(of.apply_op(un, ("mish",)), F.mish(u).numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(of.apply_op(un, ("leaky_relu", 0.01)),
                                  F.leaky_relu(u, 0.01).numpy())
    assert of.apply_op(np.array([0.0]), ("mish",))[0] == 0.0
    big = np.array([40.0, 700.0])
    np.testing.assert_array_equal(of.apply_op(big, ("mish",)), big)            # tanh(softplus) = 1 in fp64
    # slope: f(-t) = -a·t, f(t) = t
    t = np.array([0.5, 3.0])
    np.testing.assert_array_equal(of.apply_op(-t, ("leaky_relu", 0.25)), -0.25 * t)
    np.testing.assert_array_equal(of.apply_op(t, ("leaky_relu", 0.25)), t)
    with pytest.raises(ValueError):
        ref_fgemm(np.eye(2), np.eye(2), None, (), None, post_ops=(("relu",),))


# ---------------------------------------------------------------- closed forms

def test_identity_weight_reproduces_tail_of_x_plus_b():
    rng = np.random.default_rng(3)
    K = 16
    x = rng.standard_normal((5, K))
    b = rng.standard_normal(K)
    ops = (("scale", 0.5), ("gelu_tanh",), ("clamp", -1.0, 1.0))
    got = ref_fgemm(x, np.eye(K), b, ops)
    u = (x + b) * 0.5
    want = np.clip(0.5 * u * (1 + np.tanh(math.sqrt(2 / math.pi) * (u + 0.044715 * u ** 3))), -1, 1)
    np.testing.assert_array_equal(got, want)


def test_zero_weight_gives_tail_of_bias():
    b = np.linspace(-3, 3, 12)
    got = ref_fgemm(np.ones((4, 7)), np.zeros((12, 7)), b, (("relu",), ("scale", 2.0)))
    np.testing.assert_array_equal(got, np.tile(np.maximum(b, 0) * 2, (4, 1)))


def test_gelu_and_silu_closed_forms():
    u = np.linspace(-9, 9, 1001)
    g = of.apply_op(u, ("gelu_tanh",))
    s = of.apply_op(u, ("silu",))
    assert of.apply_op(np.array([0.0]), ("gelu_tanh",))[0] == 0.0
    assert of.apply_op(np.array([0.0]), ("silu",))[0] == 0.0
    # tanh and the logistic are odd around 0 / ½: f(u) − f(−u) = u exactly in real arithmetic
    np.testing.assert_allclose(g - g[::-1], u, atol=1e-14)
    np.testing.assert_allclose(s - s[::-1], u, atol=1e-14)
    # limits
    big = np.array([30.0, -30.0])
    np.testing.assert_allclose(of.apply_op(big, ("gelu_tanh",)), [30.0, 0.0], atol=1e-12)
    np.testing.assert_allclose(of.apply_op(big, ("silu",)), [30.0, -30 * math.exp(-30)], rtol=1e-12)
    assert np.all(np.isfinite(of.apply_op(np.array([-800.0, 800.0]), ("silu",))))


def test_elementwise_ops_match_torch_float64():
    u = torch.linspace(-12, 12, 4097, dtype=torch.float64)
    un = u.numpy()
    np.testing.assert_allclose(of.apply_op(un, ("gelu_tanh",)),
                               F.gelu(u, approximate="tanh").numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(of.apply_op(un, ("silu",)), F.silu(u).numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(of.apply_op(un, ("clamp", -1.0, 1.0)), u.clamp(-1, 1).numpy())
    np.testing.assert_array_equal(of.apply_op(un, ("relu",)), F.relu(u).numpy())


def test_op_order_is_respected():
    z = np.array([[2.0]])
    a = ref_fgemm(np.eye(1), np.eye(1), None, (("scale", 3.0), ("add", 1.0)))
    b_ = ref_fgemm(np.eye(1), np.eye(1), None, (("add", 1.0), ("scale", 3.0)))
    assert a[0, 0] == 4.0 and b_[0, 0] == 6.0 and z.shape == (1, 1)


# ---------------------------------------------------------------- LogSumExp

def test_lse_constant_row_is_c_plus_ln_n():
    N = 8192
    c = 0.7
    # W = 0 and b = c: every column of row m is c − 0.25
    got = ref_fgemm(np.ones((3, 8)), np.zeros((N, 8)), np.full(N, c), (("add", -0.25),), "lse")
    np.testing.assert_allclose(got, c - 0.25 + math.log(N), rtol=0, atol=1e-13)


def test_lse_invariants_and_torch():
    rng = np.random.default_rng(4)
    z = rng.standard_normal((6, 300)) * 5
    l = of.row_logsumexp(z)
    np.testing.assert_allclose(of.row_logsumexp(z + 3.25), l + 3.25, atol=1e-12)
    np.testing.assert_allclose(of.row_logsumexp(z[:, rng.permutation(300)]), l, atol=1e-12)
    assert np.all(z.max(1) <= l) and np.all(l <= z.max(1) + math.log(300))
    np.testing.assert_allclose(l, torch.logsumexp(torch.from_numpy(z), 1).numpy(), rtol=1e-14)
    # no overflow for huge values
    assert np.isfinite(of.row_logsumexp(np.array([[1000.0, 999.0]])))[0]


def test_lse_tile_split_combine_equals_direct():
    """The two-pass form used on the GPU — per tile j (m_j, s_j = Σ e^(z−m_j)),
    then m = max m_j, S = Σ s_j e^(m_j − m), LSE = m + ln S — is the same
    function as the direct definition for every tile width."""
    rng = np.random.default_rng(5)
    z = rng.standard_normal((4, 8192)) * 3
    direct = of.row_logsumexp(z)
    for bn in (64, 128, 256, 1000, 8192):
        parts = [z[:, i:i + bn] for i in range(0, z.shape[1], bn)]
        m_j = np.stack([p.max(1) for p in parts], 1)
        s_j = np.stack([np.exp(p - p.max(1, keepdims=True)).sum(1) for p in parts], 1)
        m = m_j.max(1, keepdims=True)
        lse = m[:, 0] + np.log((s_j * np.exp(m_j - m)).sum(1))
        np.testing.assert_allclose(lse, direct, rtol=1e-15, atol=1e-13)


# ---------------------------------------------------------------- GroupNorm

def test_groupnorm_moments_with_unit_affine():
    rng = np.random.default_rng(6)
    z = rng.standard_normal((5, 4096)) * 0.3 + 0.1
    eps = 1e-5
    y = of.group_norm(z, 32, eps, np.ones(4096), np.zeros(4096))
    yg = y.reshape(5, 32, 128)
    zg = z.reshape(5, 32, 128)
    var_z = zg.var(axis=-1)
    np.testing.assert_allclose(yg.mean(-1), 0, atol=1e-14)
    # biased variance after normalisation is σ²/(σ²+eps), exactly 1 only at eps = 0
    np.testing.assert_allclose(yg.var(-1), var_z / (var_z + eps), rtol=1e-12)
    y0 = of.group_norm(z, 32, 0.0, np.ones(4096), np.zeros(4096)).reshape(5, 32, 128)
    np.testing.assert_allclose(y0.var(-1), 1.0, rtol=1e-12)


def test_groupnorm_affine_invariance_and_torch():
    rng = np.random.default_rng(7)
    z = rng.standard_normal((3, 512))
    gamma = rng.random(512) + 0.5
    beta = rng.standard_normal(512) * 0.1
    y = of.group_norm(z, 4, 0.0, gamma, beta)
    a = np.repeat(rng.random(4) * 3 + 0.1, 128)      # positive per-group scale
    c = np.repeat(rng.standard_normal(4), 128)        # per-group shift
    np.testing.assert_allclose(of.group_norm(z * a + c, 4, 0.0, gamma, beta), y, atol=1e-12)
    ref = F.group_norm(torch.from_numpy(z), 4, torch.from_numpy(gamma), torch.from_numpy(beta), eps=1e-5)
    np.testing.assert_allclose(of.group_norm(z, 4, 1e-5, gamma, beta), ref.numpy(), rtol=1e-12, atol=1e-13)


def test_full_tail_c4_small_matches_torch_pipeline():
    spec = FGEMM_SPECS["bf16_silu_gn"].scaled(M=16, N=512, K=64)
    inp = make_fgemm_inputs(spec, seed=0)
    x, W = bf16_decode(inp["x"]), bf16_decode(inp["W"])
    b, g, be = (inp[k].astype(np.float64) for k in ("b", "gamma", "beta"))
    got = ref_fgemm(x, W, b, spec.ops, "groupnorm", spec.gn_groups, 1e-5, g, be)
    z = F.silu(torch.from_numpy(x) @ torch.from_numpy(W).T + torch.from_numpy(b))
    ref = F.group_norm(z, spec.gn_groups, torch.from_numpy(g), torch.from_numpy(be), eps=1e-5)
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-11, atol=1e-12)


# ---------------------------------------------------------------- planted mistakes

def _pins_pass():
    for ops, red in TAILS:
        test_bruteforce_mpmath(ops, red)
    test_identity_weight_reproduces_tail_of_x_plus_b()
    test_gelu_and_silu_closed_forms()
    test_elementwise_ops_match_torch_float64()
    test_lse_constant_row_is_c_plus_ln_n()
    test_lse_invariants_and_torch()
    test_groupnorm_moments_with_unit_affine()
    test_groupnorm_affine_invariance_and_torch()
    for ops, red, post in POST_TAILS:
        test_bruteforce_mpmath_post_ops(ops, red, post)
    test_mish_and_leaky_relu_closed_forms_and_torch()


# the planted LogSumExp without its max shift overflows by design
@pytest.mark.filterwarnings("ignore:overflow encountered:RuntimeWarning")
def test_pins_catch_planted_mistakes(monkeypatch):
    """Plant plausible mistakes in the oracle (on the CPU) and require that
    at least one pin fails for each: a wrong GELU constant, a dropped
    max-shift in LSE, unbiased variance in GroupNorm, eps outside the sqrt,
    Mish with ReLU in place of softplus, post-reduction ops applied before
    the reduction, and a transposed weight operand."""
    good_gelu = of._gelu_tanh
    mutants = {
        "gelu_const": ("_gelu_tanh", lambda u: 0.5 * u * (1 + np.tanh(of._SQRT_2_OVER_PI * (u + 0.0447 * u ** 3)))),
        "gelu_sign": ("_gelu_tanh", lambda u: 0.5 * u * (1 - np.tanh(of._SQRT_2_OVER_PI * (u + 0.044715 * u ** 3)))),
        "lse_no_shift": ("row_logsumexp", lambda z: np.log(np.sum(np.exp(np.minimum(z, 700.0)) * np.exp(np.maximum(z - 700.0, 0.0)), axis=-1))),
        "lse_log2": ("row_logsumexp", lambda z: z.max(-1) + np.log2(np.sum(np.exp(z - z.max(-1, keepdims=True)), -1))),
        "gn_unbiased": ("group_norm", lambda z, G, eps, g, b: (
            ((z.reshape(z.shape[0], G, -1) - z.reshape(z.shape[0], G, -1).mean(-1, keepdims=True))
             / np.sqrt(z.reshape(z.shape[0], G, -1).var(-1, ddof=1, keepdims=True) + eps)).reshape(z.shape) * g + b)),
        "gn_eps_outside": ("group_norm", lambda z, G, eps, g, b: (
            ((z.reshape(z.shape[0], G, -1) - z.reshape(z.shape[0], G, -1).mean(-1, keepdims=True))
             / (np.sqrt(z.reshape(z.shape[0], G, -1).var(-1, keepdims=True)) + eps)).reshape(z.shape) * g + b)),
        "silu_sign": ("_silu", lambda u: u / (1 + np.exp(u))),
        "mish_relu_softplus": ("_mish", lambda u: u * np.tanh(np.maximum(u, 0.0))),
    }
    assert good_gelu is of._gelu_tanh
    for name, (attr, fn) in mutants.items():
        with monkeypatch.context() as m:
            m.setattr(of, attr, fn)
            with pytest.raises(AssertionError):
                _pins_pass()
    # post ops applied before the reduction instead of after it
    good_ref = of.ref_fgemm

    def post_before(x, W, b=None, ops=(), reduction=None, post_ops=(), **kw):
        return good_ref(x, W, b, tuple(ops) + tuple(post_ops), reduction, **kw)
    with monkeypatch.context() as m:
        m.setattr(of, "ref_fgemm", post_before)
        with pytest.raises(AssertionError):
            for ops, red, post in POST_TAILS[:3]:
                x, W, b = _tiny_bf16(3, 8, 8, seed=11 + len(ops) + len(post), scale=2.0)
                kw = {}
                if red == "groupnorm":
                    rng = np.random.default_rng(10)
                    kw = dict(gn_groups=2, gn_eps=1e-5, gamma=rng.random(8) + 0.5, beta=rng.standard_normal(8) * 0.1)
                got = of.ref_fgemm(x, W, b, ops, red, post_ops=post, **kw)
                want = _mp_fgemm(x, W, b, ops, red, kw.get("gn_groups", 0), 1e-5, kw.get("gamma"),
                                 kw.get("beta"), post)
                want = np.array([[float(v) for v in r] for r in want]) if red != "lse" \
                    else np.array([float(v) for v in want])
                np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-14)
    # transposed operand (x·W instead of x·Wᵀ, square W): the brute force disagrees
    x, W, b = _tiny_bf16(3, 8, 8, seed=1)
    bad = ref_fgemm(x, W.T, b, TAILS[0][0])
    want = np.array([[float(v) for v in r] for r in _mp_fgemm(x, W, b, TAILS[0][0])])
    assert not np.allclose(bad, want, rtol=1e-13, atol=1e-14)
