"""Write ``oracle_small_cases.json``: small seeded inputs and the fp64 oracle's
outputs for every oracle entry point.

The paper prints no worked example, so these are not paper values: they are
a regression record of the oracle itself, written by this script, which calls
only ``oracle/`` (and numpy for the seeded draws). A later change to the
oracle's arithmetic shows up as a diff of this file, to be justified by the
passage of the paper (or the reading of it) that it follows.

Usage: python tests/golden/make_golden.py
"""

import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import (ref_add_rmsnorm, ref_bias_rope_kv_update, ref_fgemm, ref_moe,  # noqa: E402
                    ref_moe_finalize)

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_small_cases.json")


def hexlist(a):
    return [float(v).hex() for v in np.asarray(a, dtype=np.float64).ravel()]


def dyadic(rng, shape, scale=1.0):
    """Values k/64·scale with small integer k: exact in bf16 and fp64."""
    return rng.integers(-64, 65, shape).astype(np.float64) / 64.0 * scale


def cases():
    rng = np.random.default_rng(2606)
    out = []
    x, W, b = dyadic(rng, (4, 8)), dyadic(rng, (6, 8), 0.25), dyadic(rng, (6,), 0.25)
    for name, kw in [
        ("fgemm_gelu_clamp", dict(ops=(("scale", 0.5), ("gelu_tanh",), ("clamp", -1.0, 1.0)))),
        ("fgemm_mish_lrelu", dict(ops=(("mish",), ("leaky_relu", 0.1)))),
        ("fgemm_lse_mish", dict(ops=(("add", -0.25),), reduction="lse", post_ops=(("mish",),))),
        ("fgemm_silu_gn_swish", dict(ops=(("silu",),), reduction="groupnorm", gn_groups=2, gn_eps=1e-5,
                                     gamma=np.linspace(0.5, 1.5, 6), beta=np.linspace(-0.1, 0.1, 6),
                                     post_ops=(("silu",), ("scale", 1.5)))),
    ]:
        y = ref_fgemm(x, W, b, **kw)
        out.append({"fn": "ref_fgemm", "name": name, "inputs": {"x": hexlist(x), "W": hexlist(W), "b": hexlist(b)},
                    "shape": list(np.shape(y)), "out": hexlist(y)})
    T, H, I, E, k = 3, 8, 4, 4, 2
    xm, lg = dyadic(rng, (T, H)), dyadic(rng, (T, E))
    Wgu, Wd = dyadic(rng, (E, 2 * I, H), 0.25), dyadic(rng, (E, H, I), 0.25)
    r = ref_moe(xm, lg, (Wgu, Wd), k)
    out.append({"fn": "ref_moe", "name": "moe_T3_E4_k2", "inputs": {"x": hexlist(xm), "logits": hexlist(lg),
                "Wgu": hexlist(Wgu), "Wd": hexlist(Wd)}, "shape": [T, H], "out": hexlist(r["out"]),
                "idx": np.asarray(r["idx"]).ravel().tolist(), "perm": np.asarray(r["perm"]).ravel().tolist(),
                "offsets": np.asarray(r["offsets"]).ravel().tolist(), "w": hexlist(r["w"])})
    ys = dyadic(rng, (3 * 4, 8))
    out.append({"fn": "ref_moe_finalize", "name": "finalize_T3_k4", "inputs": {"y_slot": hexlist(ys)},
                "shape": [3, 8], "out": hexlist(ref_moe_finalize(ys, 4))})
    xn, rn, wn = dyadic(rng, (2, 8)), dyadic(rng, (2, 8), 4.0), 1.0 + dyadic(rng, (8,), 0.5)
    s, o = ref_add_rmsnorm(xn, rn, wn, 1e-5)
    out.append({"fn": "ref_add_rmsnorm", "name": "rmsnorm_T2_H8", "inputs": {"x": hexlist(xn), "r": hexlist(rn),
                "w": hexlist(wn)}, "shape": [2, 8], "out": hexlist(o), "s": hexlist(s)})
    nq, nkv, D, bs = 2, 1, 8, 4
    qkv, bias = dyadic(rng, (2, (nq + 2 * nkv) * D)), dyadic(rng, ((nq + 2 * nkv) * D,), 0.1)
    pos, table = np.array([5, 2]), np.array([[3, 1], [0, 2]])
    cache = np.zeros((4, 2, nkv, bs, D))
    q, c, _ = ref_bias_rope_kv_update(qkv, bias, pos, table, cache, nq, nkv, D, bs, 10000.0)
    out.append({"fn": "ref_bias_rope_kv_update", "name": "rope_T2", "inputs": {"qkv": hexlist(qkv),
                "bias": hexlist(bias), "positions": pos.tolist(), "block_table": table.ravel().tolist()},
                "shape": [2, nq, D], "out": hexlist(q), "cache": hexlist(c)})
    return out


if __name__ == "__main__":
    with open(OUT, "w") as fh:
        json.dump({"source": "tests/golden/make_golden.py (fp64 oracle, seed 2606)", "cases": cases()}, fh,
                  indent=0)
    print("wrote", OUT)
