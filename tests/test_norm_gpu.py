"""GPU parity of the fused residual add + RMSNorm (paper §IV-A, Table I)
against the fp64 oracle.

The updated residual must equal the bf16 rounding of the exact sum bit for
bit (a sum of two bf16 values is exact in fp32 at these magnitudes); each
output must be one of the two bf16 neighbours of the exact normalised value
(the kernel evaluates in fp32, so it may round either way only inside the
fp32 noise of a midpoint) and the rows must pass the bf16 tolerance. Covers
the Table I batch sizes at H = 2880, the narrowest and widest rows, odd
batch sizes, a row that cancels to zero, eps = 0, and the error paths."""

import numpy as np
import pytest
import torch

from oracle import bf16_decode, bf16_encode_rne, compare, ref_add_rmsnorm
from paper_2606_02963_amd import _lib as L
from paper_2606_02963_amd import api
from paper_2606_02963_amd.synth import FINALIZE_BATCHES, NORM_H, make_norm_inputs
from tests.gpu_helpers import dev_bf16, log, require_gpu

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.cpu().view(torch.int16).numpy().view(np.uint16)


def _neighbours_ok(got_bits, want):
    """Every output lies within one bf16 spacing of the exact value (so it is
    one of its two bf16 neighbours); exact zeros stay zero."""
    got = bf16_decode(got_bits)
    nz = want != 0
    spacing = np.exp2(np.floor(np.log2(np.abs(want[nz]))) - 7)
    return bool(np.all(np.abs(got[nz] - want[nz]) <= spacing) and np.all(got[~nz] == 0))


def _run(x, r, w, eps):
    xd, rd, wd = dev_bf16(x), dev_bf16(r), dev_bf16(w)
    out = api.add_rmsnorm(xd, rd, wd, eps)
    torch.cuda.synchronize()
    return _bits(rd), _bits(out)


def _check(x, r, w, eps):
    res_bits, out_bits = _run(x, r, w, eps)
    s, want = ref_add_rmsnorm(bf16_decode(x), bf16_decode(r), bf16_decode(w), eps)
    assert np.array_equal(res_bits, bf16_encode_rne(s)), "residual differs from RNE(x + residual)"
    assert _neighbours_ok(out_bits, want), "an output is not a bf16 neighbour of the exact value"
    rep = compare(bf16_decode(out_bits), want, "bf16")
    log(f"    {rep}")
    assert rep.ok, rep
    return out_bits, want


@pytest.mark.parametrize("T", FINALIZE_BATCHES)
def test_add_rmsnorm_table_i_batches(T):
    require_gpu()
    log(f"[add_rmsnorm] T={T} H={NORM_H}")
    x, r, w = make_norm_inputs(T, seed=1)
    _check(x, r, w, 1e-5)


@pytest.mark.parametrize("T,H,eps,zero_row", [(1, 8, 1e-5, False), (5, 4096, 1e-6, True),
                                              (3, 136, 0.0, False), (9, 2880, 1e-2, True),
                                              (20000, 512, 1e-5, True)])      # a prefill-sized grid
def test_add_rmsnorm_edge_shapes(T, H, eps, zero_row):
    require_gpu()
    log(f"[add_rmsnorm] T={T} H={H} eps={eps} zero_row={zero_row}")
    x, r, w = make_norm_inputs(T, H, seed=2)
    if zero_row:
        r[1] = x[1] ^ np.uint16(0x8000)          # row 1 cancels: x + r = 0 exactly
    out_bits, _ = _check(x, r, w, eps)
    if zero_row:
        assert not bf16_decode(out_bits[1]).any()


def test_add_rmsnorm_errors_and_empty():
    require_gpu()
    t = torch.zeros((2, 16), dtype=torch.bfloat16, device="cuda")
    w = torch.ones(16, dtype=torch.bfloat16, device="cuda")
    p = t.data_ptr()
    L.add_rmsnorm(p, p, w.data_ptr(), p, 0, 16, 1e-5, None)                  # T = 0: nothing enqueued
    for args, status in [((2, 12, 1e-5), L.FG_ERR_ALIGNMENT),
                         ((2, 4104, 1e-5), L.FG_ERR_UNSUPPORTED),
                         ((2, 16, -1.0), L.FG_ERR_INVALID_ARG),
                         ((2, 16, float("nan")), L.FG_ERR_INVALID_ARG),
                         ((-1, 16, 1e-5), L.FG_ERR_INVALID_ARG)]:
        with pytest.raises(L.FgError) as ei:
            L.add_rmsnorm(p, p, w.data_ptr(), p, *args, None)
        assert ei.value.status == status
    with pytest.raises(L.FgError) as ei:
        L.add_rmsnorm(p + 2, p, w.data_ptr(), p, 2, 16, 1e-5, None)
    assert ei.value.status == L.FG_ERR_ALIGNMENT
