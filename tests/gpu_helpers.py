"""Shared helpers of the GPU parity tests: move seeded inputs to the device,
run the library, bring results back as fp64 for the oracle comparison."""

import numpy as np
import torch

from oracle import bf16_decode
from oracle.compare import compare, count_above


def require_gpu():
    import pytest
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def dev_bf16(bits):
    """uint16 bf16 bit patterns -> device bfloat16 tensor (same bits)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).cuda()


def dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def dev_u8(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).cuda()


def host64(t):
    """Device tensor -> fp64 numpy (bf16 decoded exactly)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return bf16_decode(t.view(torch.int16).numpy().view(np.uint16))
    return t.numpy().astype(np.float64)


def log(msg):
    print(msg, flush=True)


# share of output elements that may exceed the tolerance after the narrow
# bound (h within fp32 evaluation noise): the rare storage decisions that the
# e4m3 MFMA's accumulation noise moves further
NARROW_EXCESS = 1e-4


def check_moe_outputs(got, ref, dtype, label=""):
    """MoE step outputs against ref_moe(..., with_bound=True): every element
    within the tolerance after the full legitimate-deviation bound, the
    normwise error within it without any bound, and at most NARROW_EXCESS of
    the elements beyond it after the narrow bound."""
    rep = compare(got, ref["out"], dtype, slack=ref["out_bound"])
    over = count_above(got, ref["out"], dtype, slack=ref["out_bound_narrow"])
    log(f"    {label}{rep}; beyond the tolerance after the narrow bound: {over} of {np.size(got)}")
    assert rep.ok and rep.normwise <= rep.tol and over <= NARROW_EXCESS * np.size(got), f"{label}{rep}, {over} over"
    return rep
