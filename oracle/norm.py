"""fp64 oracle for the fused residual add + RMSNorm of the gpt-oss-20b decode
path (paper §IV-A, "Fused Add + RMSNorm" in Table I).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The step adds a layer's output to the residual stream and normalises the sum
with RMSNorm (root-mean-square layer normalisation: divide by the RMS of the
row, then scale per channel by a learned weight):

  s        = x + residual                         (the new residual stream)
  rms      = sqrt(mean_h s[h]² + eps)
  out[h]   = s[h] / rms · weight[h]

Storage (the method's declared formats, modelled here by the caller): the
updated residual is stored as bf16 (RNE of s) and out as bf16; the
statistics and the normalisation use s itself, before that rounding. With
bf16 inputs s is exact in fp64.
"""

import numpy as np


def ref_add_rmsnorm(x, residual, weight, eps=1e-5):
    """x, residual [T, H], weight [H] (fp64 values of the stored inputs).
    Returns (s, out): the new residual stream s = x + residual and the
    normalised rows, both [T, H] fp64, before any storage rounding."""
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(residual, dtype=np.float64)
    w = np.asarray(weight, dtype=np.float64)
    s = x + r
    rms = np.sqrt(np.mean(s * s, axis=1, keepdims=True) + eps)
    return s, s / rms * w[None, :]
