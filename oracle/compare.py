"""Comparison metric between a GPU result and the oracle (test infrastructure).

The paper's verification step accepts a candidate when it returns tensors of
the expected shape whose values match the reference within datatype-dependent
tolerances (§III-C, program verification; §V). The tolerances used here are
max relative error ≤ 1e-2 for bf16 inputs, ≤ 4e-2 for fp8 and ≤ 1e-4 for the
fp32 configuration.

"Relative error" is read as an RMS-floored elementwise error:

    rel_err(y, r) = max_i |y_i − r_i| / max(|r_i|, rms(r))

A plain elementwise relative error is undefined at the exact zeros that ReLU,
clamp and GELU(0) produce and explodes where GroupNorm's β cancels γ·n̂; the
floor at the RMS of the reference keeps the measure meaningful there while
staying elementwise for every entry of typical magnitude.
"""

from dataclasses import dataclass

import numpy as np

TOL = {"f32": 1e-4, "bf16": 1e-2, "e4m3": 4e-2}


def rel_err(y, r, slack=None):
    """RMS-floored max relative error. ``slack`` (optional, same shape):
    per-element absolute deviation that is known to be legitimate (a
    rounding decision either way is correct) and is subtracted first."""
    y = np.asarray(y, dtype=np.float64).ravel()
    r = np.asarray(r, dtype=np.float64).ravel()
    if y.shape != r.shape:
        raise ValueError(f"shape mismatch {y.shape} vs {r.shape}")
    if r.size == 0:
        return 0.0
    if not np.all(np.isfinite(y)):
        return float("inf")
    rms = float(np.sqrt(np.mean(r * r)))
    floor = np.maximum(np.abs(r), rms if rms > 0 else 1.0)
    d = np.abs(y - r)
    if slack is not None:
        d = np.maximum(d - np.asarray(slack, dtype=np.float64).ravel(), 0.0)
    return float(np.max(d / floor))


@dataclass
class ComparisonReport:
    rel_err: float
    normwise: float
    max_abs: float
    tol: float

    @property
    def ok(self):
        return self.rel_err <= self.tol

    def __str__(self):
        return (f"rel_err={self.rel_err:.3e} (tol {self.tol:.0e}) "
                f"normwise={self.normwise:.3e} max_abs={self.max_abs:.3e}")


def compare(y, r, dtype, slack=None):
    """Full report: the pass metric (after the optional legitimate-deviation
    slack) plus the normwise max|y−r|/max|r| (without it)."""
    y = np.asarray(y, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    if y.shape != r.shape:
        raise ValueError(f"shape mismatch {y.shape} vs {r.shape}")
    d = np.abs(y - r)
    mx = float(np.max(np.abs(r))) if r.size else 0.0
    max_abs = float(np.max(d)) if d.size else 0.0
    return ComparisonReport(rel_err(y, r, slack), max_abs / mx if mx else max_abs,
                            max_abs, TOL[dtype])


def count_above(y, r, dtype, slack=None):
    """Number of elements whose RMS-floored error, after the optional slack,
    exceeds the tolerance of ``dtype``."""
    y = np.asarray(y, dtype=np.float64).ravel()
    r = np.asarray(r, dtype=np.float64).ravel()
    if y.shape != r.shape:
        raise ValueError(f"shape mismatch {y.shape} vs {r.shape}")
    if r.size == 0:
        return 0
    if not np.all(np.isfinite(y)):
        return int(y.size)
    rms = float(np.sqrt(np.mean(r * r)))
    floor = np.maximum(np.abs(r), rms if rms > 0 else 1.0)
    d = np.abs(y - r)
    if slack is not None:
        d = np.maximum(d - np.asarray(slack, dtype=np.float64).ravel(), 0.0)
    return int(np.sum(d / floor > TOL[dtype]))
