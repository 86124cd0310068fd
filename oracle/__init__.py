"""Plain fp64 CPU oracle for the fused GEMM + tail path and the MoE expert FFN.

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it. It shares no code, tables or
helpers with the HIP library; the two meet only in the seeded input
generators (``paper_2606_02963_amd/synth.py``), which hold none of the
method's arithmetic.

What it computes (paper §IV-B, "Triton kernels on Intel Arc B580"): the
generated kernels fuse the post-GEMM sequence of a GEMM + tail-ops problem
into one pass with fp32 accumulation and post-processing; fusion reschedules
the same operations, so the result it must reach is the plain definition
y = tail(x·Wᵀ + b), here evaluated in fp64 on the exact values the GPU reads.
The MoE expert FFN (paper §IV-A, the gpt-oss-20b decode path: MoE finalize,
and the MoE-MLP block named as future work in §V) is written out step by step
in the order routing → permutation → grouped gate/up GEMM → clamped SwiGLU →
grouped down GEMM → routing-weighted finalize. The other two decode kernels
of Table I are here too: the fused residual add + RMSNorm (``norm``) and the
QKV bias + rotary embedding + KV-cache update (``rope``).

Every function is pinned by tests in ``tests/test_oracle_*.py`` against closed
forms, invariants, brute force (mpmath) and library special cases; none is
"parity unpinned".
"""

from .codecs import (bf16_decode, bf16_encode_rne, e4m3_decode,
                     e4m3_encode_rne_sat, f32_round)
from .fgemm import ref_fgemm, OPS
from .moe import ref_route, ref_permute, ref_swiglu_clamped, ref_moe, ref_moe_finalize, ref_quant_rows_e4m3
from .norm import ref_add_rmsnorm
from .rope import ref_rope, ref_bias_rope_kv_update
from .compare import rel_err, ComparisonReport, compare

__all__ = [
    "bf16_decode", "bf16_encode_rne", "e4m3_decode", "e4m3_encode_rne_sat",
    "f32_round", "ref_fgemm", "OPS", "ref_route", "ref_permute",
    "ref_swiglu_clamped", "ref_moe", "ref_moe_finalize", "ref_quant_rows_e4m3", "ref_add_rmsnorm",
    "ref_rope", "ref_bias_rope_kv_update", "rel_err",
    "ComparisonReport", "compare",
]
