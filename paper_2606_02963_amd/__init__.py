"""MI355X (gfx950) fused GEMM + epilogue and MoE expert-FFN library.

The computation the generated kernels of arxiv 2606.02963 ("KForge")
accelerate — a dense GEMM with its tail ops fused into one kernel,
y = tail(x·Wᵀ + b), and the MoE expert grouped GEMM of an inference step —
implemented as hand-written HIP kernels behind a C ABI (``include/fgemm.h``).
``_lib`` is the ctypes binding of that ABI, ``api`` the torch-facing
wrappers, ``synth`` the seeded synthetic inputs, ``build`` the in-tree build.
"""

from . import _lib  # noqa: F401
