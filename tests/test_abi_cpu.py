"""Host-side checks of the C ABI (no GPU needed).

The library loads without a GPU, exports every function ``include/fgemm.h``
declares, and its validation rejects bad requests with the documented status
before any HIP call: fgemm_plan is host-only, and fgemm_run /
moe_grouped_ffn / fg_quantize_rows_e4m3 return on invalid arguments before
enqueueing anything."""

import ctypes as C
import os
import re

import pytest

from paper_2606_02963_amd import _lib as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "fgemm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_]\w*\s*\**\s*([A-Za-z_]\w*)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "while")))


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("fgemm_plan", "fgemm_run", "fgemm_destroy", "fgemm_workspace_bytes",
                 "moe_grouped_ffn", "moe_workspace_bytes", "fg_status_str", "fg_last_error"):
        assert want in names


def test_library_exports_every_declared_symbol():
    lib = C.CDLL(L.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def E(**kw):
    return L.make_epilogue(**kw)


def plan_status(M, N, K, i, o, epi):
    try:
        L.fgemm_plan(M, N, K, i, o, epi)
        return L.FG_OK
    except L.FgError as e:
        return e.status


def test_plan_validation_statuses():
    ok = E(has_bias=True, ops=(("relu",), ("scale", 2.0)))
    assert plan_status(128, 256, 256, "f32", "f32", ok) == L.FG_OK
    assert plan_status(0, 256, 256, "bf16", "bf16", ok) == L.FG_OK          # empty problem is valid
    assert plan_status(8, 256, 0, "bf16", "bf16", ok) == L.FG_OK            # K = 0: z = b
    assert plan_status(-1, 256, 256, "bf16", "bf16", ok) == L.FG_ERR_INVALID_ARG
    assert plan_status(8, 0, 256, "bf16", "bf16", ok) == L.FG_ERR_INVALID_ARG
    assert plan_status(8, 256, 2 ** 31, "bf16", "bf16", ok) == L.FG_ERR_INVALID_ARG
    # rows of at most 4 MiB: K = 2^21 bf16 / 2^22 e4m3 / 2^20 fp32, not one chunk more
    assert plan_status(8, 256, 2 ** 21, "bf16", "bf16", ok) == L.FG_OK
    assert plan_status(8, 256, 2 ** 21 + 8, "bf16", "bf16", ok) == L.FG_ERR_UNSUPPORTED
    assert plan_status(8, 256, 2 ** 22, "e4m3", "bf16", ok) == L.FG_OK
    assert plan_status(8, 256, 2 ** 22 + 16, "e4m3", "bf16", ok) == L.FG_ERR_UNSUPPORTED
    assert plan_status(8, 256, 2 ** 20 + 4, "f32", "f32", ok) == L.FG_ERR_UNSUPPORTED
    assert plan_status(2 ** 31 - 1, 8, 8, "bf16", "bf16", ok) == L.FG_OK      # M up to 2^31 - 1
    assert plan_status(8, 256, 260, "bf16", "bf16", ok) == L.FG_ERR_ALIGNMENT  # K % 8
    assert plan_status(8, 256, 258, "f32", "f32", ok) == L.FG_ERR_ALIGNMENT    # K % 4
    assert plan_status(8, 252, 256, "bf16", "bf16", ok) == L.FG_ERR_ALIGNMENT  # N % 8 (bf16 out)
    assert plan_status(8, 256, 256, "e4m3", "bf16", ok) == L.FG_OK           # W8A8
    assert plan_status(8, 256, 264, "e4m3", "bf16", ok) == L.FG_ERR_ALIGNMENT  # K % 16
    assert plan_status(8, 256, 256, 7, "bf16", ok) == L.FG_ERR_INVALID_ARG
    assert plan_status(8, 256, 256, "bf16", 9, ok) == L.FG_ERR_INVALID_ARG
    assert plan_status(8, 256, 256, "bf16", "bf16", None) == L.FG_ERR_INVALID_ARG
    bad_kind = E(ops=((17, 0.0),))
    assert plan_status(8, 256, 256, "bf16", "bf16", bad_kind) == L.FG_ERR_INVALID_ARG
    bad_clamp = E(ops=(("clamp", 1.0, -1.0),))
    assert plan_status(8, 256, 256, "bf16", "bf16", bad_clamp) == L.FG_ERR_INVALID_ARG
    nan_op = E(ops=(("scale", float("nan")),))
    assert plan_status(8, 256, 256, "bf16", "bf16", nan_op) == L.FG_ERR_INVALID_ARG
    e = E(ops=(("relu",),))
    e.n_ops = 9
    assert plan_status(8, 256, 256, "bf16", "bf16", e) == L.FG_ERR_INVALID_ARG
    lse = E(reduction="lse")
    assert plan_status(8, 100, 256, "bf16", "f32", lse) == L.FG_OK          # any N for a row LSE
    assert plan_status(8, 256, 256, "bf16", "bf16", lse) == L.FG_ERR_INVALID_ARG
    gn = dict(reduction="groupnorm", gn_groups=32, gn_eps=1e-5)
    assert plan_status(8, 4096, 256, "bf16", "bf16", E(**gn)) == L.FG_OK      # width 128
    assert plan_status(8, 2048, 256, "bf16", "bf16", E(**gn)) == L.FG_OK      # width 64
    assert plan_status(8, 1024, 256, "bf16", "bf16", E(**gn)) == L.FG_OK      # width 32
    assert plan_status(8, 4000, 256, "bf16", "bf16", E(**gn)) == L.FG_OK      # width 125 (second launch)
    assert plan_status(8, 4008, 256, "bf16", "bf16", E(**gn)) == L.FG_ERR_INVALID_ARG  # not divisible
    gn_neg = E(reduction="groupnorm", gn_groups=32, gn_eps=-1.0)
    assert plan_status(8, 4096, 256, "bf16", "bf16", gn_neg) == L.FG_ERR_INVALID_ARG


def test_post_op_validation():
    gn = dict(reduction="groupnorm", gn_groups=32, gn_eps=1e-5)
    chain = (("silu",), ("scale", 1.5), ("mish",), ("leaky_relu", 0.01))
    assert plan_status(8, 4096, 256, "bf16", "bf16", E(post_ops=chain, **gn)) == L.FG_OK
    assert plan_status(8, 100, 256, "bf16", "f32", E(reduction="lse", post_ops=chain)) == L.FG_OK
    assert plan_status(8, 256, 256, "bf16", "bf16", E(ops=chain)) == L.FG_OK     # new kinds as ops
    # post ops without a reduction are rejected: they would be ordinary ops
    assert plan_status(8, 256, 256, "bf16", "bf16", E(post_ops=(("relu",),))) == L.FG_ERR_INVALID_ARG
    assert plan_status(8, 4096, 256, "bf16", "bf16", E(post_ops=((8, 0.0),), **gn)) == L.FG_ERR_INVALID_ARG
    assert plan_status(8, 4096, 256, "bf16", "bf16",
                       E(post_ops=(("clamp", 2.0, 1.0),), **gn)) == L.FG_ERR_INVALID_ARG
    assert plan_status(8, 4096, 256, "bf16", "bf16",
                       E(post_ops=(("leaky_relu", float("inf")),), **gn)) == L.FG_ERR_INVALID_ARG
    for n in (-1, 9):
        e = E(post_ops=(("relu",),), **gn)
        e.n_post_ops = n
        assert plan_status(8, 4096, 256, "bf16", "bf16", e) == L.FG_ERR_INVALID_ARG
    with pytest.raises(L.FgError):
        L.fgemm_plan(8, 256, 256, "bf16", "bf16", E(post_ops=(("relu",),)))
    assert "post op" in L.last_error()


def test_last_error_describes_the_failure():
    with pytest.raises(L.FgError) as ei:
        L.fgemm_plan(8, 256, 260, "bf16", "bf16", E())
    assert "K=260" in str(ei.value) and "multiple of 8" in L.last_error()


def test_groupnorm_group_widths():
    """Any width that divides N is accepted. Widths of 16, 32 and 64
    channels run inside the tile (one launch, no workspace), 256 on the
    256×256 tile; widths no tile holds in registers take a second launch with
    an fp32 workspace of M·N values."""
    def gn(M, N, groups, dt="bf16"):
        p = L.fgemm_plan(M, N, 256, dt, "bf16", E(reduction="groupnorm", gn_groups=groups, gn_eps=1e-5))
        return p.info(), p.workspace_bytes()
    for groups in (32, 16, 8, 4):                       # 16, 32, 64, 128 channels
        i, ws = gn(300, 512, groups)
        assert i["launches"] == 1 and ws == 0, groups
    i, ws = gn(512, 2048, 8)                            # 256 channels
    assert (i["tile_m"], i["tile_n"], i["launches"], ws) == (256, 256, 1, 0)
    for M, N, groups in ((300, 4096, 8), (130, 480, 20), (77, 384, 4), (130, 4096, 1)):
        i, ws = gn(M, N, groups)
        assert i["launches"] == 2 and ws == M * N * 4, (M, N, groups)
    i, ws = gn(256, 2048, 8, "e4m3")                   # no e4m3 tile holds 256 channels
    assert i["launches"] == 2 and ws == 256 * 2048 * 4
    assert plan_status(8, 480, 256, "bf16", "bf16", E(reduction="groupnorm", gn_groups=7)) == L.FG_ERR_INVALID_ARG


def test_tile_choice_and_workspace():
    p = L.fgemm_plan(1024, 8192, 8192, "bf16", "bf16", E(has_bias=True))
    assert p.info() == {"tile_m": 256, "tile_n": 128, "workgroups": 256, "launches": 1, "k_slices": 1}
    assert p.workspace_bytes() == 0
    p = L.fgemm_plan(300, 520, 264, "bf16", "bf16", E())
    assert p.info()["tile_m"] == 128 and p.info()["workgroups"] == 3 * 5 and p.info()["k_slices"] == 1
    assert p.workspace_bytes() == 0
    p = L.fgemm_plan(4096, 8192, 4096, "bf16", "f32", E(reduction="lse"))
    assert p.info() == {"tile_m": 256, "tile_n": 256, "workgroups": 512, "launches": 2, "k_slices": 1}
    assert p.workspace_bytes() == 4096 * 32 * 8
    # few tiles and a long K: split K over 4 slices (36 tiles → 144 workgroups)
    p = L.fgemm_plan(1000, 2056, 4104, "bf16", "bf16", E())
    assert p.info() == {"tile_m": 256, "tile_n": 256, "workgroups": 144, "launches": 1, "k_slices": 4}
    assert p.workspace_bytes() == 512 + 36 * 4 * 256 * 256 * 4        # counter words, then partials
    # the shapes the GPU parity tests use for each large-tile configuration
    for shape, want in (((4000, 4000, 200), (256, 256, 1)), ((2000, 4104, 136), (256, 256, 1)),
                        ((2048, 4096, 128), (256, 128, 1)), ((512, 1024, 8192), (256, 256, 4))):
        i = L.fgemm_plan(*shape, "bf16", "bf16", E()).info()
        assert (i["tile_m"], i["tile_n"], i["k_slices"]) == want, shape
    with pytest.raises(L.FgError) as ei:
        L.fgemm_plan(64, 64, 1 << 22, "bf16", "bf16", E())            # 8 MiB rows
    assert ei.value.status == L.FG_ERR_UNSUPPORTED
    p = L.fgemm_plan(0, 8192, 4096, "bf16", "bf16", E())
    assert p.info()["workgroups"] == 0 and p.info()["launches"] == 0
    p = L.fgemm_plan(128, 256, 256, "f32", "f32", E())
    assert (p.info()["tile_m"], p.info()["tile_n"]) == (64, 128)


def test_run_validation_enqueues_nothing():
    p = L.fgemm_plan(64, 256, 256, "bf16", "bf16", E(has_bias=True))
    fake = 1 << 40          # never dereferenced: validation fails first
    with pytest.raises(L.FgError) as ei:
        L.fgemm_run(p, None, fake, fake, None, None, fake, None, 0)
    assert ei.value.status == L.FG_ERR_INVALID_ARG
    with pytest.raises(L.FgError) as ei:
        L.fgemm_run(p, fake, fake, None, None, None, fake, None, 0)       # bias missing
    assert ei.value.status == L.FG_ERR_INVALID_ARG
    with pytest.raises(L.FgError) as ei:
        L.fgemm_run(p, fake + 2, fake, fake, None, None, fake, None, 0)   # misaligned A
    assert ei.value.status == L.FG_ERR_ALIGNMENT
    lse = L.fgemm_plan(64, 256, 256, "bf16", "f32", E(reduction="lse"))
    with pytest.raises(L.FgError) as ei:
        L.fgemm_run(lse, fake, fake, None, None, None, fake, fake, 8)     # workspace too small
    assert ei.value.status == L.FG_ERR_WORKSPACE
    gn = L.fgemm_plan(64, 256, 256, "bf16", "bf16", E(reduction="groupnorm", gn_groups=2))
    with pytest.raises(L.FgError) as ei:
        L.fgemm_run(gn, fake, fake, None, None, None, fake, None, 0)      # gamma/beta missing
    assert ei.value.status == L.FG_ERR_INVALID_ARG
    empty = L.fgemm_plan(0, 256, 256, "bf16", "bf16", E())
    L.fgemm_run(empty, None, None, None, None, None, None, None, 0)       # M = 0: nothing to do


def test_quantize_validation():
    with pytest.raises(L.FgError) as ei:
        L.fg_quantize_rows_e4m3(1 << 40, 4, 12, 1 << 40, 1 << 40)
    assert ei.value.status == L.FG_ERR_ALIGNMENT
    with pytest.raises(L.FgError) as ei:
        L.fg_quantize_rows_e4m3(None, 4, 16, 1 << 40, 1 << 40)
    assert ei.value.status == L.FG_ERR_INVALID_ARG
    L.fg_quantize_rows_e4m3(None, 0, 16, None, None)                       # zero rows: no-op


def test_status_strings():
    for st in range(6):
        assert L.status_str(st).startswith("FG_")
    assert "unknown" in L.status_str(42)


def test_moe_workspace_and_validation():
    d = L.moe_desc(4096, 2880, 2880, 32, 4)
    ws = L.moe_workspace_bytes(d)
    S = 4096 * 4
    assert ws >= S * 2880 * 2 * 2          # h and the per-slot outputs, bf16
    d8 = L.moe_desc(4096, 2880, 2880, 32, 4, "e4m3")
    assert L.moe_workspace_bytes(d8) > ws   # plus quantised activations and scales
    assert L.moe_workspace_bytes(L.moe_desc(8, 100, 64, 8, 2)) == 0   # invalid -> 0
    fake = 1 << 40
    cases = [
        (L.moe_desc(8, 100, 64, 8, 2), L.FG_ERR_ALIGNMENT),            # H % 64
        (L.moe_desc(8, 128, 64, 0, 1), L.FG_ERR_INVALID_ARG),          # E = 0
        (L.moe_desc(8, 128, 64, 300, 2), L.FG_ERR_INVALID_ARG),        # E > 256
        (L.moe_desc(8, 128, 64, 8, 9), L.FG_ERR_INVALID_ARG),          # top_k > 8
        (L.moe_desc(8, 128, 64, 2, 3), L.FG_ERR_INVALID_ARG),          # top_k > E
        (L.moe_desc(8, 128, 64, 8, 2, "f32"), L.FG_ERR_UNSUPPORTED),
        (L.moe_desc(-1, 128, 64, 8, 2), L.FG_ERR_INVALID_ARG),
        (L.moe_desc(8, 128, 64, 8, 2, limit=-1.0), L.FG_ERR_INVALID_ARG),
    ]
    for desc, want in cases:
        with pytest.raises(L.FgError) as ei:
            L.moe_grouped_ffn(desc, *([fake] * 12), 1 << 30, None)
        assert ei.value.status == want, (desc.T, desc.H, desc.E, desc.top_k)
    d = L.moe_desc(8, 128, 64, 8, 2)
    with pytest.raises(L.FgError) as ei:                                   # workspace too small
        L.moe_grouped_ffn(d, *([fake] * 11), None, 0, None)
    assert ei.value.status == L.FG_ERR_WORKSPACE
    with pytest.raises(L.FgError) as ei:                                   # e4m3 without scales
        L.moe_grouped_ffn(L.moe_desc(8, 128, 64, 8, 2, "e4m3"), fake, fake, fake, fake, None, None,
                          fake, fake, fake, fake, fake, fake, 1 << 30, None)
    assert ei.value.status == L.FG_ERR_INVALID_ARG
    with pytest.raises(L.FgError) as ei:                                   # misaligned tokens
        L.moe_grouped_ffn(d, fake + 4, *([fake] * 11), 1 << 30, None)
    assert ei.value.status == L.FG_ERR_ALIGNMENT


def test_rope_kv_validation():
    fake = 1 << 40

    def st(desc, qkv=fake, bias=fake, pos=fake, table=fake, q=fake, cache=fake):
        try:
            L.bias_rope_kv_update(desc, qkv, bias, pos, table, q, cache)
            return L.FG_OK
        except L.FgError as e:
            return e.status

    D = lambda **kw: L.rope_desc(**{**dict(T=4, n_q=64, n_kv=8, D=64, block_size=64, max_blocks=8,  # noqa: E731
                                          num_blocks=16, base=150000.0), **kw})
    assert st(D(T=0), None, None, None, None, None, None) == L.FG_OK          # nothing to do
    assert st(None) == L.FG_ERR_INVALID_ARG
    assert st(D(T=-1)) == L.FG_ERR_INVALID_ARG
    assert st(D(n_q=0)) == L.FG_ERR_INVALID_ARG
    assert st(D(n_kv=0)) == L.FG_ERR_INVALID_ARG
    assert st(D(D=8)) == L.FG_ERR_INVALID_ARG
    assert st(D(D=72)) == L.FG_ERR_ALIGNMENT                                  # not a multiple of 16
    assert st(D(D=272)) == L.FG_ERR_UNSUPPORTED
    assert st(D(block_size=0)) == L.FG_ERR_INVALID_ARG
    assert st(D(max_blocks=0)) == L.FG_ERR_INVALID_ARG
    assert st(D(num_blocks=0)) == L.FG_ERR_INVALID_ARG
    assert st(D(base=0.0)) == L.FG_ERR_INVALID_ARG
    assert st(D(base=float("inf"))) == L.FG_ERR_INVALID_ARG
    d = D()
    d.interleaved = 2
    assert st(d) == L.FG_ERR_INVALID_ARG
    assert st(D(), qkv=None) == L.FG_ERR_INVALID_ARG
    assert st(D(), cache=None) == L.FG_ERR_INVALID_ARG
    assert st(D(), qkv=fake + 8) == L.FG_ERR_ALIGNMENT
    assert st(D(), bias=fake + 2) == L.FG_ERR_ALIGNMENT
    assert st(D(), pos=fake + 2) == L.FG_ERR_ALIGNMENT
    assert "bias_rope_kv_update" in L.last_error()


def test_finalize_and_rmsnorm_validation_on_the_host():
    # every case fails (or, for T = 0, returns) before any HIP call, so fake
    # device addresses are never touched
    fake = 1 << 40
    L.moe_finalize(fake, fake, 0, 16, 4, None)                              # T = 0: nothing to do
    for args, status in [((2, 12, 4), L.FG_ERR_ALIGNMENT), ((2, 16, 9), L.FG_ERR_INVALID_ARG),
                         ((2, 16, 0), L.FG_ERR_INVALID_ARG), ((-1, 16, 4), L.FG_ERR_INVALID_ARG)]:
        with pytest.raises(L.FgError) as ei:
            L.moe_finalize(fake, fake, *args, None)
        assert ei.value.status == status
    with pytest.raises(L.FgError) as ei:
        L.moe_finalize(fake + 2, fake, 2, 16, 4, None)
    assert ei.value.status == L.FG_ERR_ALIGNMENT
    with pytest.raises(L.FgError) as ei:
        L.moe_finalize(None, fake, 2, 16, 4, None)
    assert ei.value.status == L.FG_ERR_INVALID_ARG
    L.add_rmsnorm(fake, fake, fake, fake, 0, 16, 1e-5, None)               # T = 0
    for args, status in [((2, 12, 1e-5), L.FG_ERR_ALIGNMENT), ((2, 4104, 1e-5), L.FG_ERR_UNSUPPORTED),
                         ((2, 16, -1.0), L.FG_ERR_INVALID_ARG), ((2, 16, float("nan")), L.FG_ERR_INVALID_ARG),
                         ((-1, 16, 1e-5), L.FG_ERR_INVALID_ARG)]:
        with pytest.raises(L.FgError) as ei:
            L.add_rmsnorm(fake, fake, fake, fake, *args, None)
        assert ei.value.status == status
    with pytest.raises(L.FgError) as ei:
        L.add_rmsnorm(fake + 2, fake, fake, fake, 2, 16, 1e-5, None)
    assert ei.value.status == L.FG_ERR_ALIGNMENT
    with pytest.raises(L.FgError) as ei:
        L.add_rmsnorm(None, fake, fake, fake, 2, 16, 1e-5, None)
    assert ei.value.status == L.FG_ERR_INVALID_ARG


def test_e4m3_run_needs_scales_on_the_host():
    fake = 1 << 40
    p = L.fgemm_plan(64, 256, 256, "e4m3", "bf16", E())
    assert p.info()["tile_m"] in (128, 256)
    for sx, sw in ((None, None), (fake, None), (None, fake)):
        with pytest.raises(L.FgError) as ei:
            L.fgemm_run_scaled(p, fake, fake, sx, sw, None, None, None, fake, None, 0)
        assert ei.value.status == L.FG_ERR_INVALID_ARG
    with pytest.raises(L.FgError) as ei:
        L.fgemm_run(p, fake, fake, None, None, None, fake, None, 0)
    assert ei.value.status == L.FG_ERR_INVALID_ARG and "scale" in L.last_error()


def test_header_is_plain_c():
    # the boundary carries no C++ types: the header compiles as C99 (and C++)
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    for lang, std in (("c", "-std=c99"), ("c++", "-std=c++17")):
        r = subprocess.run([gcc, std, "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only", "-x", lang,
                            HEADER], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_trace_validation_without_gpu():
    """The launch-trace calls reject bad requests before any HIP call."""
    for cap in (0, -3, (1 << 20) + 1):
        with pytest.raises(L.FgError) as ei:
            L.fg_trace_begin(cap)
        assert ei.value.status == L.FG_ERR_INVALID_ARG
    assert L.fg_trace_end() == 0                         # closing with nothing traced
    for i in (0, -1, 5):
        with pytest.raises(L.FgError) as ei:
            L.fg_trace_read(i)
        assert ei.value.status == L.FG_ERR_INVALID_ARG


def test_noalloc_moe_rejects_before_any_hip_call():
    """moe_grouped_ffn_noalloc validates the descriptor and the scratch size
    on the host: an invalid descriptor gives its usual status and a problem
    larger than the static scratch FG_ERR_UNSUPPORTED, without a GPU."""
    assert L.moe_noalloc_scratch_bytes() == 64 << 20
    bad = L.moe_desc(8, 100, 64, 8, 2)                       # H not a multiple of 64
    with pytest.raises(L.FgError) as ei:
        L.moe_grouped_ffn_noalloc(bad, *([1 << 40] * 11), None)
    assert ei.value.status == L.FG_ERR_ALIGNMENT
    big = L.moe_desc(4096, 2880, 2880, 32, 4)                # the prefill step needs ~290 MB
    assert L.moe_workspace_bytes(big) > L.moe_noalloc_scratch_bytes()
    with pytest.raises(L.FgError) as ei:
        L.moe_grouped_ffn_noalloc(big, *([1 << 40] * 11), None)
    assert ei.value.status == L.FG_ERR_UNSUPPORTED
    assert "static scratch" in str(ei.value)
    fits = L.moe_desc(900, 2880, 2880, 32, 4)
    assert L.moe_workspace_bytes(fits) <= L.moe_noalloc_scratch_bytes()
