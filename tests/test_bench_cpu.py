"""Host-side checks of the measurement code in bench.py (no GPU).

The roofline fractions bench.py reports divide measured times into
algorithmic FLOP and bytes; these tests recompute those figures from the
workload shapes by hand (each input read once, each output written once,
2MNK FLOP), check the published MI355X peaks the fractions are taken
against, the parsing of kernel names into gate/up and down launches, and
that the committed counter summaries are matched to the kernel sources by a
hash that ignores comments but not code."""

import os
import shutil

import pytest

import bench
from paper_2606_02963_amd.synth import FGEMM_SPECS, MOE_SPECS


def test_peaks_are_the_published_dense_figures():
    # 256 CUs × 2.4 GHz × 4096 bf16 FLOP per clock per CU; fp8 twice that
    assert bench.PEAK_BF16_TFLOPS == pytest.approx(256 * 2.4e9 * 4096 / 1e12, rel=1e-4)
    assert bench.PEAK_FP8_TFLOPS == pytest.approx(2 * bench.PEAK_BF16_TFLOPS, rel=1e-4)
    assert bench.PEAK_FP32_TFLOPS == 157.3
    assert bench.PEAK_HBM_GBS == 8000.0


@pytest.mark.parametrize("name,M,N,K,gflop,mbytes", [
    # x [M,K] and W [N,K] bf16, b fp32 [N], out bf16 [M,N] (LSE: fp32 [M];
    # GroupNorm: γ, β fp32 [N] as well)
    ("bf16_gelu_clamp", 1024, 8192, 8192, 137.44, 167.8),
    ("bf16_lse", 4096, 8192, 4096, 274.88, 100.7),
    ("bf16_silu_gn", 2048, 4096, 4096, 68.72, 67.2),
])
def test_dense_algorithmic_work(name, M, N, K, gflop, mbytes):
    spec = FGEMM_SPECS[name]
    assert (spec.M, spec.N, spec.K) == (M, N, K)
    assert spec.flops() / 1e9 == pytest.approx(gflop, abs=0.01)
    assert spec.bytes() / 1e6 == pytest.approx(mbytes, abs=0.05)


def test_moe_step_algorithmic_work():
    T, H, I, E, k = 4096, 2880, 2880, 32, 4
    s = MOE_SPECS["moe_prefill_bf16"]
    assert (s.T, s.H, s.I, s.E, s.k) == (T, H, I, E, k)
    # gate/up 2·(T·k)·(2I)·H plus down 2·(T·k)·I·H
    assert s.flops() / 1e9 == pytest.approx(815.4, abs=0.05)
    weights = E * (2 * I * H + H * I) * 2
    assert weights / 1e9 == pytest.approx(1.59, abs=0.01)
    step = T * H * 2 + T * E * 4 + weights + T * H * 2      # tokens, logits, weights, output
    assert s.bytes(E) == step
    assert s.bytes(E) / 1e9 == pytest.approx(1.64, abs=0.01)
    f8 = MOE_SPECS["moe_prefill_e4m3"]
    assert f8.bytes(E) / 1e9 == pytest.approx(0.85, abs=0.01)
    assert MOE_SPECS["moe_decode_bf16"].flops() / 1e9 == pytest.approx(12.7, abs=0.05)


def test_grouped_gemm_work_per_launch():
    s = MOE_SPECS["moe_prefill_bf16"]
    S = s.T * s.k
    f_gu, b_gu = bench.moe_kernel_work(s, 0, 32, S)
    f_dn, b_dn = bench.moe_kernel_work(s, 1, 32, S)
    assert f_gu / 1e9 == pytest.approx(543.6, abs=0.05)
    assert f_dn / 1e9 == pytest.approx(271.8, abs=0.05)
    assert f_gu + f_dn == pytest.approx(s.flops())
    # gate/up: its weights, the token rows, h written (bf16)
    assert b_gu == 32 * 2 * s.I * s.H * 2 + s.T * s.H * 2 + S * s.I * 2
    # down: its weights, h read, the fp32 slot outputs written
    assert b_dn == 32 * s.H * s.I * 2 + S * s.I * 2 + S * s.H * 4
    assert b_gu / 1e6 == pytest.approx(1179.6, abs=0.1)
    assert b_dn / 1e6 == pytest.approx(814.0, abs=0.1)


@pytest.mark.parametrize("name,epi", [
    ("void fg::grouped_kernel<fg::Tile<(fg::In)1, 128, 192, 2, 2, true>, 0>(fg::GroupedArgs)", 0),
    ("void fg::grouped_kernel<fg::Tile<(fg::In)2, 128, 192, 2, 2, false>, 1>(fg::GroupedArgs)", 1),
    ("_ZN2fg14grouped_kernelINS_4TileILNS_2InE1ELi32ELi128ELi2ELi2ELb0EEELi1EEEvNS_11GroupedArgsE", 1),
    ("void fg::grouped_kernel<fg::Tile<(fg::In)1, 128, 192, 2, 2, true>, 0, false>(fg::GroupedArgs)", 0),
    ("void fg::grouped_kernel<fg::Tile<(fg::In)2, 128, 192, 2, 2, false>, 1, false>(fg::GroupedArgs)", 1),
    ("void fg::grouped_kernel<fg::Tile<(fg::In)2, 32, 192, 2, 2, false>, 0, true>(fg::GroupedArgs)", 0),
    ("_ZN2fg14grouped_kernelINS_4TileILNS_2InE1ELi32ELi128ELi2ELi2ELb0EEELi0ELb1EEEvNS_11GroupedArgsE", 0),
    ("_ZN2fg14grouped_kernelINS_4TileILNS_2InE2ELi128ELi192ELi2ELi2ELb0EEELi1ELb0EEEvNS_11GroupedArgsE", 1),
    ("void fg::moe_finalize_kernel<4, float>(float const*, float const*, unsigned short*, int, long)", None),
])
def test_grouped_kernel_names_parse(name, epi):
    assert bench.grouped_epi(name) == epi


def test_source_hash_ignores_comments_but_not_code(tmp_path, monkeypatch):
    src = os.path.join(bench.ROOT, "paper_2606_02963_amd", "csrc")
    dst = tmp_path / "paper_2606_02963_amd" / "csrc"
    shutil.copytree(src, dst)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_source_hash(bench.MOE_KERNEL_SOURCES)
    f = dst / "moe.hip"
    text = f.read_text()
    f.write_text("// a new comment\n/* and a block\n   comment */\n" + text.replace("\n", "\n\n", 3))
    assert bench.kernel_source_hash(bench.MOE_KERNEL_SOURCES) == h0
    f.write_text(text.replace("{", "{ (void)0;", 1))
    assert bench.kernel_source_hash(bench.MOE_KERNEL_SOURCES) != h0


def test_committed_counter_summaries_match_the_present_sources():
    # every .pmc.json under profiles/ was taken on the kernels as they are
    for name, sources in [("moe_prefill_bf16", bench.MOE_KERNEL_SOURCES),
                          ("moe_prefill_bf16_gateup", bench.MOE_KERNEL_SOURCES),
                          ("moe_decode_e4m3", bench.MOE_KERNEL_SOURCES),
                          ("fgemm_bf16_gelu_clamp_1024x8192x8192", bench.KERNEL_SOURCES),
                          ("fgemm_bf16_silu_gn_2048x4096x4096", bench.KERNEL_SOURCES)]:
        assert bench.measured_traffic(name, sources) is not None, name
