"""Host-side accounting of bench.py: FLOPs per step, the expert GEMMs' HBM
floors and the two-sided roofline (no GPU)."""
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402
from moe_inputs import config  # noqa: E402


def test_step_flops_are_three_forwards():
    cfg = config("qwen3")
    fwd, bwd = bench.layer_flops(cfg)
    T, d, E, k, f = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["f"]
    assert fwd == 2 * T * d * E + 6 * T * k * d * f
    assert bwd == 2 * fwd


def test_hbm_floor_counts_weights_of_experts_with_rows_only():
    cfg = dict(config("qwen3"), T=16, k=2, E=4)
    d, f = cfg["d"], cfg["f"]
    counts = [10, 0, 22, 0]  # 32 rows = T k; two experts without rows
    R = 32
    fl = bench.gemm_hbm_floor(cfg, counts)
    assert fl["gemm_gateup_fwd"] == 2 * (2 * d * f * 2) + R * d * 2 + R * 3 * f * 2
    assert fl["gemm_down_fwd"] == 2 * (f * d * 2) + R * f * 2 + R * d * 2
    assert fl["gemm_down_dgrad"] == 2 * (f * d * 2) + R * d * 2 + R * 4 * f * 2
    assert fl["gemm_gateup_dgrad"] == 2 * (2 * d * f * 2) + R * 2 * f * 2 + R * d * 2
    # every expert's weight gradient is written, zero or not
    assert fl["gemm_down_wgrad"] == 4 * f * d * 2 + R * (f + d) * 2
    assert fl["gemm_gateup_wgrad"] == 4 * 2 * d * f * 2 + R * (d + 2 * f) * 2


def test_hbm_floor_fp8_reads_one_byte_codes():
    cfg = dict(config("qwen3"), T=16, k=2, E=4, fp8=2)
    d, f = cfg["d"], cfg["f"]
    fl = bench.gemm_hbm_floor(cfg, [32, 0, 0, 0])
    assert fl["gemm_gateup_fwd"] == 2 * d * f + 32 * d + 32 * 3 * f * 2
    assert fl["gemm_down_dgrad"] == f * d + 32 * d + 32 * 4 * f * 2
    assert fl["gemm_gateup_wgrad"] == 4 * 2 * d * f * 2 + 32 * (d + 2 * f) * 2  # bf16 in every FP8 level


@pytest.mark.parametrize("flops,bytes_,secs,bound", [(2.5e12, 4e9, 1e-3, "mfma"), (1e12, 8e9, 2e-3, "hbm")])
def test_two_sided_roofline(flops, bytes_, secs, bound):
    r = bench.gemm_roof(flops, bytes_, secs, 2500.0)
    assert r["bound"] == bound and r["other_side"]["bound"] != bound
    t_c, t_m = flops / 2.5e15, bytes_ / 8e12
    assert r["frac"] == pytest.approx(max(t_c, t_m) / secs)
    assert r["mfma_ceiling"] == pytest.approx(min(1.0, t_c / max(t_c, t_m)))
    mf = r if bound == "mfma" else r["other_side"]
    assert mf["achieved"] == pytest.approx(flops / secs / 1e12)


def test_fp8_gather_kernels_count_their_code_rows():
    base = config("qwen3")
    T, d, k = base["T"], base["d"], base["k"]
    R = T * k
    w0, w1, w2 = (bench.kernel_work(dict(base, fp8=lv)) for lv in (0, 1, 2))
    assert w1["scatter"][1] - w0["scatter"][1] == R * (d + 4)
    assert w1["combine_bwd"][1] == w0["combine_bwd"][1]
    assert w2["combine_bwd"][1] - w0["combine_bwd"][1] == R * (d + 4)
