"""The benchmark's cost accounting and the workload recipe reproduce the
numbers the paper prints (tests/golden/paper_numbers.json, cited there)."""
import json
import os

import pytest
import torch

import bench
from paper_2605_09204_amd import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


def _matmul_macs_per_combine(r):
    # flops of one combine minus its matvec and add, halved: multiply-adds of A A'
    wl = synth.Workload("one", B=1, K=2, r=r, dtype="f32", seed=0)
    apply = 2 * (2 * r * r + r)
    return (bench.flops_alg(wl) - apply - (2 * r * r + r)) // 2


def test_scan_work_counts_r_cubed_per_combine():
    g = GOLD["scan_negligibility"]
    assert _matmul_macs_per_combine(g["r"]) == g["r"] ** 3
    assert g["K"] * _matmul_macs_per_combine(g["r"]) == g["Kr3"]
    assert _matmul_macs_per_combine(64) == pytest.approx(GOLD["per_combine"]["r3_approx"], rel=0.01)


def test_full_rank_comparison():
    g = GOLD["full_rank_scan"]
    d = g["B"] * g["L"] * g["D"]
    assert d == pytest.approx(g["d_approx"], rel=0.01)
    assert d ** 3 == pytest.approx(g["d3_approx"], rel=0.01)
    ratio = d ** 3 / _matmul_macs_per_combine(64)
    assert 0.5 * g["ratio_order"] < ratio < 2 * g["ratio_order"]


def test_scan_payload_56_kb():
    g = GOLD["scan_payload"]
    n = bench.scan_payload_bytes(g["K"], g["r"], 2)
    assert n == 57344 and round(n / 1024) == g["approx_KB"]


def test_concentrated_recipe_matches_spectral_table():
    g = GOLD["spectral_r64"]
    assert g["local_spectral_norm"] / g["rms_singular_value"] == pytest.approx(g["stated_ratio"], rel=0.02)
    x = synth.generate(synth.WORKLOADS["long_chain"].with_(B=1, K=8))
    s = torch.linalg.svdvals(x.A[0].double())
    ratio = s[:, 0] / torch.sqrt((s * s).mean(-1))
    assert torch.allclose(ratio, torch.full_like(ratio, g["stated_ratio"]), rtol=1e-4)


def test_work_inflation_floor():
    # F_alg / F_seq at r = 64 is about r (Table 'transport-size-comparison': the
    # scan replaces Theta(r^2) matvecs with Theta(r^3) combines)
    for name in ("paper_width", "bf16_tokens", "long_chain"):
        wl = synth.WORKLOADS[name]
        infl = bench.flops_alg(wl) / bench.flops_seq(wl)
        assert 60 < infl < 66
