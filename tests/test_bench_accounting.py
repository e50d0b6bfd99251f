"""The benchmark's per-launch accounting, written out from the shapes: the
algorithmic bytes (every input byte read once, every adjoint written once in
fp32), the matrix-core work each arithmetic executes, and the one-GPU guard.
These figures feed the roofline fields of the JSON line."""
import pytest

import bench
from paper_2605_09204_amd import synth


def test_algorithmic_bytes_long_chain():
    wl = synth.WORKLOADS["long_chain"]
    B, K, r = wl.B, wl.K, wl.r
    assert (B, K, r, wl.dtype, wl.affine) == (512, 512, 64, "f32", True)
    want = B * (K * r * r * 4 + K * r * 4 + r * 4) + B * K * r * 4
    assert bench.bytes_alg(wl) == want == 4429316096


def test_algorithmic_bytes_bf16_tokens_without_b():
    wl = synth.WORKLOADS["bf16_tokens"]
    B, K, r = wl.B, wl.K, wl.r
    assert (wl.dtype, wl.affine) == ("bf16", False)
    assert bench.bytes_alg(wl) == B * (K * r * r * 2 + r * 2) + B * K * r * 4


def test_algorithmic_bytes_mixed_widths_count_true_widths():
    wl = synth.WORKLOADS["mixed_widths"]
    w = bench.widths_of(wl)
    assert len(w) == wl.K + 1 and max(w) == wl.r
    a = sum(w[j] * w[j + 1] for j in range(wl.K))
    b = sum(w[:wl.K])
    padded_out = wl.K * wl.r * 4
    assert bench.bytes_alg(wl) == wl.B * ((a + b + w[wl.K]) * 2 + padded_out)
    assert bench.bytes_alg(wl, compact_out=True) == wl.B * ((a + b + w[wl.K]) * 2 + b * 4)
    # padded storage reads whole r x r tiles
    assert bench.bytes_alg(wl, padded=True) == wl.B * (
        (wl.K * wl.r * wl.r + wl.K * wl.r + wl.r) * 2 + padded_out)


@pytest.mark.parametrize("math,dtype,reps", [("split", "f32", 6), ("mfma", "f32", 1),
                                             ("split", "bf16", 2), ("bf16single", "bf16", 1)])
def test_executed_matrix_core_work(math, dtype, reps):
    # K - 1 products of r x r by r x r per chain (the first slot is a copy),
    # repeated once per partial product of the arithmetic
    wl = synth.WORKLOADS["long_chain"].with_(B=3, K=9, dtype=dtype)
    r = wl.r
    assert bench.mfma_flops_executed(wl, math) == 3 * 8 * 2 * r * r * r * reps


def test_executed_work_rounds_k_up_for_bf16_products():
    # bf16 products take k in blocks of 32: at r = 16 the contraction runs 32 deep
    wl = synth.Workload("r16", B=2, K=5, r=16, dtype="bf16", seed=0)
    assert bench.mfma_flops_executed(wl, "split") == 2 * 4 * 2 * 16 * 32 * 16 * 2
    assert bench.mfma_flops_executed(wl.with_(dtype="f32"), "mfma") == 2 * 4 * 2 * 16 ** 3


def test_mode_names():
    f32 = synth.WORKLOADS["long_chain"]
    bf = synth.WORKLOADS["bf16_tokens"]
    assert bench.mode_of(f32, "split") == "f32-split"
    assert bench.mode_of(f32, "mfma") == "f32-mfma"
    assert bench.mode_of(f32.with_(r=128), "split") == "f32-mfma"
    assert bench.mode_of(bf, "split") == "bf16"
    assert bench.mode_of(bf, "bf16single") == "bf16-single"


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) != 0
    assert "one GPU only" in capsys.readouterr().err


def test_single_rounding_needs_bf16_storage(capsys):
    assert bench.main(["--workload", "long_chain", "--math", "bf16single"]) == 2
    assert "needs bf16 storage" in capsys.readouterr().err
