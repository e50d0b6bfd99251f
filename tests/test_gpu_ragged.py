"""Parity of the compact (ragged) entry point, lbi_scan_backward_ragged, through
the C-ABI (needs a GPU).

The ragged call runs the hinted chain scan on the same tiles, only addressed
compactly, so it must equal the padded call with the widths hint and the same
kernel bit for bit (LBI_ALGO_CHAIN_RING for the bf16 widths that the LDS-ring
kernel takes, LBI_ALGO_CHAIN otherwise); it is also held to the oracle at the tolerances of
the scan (fp32 1e-5, bf16 2e-2 relative Frobenius over the true-width values).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import binding, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
TOL = {"f32": 1e-5, "bf16": 2e-2}
MATH = {"split": binding.LBI_MATH_F32_SPLIT, "mfma": binding.LBI_MATH_F32_MFMA, None: 0}
MODES = [("f32", "split"), ("f32", "mfma"), ("bf16", None)]
MODE_IDS = ["f32-split", "f32-mfma", "bf16"]


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def ring_takes(dtype, arith, widths, R):
    """Whether the ragged call runs the LDS-ring kernel: bf16 in the default
    arithmetic, widths 32/64/128 with r_K = 64, tiles of at most 16 blocks
    (8 at R = 64); the ring sizes of these tests all fit."""
    if dtype != "bf16" or arith is not None or R not in (64, 128) or widths[-1] != 64:
        return False
    if any(w not in (32, 64, 128) for w in widths):
        return False
    return all((widths[j] // 16) * (widths[j + 1] // 32) <= (8 if R == 64 else 16)
               for j in range(len(widths) - 1))


def _run_both(x, arith):
    """(ragged result unpacked to [B, K, R], the padded hinted call with the
    same kernel: the LDS-ring chain scan where the ragged call takes it, else
    the chain scan)."""
    R = x.A.shape[-1]
    p = synth.pack_ragged(x)
    lam_c = binding.lbi_scan_backward_ragged(
        p.A.to(DEV), None if p.b is None else p.b.to(DEV), p.lamK.to(DEV), p.widths,
        MATH[arith])
    dtype = "bf16" if x.A.dtype == torch.bfloat16 else "f32"
    algo = (binding.LBI_ALGO_CHAIN_RING if ring_takes(dtype, arith, x.widths, R)
            else binding.LBI_ALGO_CHAIN)
    lam_p = binding.lbi_scan_backward_ex(
        x.A.to(DEV), None if x.b is None else x.b.to(DEV), x.lamK.to(DEV), list(x.widths),
        MATH[arith], algo)
    torch.cuda.synchronize()
    return synth.unpack_ragged(lam_c, p.widths, R).cpu(), lam_p.cpu()


def _true_rows(lam, widths):
    """The concatenated true-width values of lambda [B, K, R]."""
    return torch.cat([lam[:, j, :widths[j]] for j in range(len(widths) - 1)], dim=1)


@pytest.mark.parametrize("dtype,arith", MODES, ids=MODE_IDS)
@pytest.mark.parametrize("affine", [True, False])
@pytest.mark.parametrize("cycle,K", [((32, 64, 128), 70), ((16, 48, 32), 33), ((16,), 5),
                                     ((64, 32), 2), ((128, 16, 96, 64), 9), ((32,), 1)])
def test_ragged_equals_padded_and_oracle(dtype, arith, affine, cycle, K):
    widths = synth.cyclic_widths(K, cycle)
    R = max(widths)
    R = 16 if R <= 16 else 32 if R <= 32 else 64 if R <= 64 else 128
    _say(f"[ragged] {dtype}/{arith} affine={affine} cycle={cycle} K={K} R={R}")
    x = synth.random_chain(3, K, R, dtype=dtype, seed=67 + K, affine=affine, widths=widths)
    lam_c, lam_p = _run_both(x, arith)
    assert torch.equal(lam_c, lam_p), "ragged and padded hinted chain scans differ"
    ref = oracle.recurrence(x.A, x.b, x.lamK)
    err = oracle.rel_frobenius(_true_rows(lam_c, widths).numpy(),
                               _true_rows(torch.from_numpy(ref), widths).numpy())
    assert err <= TOL[dtype], f"rel err {err:.3g}"


def test_ragged_permutation_chain_exact():
    """Rectangular 0/1 selection blocks with integer b: every value exact."""
    widths = (32, 64, 32, 64, 32)
    K = 4
    gen = torch.Generator().manual_seed(71)
    A = torch.zeros((2, K, 64, 64))
    for j in range(K):
        rj, rn = widths[j], widths[j + 1]
        for bb in range(2):
            cols = torch.randperm(rn, generator=gen)[:min(rj, rn)]
            for i in range(min(rj, rn)):
                A[bb, j, i, cols[i]] = 1.0
    b = torch.zeros((2, K, 64))
    for j in range(K):
        b[:, j, :widths[j]] = torch.randint(-8, 9, (2, widths[j]), generator=gen).float()
    lamK = torch.zeros((2, 64))
    lamK[:, :widths[K]] = torch.randint(-8, 9, (2, widths[K]), generator=gen).float()
    wl = synth.Workload("perm_ragged", 2, K, 64, "f32", 0, "orthogonal", True, widths)
    x = synth.Inputs(A, b, lamK, widths, wl)
    lam_c, lam_p = _run_both(x, "split")
    ref = oracle.recurrence(A, b, lamK)
    assert torch.equal(lam_c, lam_p)
    assert np.array_equal(_true_rows(lam_c, widths).numpy().astype(np.float64),
                          _true_rows(torch.from_numpy(ref), widths).numpy())


def test_ragged_mixed_widths_full_size():
    """The mixed-width workload (B=1024, K=64, r_k cycling 32/64/128, bf16) in
    compact storage: 3.4x smaller than padded, identical results."""
    wl = synth.WORKLOADS["mixed_widths"]
    _say("[ragged] mixed_widths full size")
    x = synth.generate(wl, device=DEV)
    p = synth.pack_ragged(x)
    lam_c = binding.lbi_scan_backward_ragged(p.A, p.b, p.lamK, p.widths)
    # (the ragged call takes the LDS-ring kernel for these widths)
    assert ring_takes("bf16", None, p.widths, wl.r)
    lam_p = binding.lbi_scan_backward_ex(x.A, x.b, x.lamK, list(x.widths), 0,
                                         binding.LBI_ALGO_CHAIN_RING)
    torch.cuda.synchronize()
    assert p.A.numel() * 3.3 < x.A.numel()
    assert torch.equal(synth.unpack_ragged(lam_c, p.widths, wl.r), lam_p)
    idx = torch.randperm(wl.B, generator=torch.Generator().manual_seed(73))[:32]
    sub = x.chains(idx.to(DEV)).to("cpu")
    ref = oracle.recurrence(sub.A, sub.b, sub.lamK)
    got = synth.unpack_ragged(lam_c[idx.to(DEV)], p.widths, wl.r).cpu()
    err = oracle.rel_frobenius(_true_rows(got, p.widths).numpy(),
                               _true_rows(torch.from_numpy(ref), p.widths).numpy())
    assert err <= TOL["bf16"]


def test_ragged_empty_batch():
    widths = (32, 64)
    lam = binding.lbi_scan_backward_ragged(
        torch.empty((0, 2048), device=DEV), None, torch.empty((0, 64), device=DEV), widths)
    assert lam.shape == (0, 32)
