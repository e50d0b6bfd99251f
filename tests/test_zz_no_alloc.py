"""lbi_scan_backward_noalloc (the library's static scratch array in place of
a workspace) against lbi_scan_backward_ex, through the C-ABI (needs a GPU).

Two calls in a row on the same GPU share the array; the second is smaller
than the first, so it runs over what the first left there.  Tolerances are
the parity bar: relative Frobenius 1e-5 for float32 storage, 2e-2 for bf16,
against both the workspace entry point and the oracle; where both entry
points run the same plan, the results are equal bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import binding, synth

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _both(x, algo, math=binding.LBI_MATH_DEFAULT):
    dev = torch.device("cuda:0")
    A, lk = x.A.to(dev), x.lamK.to(dev)
    b = None if x.b is None else x.b.to(dev)
    want = binding.lbi_scan_backward_ex(A, b, lk, None, math, algo)
    lam = torch.full_like(want, float("nan"))
    binding.lbi_scan_backward_noalloc(A, b, lk, None, math, algo, lam=lam)
    torch.cuda.synchronize()
    return lam, want


def _check(got, want, x, tol, what):
    g = got.cpu().double().numpy()
    e_ws = oracle.rel_frobenius(g, want.cpu().double().numpy())
    e_or = oracle.rel_frobenius(g, oracle.recurrence(x.A, x.b, x.lamK))
    _say(f"  {what}: vs workspace entry {e_ws:.3e}, vs oracle {e_or:.3e}")
    assert np.isfinite(g).all()
    assert e_ws <= tol and e_or <= tol


def test_noalloc_two_calls_in_a_row():
    # 1) 8 chains of 512 slots, fp32, AUTO: the two-level scan.  Its
    #    composites (exactly 64 MiB of P, plus c and the carries) do not fit
    #    the array, so this call keeps only the segment aggregates and scans
    #    every segment again from its carry.
    x1 = synth.random_chain(8, 512, 64, dtype="f32", seed=61)
    need = binding.lbi_scan_backward_workspace_bytes_ex(8, 512, 64, 0, binding.LBI_ALGO_AUTO)
    assert need > binding.LBI_NOALLOC_SCRATCH_BYTES
    _say("[noalloc] B=8 K=512 r=64 f32 auto (two-level, aggregates only)")
    got, want = _both(x1, binding.LBI_ALGO_AUTO)
    _check(got, want, x1, TOL["f32"], "B=8 K=512 f32")
    # 2) smaller: 3 bf16 chains of 100 slots at r = 32, the two-level scan
    #    with every composite kept (the workspace call's own plan): equal bit
    #    for bit, over the first call's leftovers
    x2 = synth.random_chain(3, 100, 32, dtype="bf16", seed=62)
    _say("[noalloc] B=3 K=100 r=32 bf16 two-level")
    got, want = _both(x2, binding.LBI_ALGO_TWO_LEVEL)
    _check(got, want, x2, TOL["bf16"], "B=3 K=100 bf16")
    assert torch.equal(got, want)


def test_noalloc_without_scratch_use_matches_bit_for_bit():
    # the chain scan uses no scratch: the same kernels, the same results
    for B, K, r, dt in ((300, 20, 16, "f32"), (5, 33, 64, "bf16")):
        x = synth.random_chain(B, K, r, dtype=dt, seed=63 + K)
        _say(f"[noalloc] B={B} K={K} r={r} {dt} chain")
        got, want = _both(x, binding.LBI_ALGO_CHAIN)
        assert torch.equal(got, want)


@pytest.mark.parametrize("algo", ["ring", "auto"])
def test_noalloc_ring_kernel_with_widths(algo):
    # the LDS-ring chain kernel (explicit, and AUTO's choice at width 128 with
    # these widths: 300 chains keep AUTO on the chain scan) needs no scratch
    # either: equal bit for bit, with the hint
    widths = tuple((32, 64, 128)[k % 3] for k in range(10)) + (64,)
    x = synth.random_chain(300, 10, 128, dtype="bf16", seed=64, widths=widths)
    a = binding.LBI_ALGO_CHAIN_RING if algo == "ring" else binding.LBI_ALGO_AUTO
    dev = torch.device("cuda:0")
    A, b, lk = x.A.to(dev), x.b.to(dev), x.lamK.to(dev)
    _say(f"[noalloc] B=300 K=10 widths 32/64/128 bf16 {algo}")
    want = binding.lbi_scan_backward_ex(A, b, lk, list(widths), 0, a)
    lam = torch.full_like(want, float("nan"))
    binding.lbi_scan_backward_noalloc(A, b, lk, list(widths), 0, a, lam=lam)
    torch.cuda.synchronize()
    assert torch.equal(lam, want)
    _check(lam, want, x, TOL["bf16"], "ring widths")


def test_noalloc_tree_scan_levels_in_the_array():
    """The tree scan over levels of chunk aggregates keeps each level's
    aggregates and carries in the array: equal bit for bit to the workspace
    call (the same plan), and at the parity bar against the oracle."""
    for B, K, r, dt in ((3, 100, 64, "f32"), (2, 300, 32, "bf16")):
        x = synth.random_chain(B, K, r, dtype=dt, seed=65 + K)
        _say(f"[noalloc] B={B} K={K} r={r} {dt} tree")
        got, want = _both(x, binding.LBI_ALGO_TREE)
        _check(got, want, x, TOL[dt], f"tree B={B} K={K} {dt}")
        assert torch.equal(got, want)

