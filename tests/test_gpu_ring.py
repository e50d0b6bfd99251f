"""The LDS-ring chain scan (LBI_ALGO_CHAIN_RING) against the oracle, through
the C-ABI (needs a GPU).

The kernel computes the combines and the apply of the chain scan with the
A_j tiles loaded straight into a ring of LDS blocks and c_j formed on the
matrix cores, in bf16 storage with the hi + lo feedback of the composite.
Tolerances, as for the other bf16 paths: relative Frobenius 2e-2 (the parity
bar) and 1e-3 (the hi + lo feedback leaves about 1e-5; a lost low part or a
mis-indexed block shows far above it), over the true-width values, plus the
elementwise check of the parity suite.  Rows past r_j of a zero-padded
lambda_j must be exactly 0.  Shapes: every ring size the host picks for the
32/64/128 cycles (three rotations), uniform width 64, chains of 1 to 5 slots
(prologue and epilogue), an odd and an even number of loop steps, ragged
batch sizes, and both workloads this kernel serves at full size on sampled
chains.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import binding, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
TOL = 2e-2
EXPECTED = 1e-3
RING = binding.LBI_ALGO_CHAIN_RING


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def cycle_ending_64(K, cycle):
    """r_k = cycle[(k + o) % len(cycle)] with the offset o that makes r_K = 64."""
    n = len(cycle)
    o = next(o for o in range(n) if cycle[(K + o) % n] == 64)
    return tuple(cycle[(k + o) % n] for k in range(K + 1))


def run(x, widths, algo=RING):
    lam = binding.lbi_scan_backward_ex(
        x.A.to(DEV), None if x.b is None else x.b.to(DEV), x.lamK.to(DEV),
        None if widths is None else list(widths), 0, algo)
    torch.cuda.synchronize()
    return lam.cpu()


def true_rows(lam, widths):
    return np.concatenate([np.asarray(lam)[:, j, :widths[j]] for j in range(len(widths) - 1)],
                          axis=1)


def check(lam, x, widths, what):
    want = oracle.recurrence(x.A, x.b, x.lamK)
    got = lam.numpy().astype(np.float64)
    err = oracle.rel_frobenius(true_rows(got, widths), true_rows(want, widths))
    per = oracle.per_chain_rel_frobenius(got, want)
    _say(f"  {what}: rel-Frobenius {err:.3e}, worst chain {per.max():.3e}")
    assert np.isfinite(got).all()
    assert err <= TOL and err <= EXPECTED, f"{what}: {err:.3e}"
    scale = np.abs(want).reshape(want.shape[0], -1).max(axis=1)
    diff = np.abs(got - want).reshape(want.shape[0], -1).max(axis=1)
    assert not (diff > 4 * TOL * np.maximum(scale, 1e-30)).any(), f"{what}: elementwise"
    R = lam.shape[-1]
    for j in range(len(widths) - 1):
        assert (lam[:, j, widths[j]:] == 0).all(), f"{what}: padded rows of slot {j}"


@pytest.mark.parametrize("cycle", [(32, 64, 128), (64, 128, 32), (128, 32, 64)])
@pytest.mark.parametrize("K", [1, 2, 3, 4, 5, 8, 65])
@pytest.mark.parametrize("affine", [True, False])
def test_ring_cycles_against_oracle(cycle, K, affine):
    widths = cycle_ending_64(K, cycle)
    _say(f"[ring] cycle={cycle} K={K} affine={affine} widths[:4]={widths[:4]}")
    x = synth.random_chain(5, K, 128, dtype="bf16", seed=81 + K, affine=affine, widths=widths)
    check(run(x, widths), x, widths, f"cycle {cycle} K{K}")


@pytest.mark.parametrize("K", [1, 2, 3, 32, 33])
@pytest.mark.parametrize("affine", [True, False])
@pytest.mark.parametrize("B", [1, 7, 300])
def test_ring_uniform_64(K, affine, B):
    _say(f"[ring] uniform r=64 B={B} K={K} affine={affine}")
    x = synth.random_chain(B, K, 64, dtype="bf16", seed=83 + K + B, affine=affine)
    widths = (64,) * (K + 1)
    check(run(x, None), x, widths, f"uniform64 B{B} K{K}")
    # the hint with every width 64 is the same call
    assert torch.equal(run(x, widths), run(x, None))


@pytest.mark.parametrize("widths", [(32, 64, 32, 64), (64, 32, 32, 64, 64, 32, 64),
                                    (32, 32, 32, 64)])
def test_ring_storage_64_mixed(widths):
    K = len(widths) - 1
    _say(f"[ring] R=64 widths={widths}")
    x = synth.random_chain(9, K, 64, dtype="bf16", seed=85 + K, widths=widths)
    check(run(x, widths), x, widths, f"R64 {widths}")


def test_ring_long_chain_wraps_the_ring():
    """K = 301 slots of an irregular width sequence: the ring allocation wraps
    many times with tiles of four different sizes."""
    # widths 32 and 64 at random, and 128 always between two 32s: tiles of
    # 2, 4, 8 (32 x 128 and 128 x 32) blocks, any three within the ring
    g = torch.Generator().manual_seed(87)
    widths = []
    while len(widths) < 301:
        t = int(torch.randint(0, 4, (1,), generator=g))
        widths += [[32], [64], [32, 128, 32], [64, 64]][t]
    widths = tuple(widths[:301]) + (64,)
    _say(f"[ring] irregular K=301")
    x = synth.random_chain(6, 301, 128, dtype="bf16", seed=89, widths=widths)
    check(run(x, widths), x, widths, "irregular K301")


@pytest.mark.parametrize("name", ["mixed_widths", "bf16_tokens"])
def test_ring_workload_full_size(name):
    """The two workloads this kernel serves, at full size in the launch
    configuration of the benchmark: every chain against the chain kernel,
    sampled chains against the oracle."""
    wl = synth.WORKLOADS[name]
    _say(f"[ring] workload {name}: B={wl.B} K={wl.K} r={wl.r}")
    x = synth.generate(wl, device=DEV)
    lam = binding.lbi_scan_backward_ex(x.A, x.b, x.lamK, wl.widths, 0, RING)
    old = binding.lbi_scan_backward_ex(x.A, x.b, x.lamK, wl.widths, 0, binding.LBI_ALGO_CHAIN)
    torch.cuda.synchronize()
    widths = wl.interface_widths()
    e = oracle.rel_frobenius(true_rows(lam.cpu().double(), widths),
                             true_rows(old.cpu().double(), widths))
    _say(f"  against the chain kernel: {e:.3e}")
    assert e <= EXPECTED
    idx = torch.randperm(wl.B, generator=torch.Generator().manual_seed(91))[:24]
    idx = torch.cat([torch.tensor([0, wl.B - 1]), idx])
    sub = x.chains(idx.to(DEV)).to("cpu")
    check(lam[idx.to(DEV)].cpu(), sub, widths, f"{name} sampled")


def test_ring_bitwise_reproducible():
    widths = cycle_ending_64(64, (32, 64, 128))
    x = synth.random_chain(40, 64, 128, dtype="bf16", seed=93, widths=widths)
    assert torch.equal(run(x, widths), run(x, widths))


def test_ring_empty_batch():
    lam = binding.lbi_scan_backward_ex(torch.empty((0, 4, 64, 64), dtype=torch.bfloat16,
                                                   device=DEV), None,
                                       torch.empty((0, 64), dtype=torch.bfloat16, device=DEV),
                                       None, 0, RING)
    assert lam.shape == (0, 4, 64)


def test_auto_takes_the_ring_kernel_at_width_128():
    """AUTO runs the LDS-ring kernel for bf16 stored at width 128 with widths
    it takes (bit for bit the explicit call), and the workgroup kernel for
    uniform width 64 (bit for bit LBI_ALGO_CHAIN).  (300 chains: enough that
    AUTO's cost model keeps the chain scan rather than the two-level one.)"""
    widths = cycle_ending_64(64, (32, 64, 128))
    x = synth.random_chain(300, 64, 128, dtype="bf16", seed=95, widths=widths)
    assert torch.equal(run(x, widths, binding.LBI_ALGO_AUTO), run(x, widths, RING))
    y = synth.random_chain(300, 32, 64, dtype="bf16", seed=96)
    assert torch.equal(run(y, None, binding.LBI_ALGO_AUTO), run(y, None, binding.LBI_ALGO_CHAIN))
