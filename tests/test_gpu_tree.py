"""The log-depth tree scan (LBI_ALGO_TREE) against the oracle, through the
C-ABI (needs a GPU).

Tolerances are the parity bar: relative Frobenius 1e-5 for float32 storage
and 2e-2 for bf16 storage (every product is formed at fp32 accuracy by the
exact three-part split, so bf16 results are also held to 1e-3, as in the
other parity tests).  Chains whose products do not contract carry fp32
rounding as a random walk over the tree's levels; their bound is the same
8 sqrt(K r) 2^-24 as for the chain scan.  Permutation chains with integer b
are exact at every step and must match bit for bit.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import binding, synth

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
BF16_EXPECTED = 1e-3
TREE = binding.LBI_ALGO_TREE


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def tree(x, widths=None, math_=binding.LBI_MATH_DEFAULT, stream=None):
    dev = torch.device("cuda:0")
    lam = binding.lbi_scan_backward_ex(x.A.to(dev), None if x.b is None else x.b.to(dev),
                                       x.lamK.to(dev), widths, math_, TREE, stream=stream)
    torch.cuda.synchronize()
    return lam


def ref(x, idx=None):
    if idx is not None:
        x = x.chains(idx)
    return oracle.recurrence(x.A, x.b, x.lamK)


def check(got, want, tol, what):
    got = np.asarray(got, dtype=np.float64)
    err = oracle.rel_frobenius(got, want)
    per = oracle.per_chain_rel_frobenius(got, want)
    _say(f"  {what}: rel-Frobenius {err:.3e}, worst chain {per.max():.3e}")
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    assert err <= tol, f"{what}: relative Frobenius error {err:.3e} > {tol:.1e}"
    scale = np.abs(want).reshape(want.shape[0], -1).max(axis=1)
    diff = np.abs(got - want).reshape(want.shape[0], -1).max(axis=1)
    bad = diff > 4 * tol * np.maximum(scale, 1e-30)
    assert not bad.any(), f"{what}: elementwise error in chains {np.nonzero(bad)[0][:8]}"
    return err


# K spans one chunk (8 at r = 64, 16 below), a partial chunk, two and three
# levels of aggregates, and ragged last chunks at every level
SHAPES = [(1, 1), (3, 2), (2, 7), (1, 8), (2, 9), (3, 16), (1, 17), (2, 63), (1, 64), (2, 65),
          (3, 130), (1, 513)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("r", [16, 32, 64])
@pytest.mark.parametrize("affine", [True, False])
def test_tree_ragged_shapes(r, dtype, affine):
    for B, K in SHAPES:
        _say(f"[tree] B={B} K={K} r={r} {dtype} affine={affine}")
        x = synth.random_chain(B, K, r, dtype=dtype, seed=101 + K + r, affine=affine)
        err = check(tree(x).cpu().numpy(), ref(x), TOL[dtype], f"B{B} K{K} r{r} {dtype}")
        if dtype == "bf16":
            assert err <= BF16_EXPECTED


@pytest.mark.parametrize("r", [16, 32, 64])
def test_tree_exact_on_permutations(r):
    for K in (1, 7, 9, 64, 100):
        x = synth.permutation_chain(3, K, r, dtype="f32", seed=K + 5 * r)
        got = tree(x).cpu().numpy().astype(np.float64)
        assert np.array_equal(got, ref(x)), f"r={r} K={K}"
        xb = synth.permutation_chain(2, K, r, dtype="bf16", seed=K + 7 * r)
        assert np.array_equal(tree(xb).cpu().numpy().astype(np.float64), ref(xb)), \
            f"bf16 r={r} K={K}"


@pytest.mark.parametrize("spectrum", ["orthogonal", "uniform"])
def test_tree_long_undamped_chains(spectrum):
    """512 slots that neither decay nor grow much: the flat fp32 tolerance
    holds through three levels of aggregates."""
    x = synth.random_chain(2, 512, 64, dtype="f32", seed=7, spectrum=spectrum)
    err = check(tree(x).cpu().numpy(), ref(x), TOL["f32"], f"K=512 {spectrum}")
    assert err <= 8 * math.sqrt(512 * 64) * 2.0 ** -24


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K", [7, 16])
def test_tree_paper_operating_point(K, dtype):
    """The paper's setting: one sequence, K = 7 or 16 regions, r = 64."""
    x = synth.random_chain(1, K, 64, dtype=dtype, seed=K, affine=False)
    err = check(tree(x).cpu().numpy(), ref(x), TOL[dtype], f"B=1 K={K} r=64 {dtype}")
    if dtype == "bf16":
        assert err <= BF16_EXPECTED


def test_tree_paper_width_full_size():
    """paper_width (256 chains of 32 slots, r = 64, fp32) at full size:
    sampled chains against the oracle, the whole output against the chain
    scan."""
    wl = synth.WORKLOADS["paper_width"]
    x = synth.generate(wl, device="cuda:0")
    lam = tree(x)
    g = torch.Generator().manual_seed(3)
    idx = torch.cat([torch.tensor([0, wl.B - 1]),
                     torch.randperm(wl.B - 2, generator=g)[:46] + 1]).sort().values
    check(lam[idx.to(lam.device)].cpu().numpy(), ref(x.to("cpu"), idx), TOL["f32"],
          "paper_width tree")
    chain = binding.lbi_scan_backward_ex(x.A, x.b, x.lamK, None, binding.LBI_MATH_DEFAULT,
                                         binding.LBI_ALGO_CHAIN)
    torch.cuda.synchronize()
    d = oracle.rel_frobenius(lam.cpu().double().numpy(), chain.cpu().double().numpy())
    _say(f"  tree vs chain scan: {d:.3e}")
    assert d <= 2 * TOL["f32"]


def test_tree_hint_null_b_determinism_and_stream():
    """A widths hint changes nothing; b = NULL equals b = 0; results are
    bitwise reproducible; a non-default stream gives the same bits."""
    K, r = 40, 64
    widths = synth.cyclic_widths(K, (32, 64, 16))
    x = synth.random_chain(3, K, r, dtype="f32", seed=9, widths=widths)
    a = tree(x)
    assert torch.equal(a, tree(x, widths=widths))
    assert torch.equal(a, tree(x))
    s = torch.cuda.Stream()
    assert torch.equal(a, tree(x, stream=s))
    for j in range(K):
        if widths[j] < r:
            assert float(a[:, j, widths[j]:].abs().max()) == 0.0
    check(a.cpu().numpy(), ref(x), TOL["f32"], "hinted")
    x0 = synth.Inputs(x.A, None, x.lamK, x.widths, x.workload)
    xz = synth.Inputs(x.A, torch.zeros_like(x.b), x.lamK, x.widths, x.workload)
    assert torch.equal(tree(x0), tree(xz))


def test_tree_split_math_equals_default():
    x = synth.random_chain(2, 20, 32, dtype="f32", seed=11)
    assert torch.equal(tree(x), tree(x, math_=binding.LBI_MATH_F32_SPLIT))


def test_tree_propagates_nan():
    x = synth.random_chain(1, 9, 16, dtype="f32", seed=13)
    A = x.A.clone()
    A[0, 4, 2, 3] = float("nan")
    y = tree(synth.Inputs(A, x.b, x.lamK, None, x.workload)).cpu()
    assert torch.isnan(y[0, :5]).any() and torch.isfinite(y[0, 5:]).all()


def test_auto_takes_one_tree_launch_where_measured_faster():
    """AUTO runs one launch of the tree scan for chains within a chunk at
    r <= 32 (fp32 from K = 5, bf16 past K = 8, B <= 256): it equals the
    explicit call bit for bit there, and keeps the chain kernels elsewhere."""
    auto = binding.LBI_ALGO_AUTO

    def run(x, algo):
        lam = binding.lbi_scan_backward_ex(x.A.to("cuda:0"), x.b.to("cuda:0"),
                                           x.lamK.to("cuda:0"), None, 0, algo)
        torch.cuda.synchronize()
        return lam

    for B, K, r, dt in ((4, 16, 32, "f32"), (256, 5, 16, "f32"), (3, 12, 16, "bf16"),
                        (2, 16, 32, "bf16"), (4, 8, 16, "f32")):
        x = synth.random_chain(B, K, r, dtype=dt, seed=K + r)
        assert torch.equal(run(x, auto), run(x, TREE)), (B, K, r, dt)
    for B, K, r, dt, other in ((4, 8, 64, "f32", binding.LBI_ALGO_CHAIN_SPLITK),
                               (3, 7, 64, "bf16", binding.LBI_ALGO_CHAIN),
                               (4, 4, 32, "f32", binding.LBI_ALGO_CHAIN),
                               (3, 8, 16, "bf16", binding.LBI_ALGO_CHAIN_WAVE),
                               (300, 8, 32, "f32", binding.LBI_ALGO_CHAIN)):
        x = synth.random_chain(B, K, r, dtype=dt, seed=K + r + 1)
        assert torch.equal(run(x, auto), run(x, other)), (B, K, r, dt)
