"""Parity of Phase 1 with the token-mixing region block
(lbi_region_jacobians_ssm) against the fp64 autograd oracle
(oracle.region_jacobians / region_jacobian_columns with phi="ssm"), through
the C-ABI (needs a GPU).

Tolerance as for the token-wise block: bf16 operands with fp32 accumulation
in every product (the states s, silu(W1 s) and the tangent operands c_l Jdec
and the scaled first tangent product are rounded to bf16 where they feed one),
so the relative Frobenius error of J^T is held to 2e-2.  The paper
configuration is checked on 16 sampled (sequence, region) pairs, two columns
of J each, by forward-mode AD in the oracle.
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


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run(x, **kw):
    g = x.to(DEV)
    A, mn = binding.lbi_region_jacobians_ssm(g.params, g.x_embed, g.m, **kw)
    torch.cuda.synchronize()
    return A.cpu().numpy().astype(np.float64), mn.cpu().numpy().astype(np.float64)


def _check(x, label, tol=TOL):
    A, mn = _run(x)
    J, mref = oracle.region_jacobians(x.params, x.x_embed, x.m, phi="ssm")
    got = A.reshape(-1, A.shape[-1])
    want = np.swapaxes(J, -1, -2).reshape(-1, A.shape[-1])
    err = oracle.rel_frobenius(got, want)
    merr = oracle.rel_frobenius(mn, mref)
    _say(f"[region ssm] {label}: J^T rel err {err:.3g}, m_next rel err {merr:.3g}")
    assert np.isfinite(A).all()
    assert err <= tol, f"{label}: J^T rel err {err:.3g}"
    assert merr <= tol, f"{label}: m_next rel err {merr:.3g}"
    return A, mn


def test_region_ssm_small_matches_oracle():
    x = synth.generate_region(synth.REGION_WORKLOADS["region_small"])
    _check(x, "region_small")


@pytest.mark.parametrize("r", [16, 32, 64, 128])
@pytest.mark.parametrize("shape", [(3, 2, 200, 192, 384), (1, 1, 64, 64, 128), (2, 2, 7, 64, 128),
                                   (1, 2, 1, 128, 256)],
                         ids=["ragged", "minimal", "few_tokens", "one_token"])
def test_region_ssm_shapes(r, shape):
    """Token counts off the 128-row tile (L r a multiple of 128 or not, down
    to a single token), several column tiles of X and of D, a D that leaves a
    partial column tile."""
    B, K, L, D, X = shape
    wl = synth.RegionWorkload(f"ssm_B{B}_K{K}_L{L}_D{D}_X{X}_r{r}", B, K, L, D, X, r,
                              seed=31 + r)
    _check(synth.generate_region(wl), wl.name)


@pytest.mark.parametrize("decay", [0.0, 1.0])
def test_region_ssm_limit_decays(decay):
    """a = 0: each state is its token (no mixing); a = 1: no token enters the
    state and the block passes its input through."""
    wl = synth.RegionWorkload("ssm_limits", 2, 2, 96, 128, 256, 32, seed=37)
    x = synth.generate_region(wl)
    x.params["decay"] = torch.full_like(x.params["decay"], decay)
    _check(x, f"decay {decay}")


def test_region_ssm_decay_one_equals_token_wise_without_mlp():
    """With a = 1 the token-mixing block is the identity, as the token-wise
    block is with W1 = 0 (silu(0) = 0): the two entry points agree."""
    wl = synth.RegionWorkload("ssm_vs_mlp", 2, 3, 128, 128, 256, 32, seed=41)
    x = synth.generate_region(wl)
    x.params["decay"] = torch.ones_like(x.params["decay"])
    A1, m1 = _run(x)
    x.params["W1"] = torch.zeros_like(x.params["W1"])
    g = x.to(DEV)
    A2, m2 = binding.lbi_region_jacobians(g.params, g.x_embed, g.m)
    torch.cuda.synchronize()
    e = oracle.rel_frobenius(A1, A2.cpu().numpy().astype(np.float64))
    _say(f"[region ssm] decay 1 against the token-wise block with W1 = 0: {e:.3g}")
    assert e <= 1e-3


def test_region_ssm_deterministic_and_workspace_reuse():
    x = synth.generate_region(synth.REGION_WORKLOADS["region_small"]).to(DEV)
    need = binding.lbi_region_jacobians_ssm_workspace_bytes(2, 3, 256, 128, 256, 32)
    ws = torch.empty((need,), dtype=torch.uint8, device=DEV)
    A1, m1 = binding.lbi_region_jacobians_ssm(x.params, x.x_embed, x.m, workspace=ws)
    ws.fill_(0xFF)
    A2, m2 = binding.lbi_region_jacobians_ssm(x.params, x.x_embed, x.m, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(A1, A2) and torch.equal(m1, m2)


def _sampled_pairs(wl, n, seed):
    g = np.random.default_rng(seed)
    pairs = {(0, 0), (wl.B - 1, wl.K - 1)}
    while len(pairs) < n:
        pairs.add((int(g.integers(wl.B)), int(g.integers(wl.K))))
    return sorted(pairs)


@pytest.mark.parametrize("phi", ["ssm", "mlp"])
def test_region_paper_config_sampled_columns(phi):
    """The paper's illustrative configuration (B=8, L=2048, D=768, X=3072,
    r=64, K=16) in the launch the benchmark times: 16 sampled (sequence,
    region) pairs (the first and the last among them), two columns of J each,
    and m_next, against the oracle's forward-mode columns."""
    wl = synth.REGION_WORKLOADS["region_paper"]
    _say(f"[region {phi}] paper configuration, GPU call")
    x = synth.generate_region(wl)
    g = x.to(DEV)
    call = binding.lbi_region_jacobians_ssm if phi == "ssm" else binding.lbi_region_jacobians
    A, mn = call(g.params, g.x_embed, g.m)
    torch.cuda.synchronize()
    A = A.cpu().numpy().astype(np.float64)
    mn = mn.cpu().numpy().astype(np.float64)
    assert np.isfinite(A).all()
    got, want, mg, mw = [], [], [], []
    gen = np.random.default_rng(43)
    for b, k in _sampled_pairs(wl, 16, 47):
        cols = sorted(int(c) for c in gen.choice(wl.r, size=2, replace=False))
        c, m_ref = oracle.region_jacobian_columns(x.params, x.x_embed, x.m, b, k, cols, phi=phi)
        got.append(A[b, k][cols])  # row j of A = J^T is column j of J
        want.append(c)
        mg.append(mn[b, k])
        mw.append(m_ref)
    err = oracle.rel_frobenius(np.stack(got), np.stack(want))
    merr = oracle.rel_frobenius(np.stack(mg), np.stack(mw))
    _say(f"[region {phi}] paper configuration, 16 pairs x 2 columns: J rel err {err:.3g}, "
         f"m_next rel err {merr:.3g}")
    assert err <= TOL and merr <= TOL


@pytest.mark.parametrize("phi", ["ssm", "mlp"])
def test_region_largest_widths_sampled_columns(phi):
    """D and X at the largest sizes the entry points accept (2048, 8192), so
    that every 32-bit offset of the tile kernels reaches its largest value;
    two regions, three columns of J each and m_next against the oracle's
    forward-mode columns."""
    wl = synth.RegionWorkload(f"region_wide_{phi}", 1, 2, 40, 2048, 8192, 64, seed=53)
    _say(f"[region {phi}] D = 2048, X = 8192, GPU call")
    x = synth.generate_region(wl)
    g = x.to(DEV)
    call = binding.lbi_region_jacobians_ssm if phi == "ssm" else binding.lbi_region_jacobians
    A, mn = call(g.params, g.x_embed, g.m)
    torch.cuda.synchronize()
    A = A.cpu().numpy().astype(np.float64)
    mn = mn.cpu().numpy().astype(np.float64)
    assert np.isfinite(A).all()
    got, want, mg, mw = [], [], [], []
    for k, cols in ((0, [0, 31, 63]), (1, [5, 40, 62])):
        c, m_ref = oracle.region_jacobian_columns(x.params, x.x_embed, x.m, 0, k, cols, phi=phi)
        got.append(A[0, k][cols])
        want.append(c)
        mg.append(mn[0, k])
        mw.append(m_ref)
    err = oracle.rel_frobenius(np.stack(got), np.stack(want))
    merr = oracle.rel_frobenius(np.stack(mg), np.stack(mw))
    _say(f"[region {phi}] D = 2048, X = 8192: J rel err {err:.3g}, m_next rel err {merr:.3g}")
    assert err <= TOL and merr <= TOL
