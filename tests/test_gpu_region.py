"""Parity of Phase 1 (lbi_region_jacobians: the interface Jacobians of the
synthetic region map) with the fp64 autograd oracle, through the C-ABI (needs a
GPU).

Tolerance: the products take bf16 operands (weights and x_embed are stored in
bf16; x_embed + d and the tangent intermediates are rounded to bf16 where they
feed a product) with fp32 accumulation, so the relative Frobenius error of
J^T is held to the bf16 bound of the scan, 2e-2 (about 3e-3 is expected from
a few roundings of 2^-9).  With alpha = 0 no bf16 rounding reaches the
result (J is the fp32 LayerNorm Jacobian), so it is held to 1e-5.
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
    A, mn = binding.lbi_region_jacobians(g.params, g.x_embed, g.m, **kw)
    torch.cuda.synchronize()
    return A.cpu().numpy().astype(np.float64), mn.cpu().numpy().astype(np.float64)


def _check(x, label, tol=TOL, pairs=None):
    A, mn = _run(x)
    J, mref = oracle.region_jacobians(x.params, x.x_embed, x.m, pairs=pairs)
    sel = pairs if pairs is not None else [(b, k) for b in range(x.m.shape[0])
                                           for k in range(x.m.shape[1])]
    got = np.stack([A[b, k] for b, k in sel])
    want = np.stack([J[b, k].T for b, k in sel])
    err = oracle.rel_frobenius(got, want)
    merr = oracle.rel_frobenius(np.stack([mn[b, k] for b, k in sel]),
                                np.stack([mref[b, k] for b, k in sel]))
    _say(f"[region] {label}: J^T rel err {err:.3g}, m_next rel err {merr:.3g}")
    assert err <= tol, f"{label}: J^T rel err {err:.3g}"
    assert merr <= tol, f"{label}: m_next rel err {merr:.3g}"
    return A, mn


def test_region_small_matches_oracle():
    x = synth.generate_region(synth.REGION_WORKLOADS["region_small"])
    _check(x, "region_small")


@pytest.mark.parametrize("r", [16, 32, 64, 128])
@pytest.mark.parametrize("shape", [(3, 2, 200, 192, 384), (1, 1, 64, 64, 128), (2, 2, 7, 64, 128),
                                   (1, 2, 1, 128, 256)],
                         ids=["ragged", "minimal", "few_tokens", "one_token"])
def test_region_shapes(r, shape):
    """Token counts off the 128-row tile (down to a single token, whose tile
    is all rows past L but one), several column tiles of X, three 64-wide k
    blocks, B r off the 128-row tile."""
    B, K, L, D, X = shape
    wl = synth.RegionWorkload(f"region_B{B}_K{K}_L{L}_D{D}_X{X}_r{r}", B, K, L, D, X, r,
                              seed=11 + r)
    _check(synth.generate_region(wl), wl.name)


def test_region_alpha_zero_is_layernorm_exactly():
    wl = synth.RegionWorkload("region_alpha0", 2, 2, 128, 128, 256, 32, seed=13)
    x = synth.generate_region(wl)
    x.params["alpha"] = torch.zeros_like(x.params["alpha"])
    _check(x, "alpha = 0", tol=1e-5)


def test_region_feeds_the_scan():
    """Phase 1 -> Phase 2: the A that lbi_region_jacobians writes is the scan's
    operand; the adjoints match the oracle's recurrence over the oracle's J^T."""
    wl = synth.RegionWorkload("region_chain", 2, 6, 128, 128, 256, 32, seed=17)
    x = synth.generate_region(wl)
    g = x.to(DEV)
    A, _ = binding.lbi_region_jacobians(g.params, g.x_embed, g.m, want_m_next=False)
    lamK = torch.randn((wl.B, wl.r), generator=torch.Generator().manual_seed(19))
    lam = binding.lbi_scan_backward(A, None, lamK.to(DEV)).cpu().numpy()
    J, _ = oracle.region_jacobians(x.params, x.x_embed, x.m)
    ref = oracle.recurrence(np.ascontiguousarray(np.swapaxes(J, -1, -2)), None,
                            lamK.double().numpy())
    err = oracle.rel_frobenius(lam, ref)
    _say(f"[region] phase 1 -> scan rel err {err:.3g}")
    assert err <= TOL


def test_region_deterministic_and_workspace_reuse():
    x = synth.generate_region(synth.REGION_WORKLOADS["region_small"]).to(DEV)
    need = binding.lbi_region_jacobians_workspace_bytes(2, 3, 256, 128, 256, 32)
    ws = torch.empty((need,), dtype=torch.uint8, device=DEV)
    A1, m1 = binding.lbi_region_jacobians(x.params, x.x_embed, x.m, workspace=ws)
    ws.fill_(0xFF)
    A2, m2 = binding.lbi_region_jacobians(x.params, x.x_embed, x.m, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(A1, A2) and torch.equal(m1, m2)


def test_region_paper_config_sampled():
    """The paper's illustrative configuration (B=8, L=2048, D=768, X=3072,
    r=64, K=16) in the launch the benchmark times; two (sequence, region)
    pairs against the oracle."""
    wl = synth.REGION_WORKLOADS["region_paper"]
    _say("[region] paper configuration")
    x = synth.generate_region(wl)
    _check(x, "region_paper", pairs=[(0, 0), (wl.B - 1, wl.K - 1)])
