"""Parity of the interface-Jacobian statistics kernel (lbi_matrix_norms) with
the oracle's fp64 SVD, through the C-ABI (needs a GPU).

Tolerances, from the kernel's method (include/lbi.h): the spectral norm
within 2e-5 relative (the squaring iteration contributes at most
r / (2 e 2^24) = 1.4e-6 at r = 128, float32 rounding of the Gram products and
of the final quotient the rest); the rank-normalised Frobenius norm within
1e-5 relative (a float32 sum of r^2 squares).  Both sides see the same stored
values (bf16 widened exactly).
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import binding, synth

pytestmark = pytest.mark.gpu

SPEC_TOL = 2e-5
FRO_TOL = 1e-5
DEV = torch.device("cuda:0")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _rel(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return np.abs(x - ref) / np.where(ref > 0, ref, 1.0)


def _check(M_cpu, label):
    spec, fro = binding.lbi_matrix_norms(M_cpu.to(DEV))
    torch.cuda.synchronize()
    ws, wf = oracle.matrix_norms(M_cpu)
    es, ef = _rel(spec.cpu().numpy(), ws), _rel(fro.cpu().numpy(), wf)
    assert es.max() <= SPEC_TOL, f"{label}: spectral rel err {es.max():.3g}"
    assert ef.max() <= FRO_TOL, f"{label}: Frobenius rel err {ef.max():.3g}"
    return spec, fro


@pytest.mark.parametrize("r", [16, 32, 64, 128])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("spectrum", ["uniform", "concentrated", "orthogonal"])
def test_norms_match_oracle(r, dtype, spectrum):
    # a count that leaves the last workgroup partly empty (4 matrices per
    # workgroup for r <= 64)
    n = 13 if r <= 64 else 5
    _say(f"[norms] r={r} {dtype} {spectrum} n={n}")
    x = synth.random_chain(1, n, r, dtype=dtype, seed=31 + r, spectrum=spectrum, affine=False)
    _check(x.A[0].contiguous(), f"r={r} {dtype} {spectrum}")


def _special(r):
    g = torch.Generator().manual_seed(41)
    mats = []
    mats.append(torch.zeros(r, r, dtype=torch.float64))
    u, v = torch.randn(r, generator=g, dtype=torch.float64), torch.randn(r, generator=g,
                                                                         dtype=torch.float64)
    mats.append(torch.outer(u, v))                                   # rank one
    d = torch.full((r,), 0.5, dtype=torch.float64)
    d[3] = -2.0
    d[r - 2] = 2.0                                                   # repeated largest |d|
    mats.append(torch.diag(d))
    nn = torch.zeros(r, r, dtype=torch.float64)
    nn[:2, :2] = torch.tensor([[1.0, 3.0], [0.0, 1.0]])              # non-normal block
    mats.append(nn)
    G = torch.randn(r, r, generator=g, dtype=torch.float64)
    mats.append(G * 2.0 ** -110)                                     # tiny, still normal
    mats.append(G * 2.0 ** 100)                                      # huge
    q, _ = torch.linalg.qr(torch.randn(r, r, generator=g, dtype=torch.float64))
    mats.append(q)                                                   # every sigma = 1
    return torch.stack(mats)


@pytest.mark.parametrize("r", [16, 64, 128])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_norms_special_matrices(r, dtype):
    _say(f"[norms] special r={r} {dtype}")
    store = torch.float32 if dtype == "f32" else torch.bfloat16
    M = _special(r).to(store)
    spec, fro = _check(M, f"special r={r} {dtype}")
    assert spec[0].item() == 0.0 and fro[0].item() == 0.0


def test_norms_subnormal_matrix():
    """Entries below the float32 normal range (a deep suffix product of a
    contracting chain ends there): an exact power-of-two rescaling keeps the
    result accurate for the values as stored."""
    r = 64
    g = torch.Generator().manual_seed(43)
    M = (torch.randn(2, r, r, generator=g, dtype=torch.float64) * 2.0 ** -132).to(torch.float32)
    assert (M.abs().max() < 2.0 ** -126).item() and (M != 0).any().item()
    _say("[norms] subnormal r=64")
    _check(M, "subnormal")


def test_norms_non_finite_entries_give_nan():
    r = 32
    M = torch.eye(r).repeat(3, 1, 1)
    M[0, 3, 5] = float("nan")
    M[1, 7, 1] = float("inf")
    _say("[norms] non-finite")
    spec, fro = binding.lbi_matrix_norms(M.to(DEV))
    spec, fro = spec.cpu(), fro.cpu()
    assert torch.isnan(spec[:2]).all() and torch.isnan(fro[:2]).all()
    assert spec[2].item() == pytest.approx(1.0, rel=SPEC_TOL) and fro[2].item() == 1.0


def test_norms_outputs_independent_and_deterministic():
    x = synth.random_chain(1, 9, 64, dtype="f32", seed=47, spectrum="concentrated",
                           affine=False)
    M = x.A[0].to(DEV)
    s1, f1 = binding.lbi_matrix_norms(M)
    s2, f2 = binding.lbi_matrix_norms(M)
    s3, _ = binding.lbi_matrix_norms(M, want_fro=False)
    _, f3 = binding.lbi_matrix_norms(M, want_spec=False)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2) and torch.equal(f1, f2)
    assert torch.equal(s1, s3) and torch.equal(f1, f3)
    e, _ = binding.lbi_matrix_norms(M[:0])
    assert e.numel() == 0


@pytest.mark.parametrize("r", [16, 64])
def test_suffix_norms_through_export(r):
    """Suffix statistics: lbi_matrix_norms over the P of lbi_scan_suffix_products,
    against the oracle's norms of the oracle's suffix products."""
    K = 24
    _say(f"[norms] suffix r={r}")
    x = synth.random_chain(2, K, r, dtype="f32", seed=53, spectrum="uniform", affine=False)
    P, _ = binding.lbi_scan_suffix_products(x.A.to(DEV), None, want_c=False)
    spec, fro = binding.lbi_matrix_norms(P)
    Pref, _ = oracle.suffix_composites(x.A, None)
    ws, wf = oracle.matrix_norms(Pref)
    # P carries the scan's float32 error (1e-5 relative by its own test)
    assert _rel(spec.cpu().numpy(), ws).max() <= 1e-4
    assert _rel(fro.cpu().numpy(), wf).max() <= 1e-4


def test_norms_full_size_sample():
    """The 512 x 512 stack of r = 64 interface Jacobians of the long-chain
    workload (concentrated spectrum), in the launch the benchmark times;
    64 sampled matrices against the oracle."""
    wl = synth.WORKLOADS["long_chain"]
    _say("[norms] full size long_chain A stack")
    x = synth.generate(wl, device=DEV)
    M = x.A.reshape(-1, wl.r, wl.r)
    spec, fro = binding.lbi_matrix_norms(M)
    torch.cuda.synchronize()
    idx = torch.randperm(M.shape[0], generator=torch.Generator().manual_seed(59))[:64]
    sample = M[idx.to(DEV)].cpu()
    ws, wf = oracle.matrix_norms(sample)
    assert _rel(spec[idx.to(DEV)].cpu().numpy(), ws).max() <= SPEC_TOL
    assert _rel(fro[idx.to(DEV)].cpu().numpy(), wf).max() <= FRO_TOL
    assert torch.isfinite(spec).all() and (spec > 0).all()
