"""Pins of the oracle's interface-Jacobian statistics (appendix "Interface
Jacobian Structure": spectral norm ||M||_2 and rank-normalised Frobenius norm
||M||_F / sqrt(r)) against closed forms that do not go through an SVD.

Each check takes the function under test, so that the same checks can be
shown to reject plausible mistakes (the mutants at the end).
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle


def _haar(n, rng):
    """Haar-distributed orthogonal matrix (QR of a Gaussian matrix, sign fix)."""
    z = rng.standard_normal((n, n))
    q, r = np.linalg.qr(z)
    return q * np.sign(np.diag(r))


def check_svd_construction(fn):
    """M = Q1 diag(s) Q2 with orthogonal Q1, Q2: ||M||_2 = max s, and
    ||M||_F / sqrt(r) = RMS(s), whatever the spectrum's shape."""
    rng = np.random.default_rng(5)
    for r in (16, 32, 64):
        for spectrum in ("spread", "concentrated", "flat"):
            if spectrum == "spread":
                s = rng.uniform(0.1, 2.0, r)
            elif spectrum == "concentrated":
                s = np.exp(rng.uniform(np.log(0.3), 0.0, r))
                s[3] = 2.5
            else:
                s = np.full(r, 0.7)
            M = _haar(r, rng) @ np.diag(s) @ _haar(r, rng)
            spec, fro = fn(M[None])
            assert abs(spec[0] - s.max()) <= 1e-12 * s.max(), (r, spectrum)
            assert abs(fro[0] - math.sqrt(np.mean(s * s))) <= 1e-12, (r, spectrum)


def check_diagonal(fn):
    """A diagonal matrix: ||D||_2 = max |d|, including negative entries."""
    d = np.array([0.5, -3.0, 2.0, 1.0] + [0.25] * 12)
    spec, fro = fn(np.diag(d)[None])
    assert spec[0] == 3.0
    assert abs(fro[0] - math.sqrt(np.sum(d * d) / 16)) <= 1e-15


def check_rank_one(fn):
    """u v^T: both norms are ||u|| ||v|| (the second divided by sqrt(r))."""
    u = np.arange(1, 17, dtype=np.float64)
    v = np.linspace(-2.0, 1.0, 16)
    spec, fro = fn(np.outer(u, v)[None])
    want = np.linalg.norm(u) * np.linalg.norm(v)
    assert abs(spec[0] - want) <= 1e-12 * want
    assert abs(fro[0] - want / 4.0) <= 1e-12 * want


def check_two_by_two(fn):
    """A non-normal 2 x 2 block (zero-padded to 16): sigma_max^2 =
    (S + sqrt(S^2 - 4 det^2)) / 2, S the sum of squares.  Its eigenvalues
    (1 and 1) are not its singular values."""
    a, b, c, d = 1.0, 3.0, 0.0, 1.0
    M = np.zeros((16, 16))
    M[:2, :2] = [[a, b], [c, d]]
    S = a * a + b * b + c * c + d * d
    det = a * d - b * c
    want = math.sqrt((S + math.sqrt(S * S - 4 * det * det)) / 2)
    spec, _ = fn(M[None])
    assert abs(spec[0] - want) <= 1e-14 * want


def check_scaling_and_transpose(fn):
    """||alpha M|| = |alpha| ||M|| and ||M^T||_2 = ||M||_2."""
    rng = np.random.default_rng(7)
    M = rng.standard_normal((32, 32))
    s1, f1 = fn(M[None])
    s2, f2 = fn((-2.5 * M)[None])
    s3, f3 = fn(M.T[None])
    assert abs(s2[0] - 2.5 * s1[0]) <= 1e-12 * s2[0]
    assert abs(f2[0] - 2.5 * f1[0]) <= 1e-12 * f2[0]
    assert abs(s3[0] - s1[0]) <= 1e-12 * s1[0] and abs(f3[0] - f1[0]) <= 1e-12 * f1[0]


def check_zero_and_permutation(fn):
    """Zero matrix: 0 and 0; a scaled permutation: |alpha| and |alpha|."""
    spec, fro = fn(np.zeros((2, 16, 16)))
    assert np.all(spec == 0.0) and np.all(fro == 0.0)
    perm = np.eye(16)[np.random.default_rng(3).permutation(16)] * -0.75
    spec, fro = fn(perm[None])
    assert abs(spec[0] - 0.75) <= 1e-15 and abs(fro[0] - 0.75) <= 1e-15


CHECKS = [check_svd_construction, check_diagonal, check_rank_one, check_two_by_two,
          check_scaling_and_transpose, check_zero_and_permutation]


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_oracle_matrix_norms_pinned(check):
    check(oracle.matrix_norms)


def test_matrix_norms_keeps_leading_shape_and_widens_bf16_exactly():
    g = torch.Generator().manual_seed(11)
    M = torch.randn((3, 2, 16, 16), generator=g).to(torch.bfloat16)
    spec, fro = oracle.matrix_norms(M)
    assert spec.shape == (3, 2) and fro.shape == (3, 2)
    s64, f64 = oracle.matrix_norms(M.to(torch.float64))
    assert np.array_equal(spec, s64) and np.array_equal(fro, f64)


def test_suffix_norms_of_orthogonal_chain_are_one():
    """The suffix products of orthogonal matrices are orthogonal: norm 1."""
    rng = np.random.default_rng(9)
    A = np.stack([_haar(16, rng) for _ in range(6)])[None]
    P, _ = oracle.suffix_composites(A, None)
    spec, fro = oracle.matrix_norms(P)
    assert np.allclose(spec, 1.0, atol=1e-13) and np.allclose(fro, 1.0, atol=1e-13)


# --- plausible mistakes each check set must reject ---------------------------

def _mut_smallest(M):
    a = np.asarray(M, dtype=np.float64)
    s = np.linalg.svd(a, compute_uv=False)
    return s[..., -1], np.sqrt(np.sum(a * a, axis=(-2, -1)) / a.shape[-1])


def _mut_no_rank_normalisation(M):
    spec, fro = oracle.matrix_norms(M)
    return spec, fro * math.sqrt(np.asarray(M).shape[-1])


def _mut_eigenvalue(M):
    a = np.asarray(M, dtype=np.float64)
    lam = np.abs(np.linalg.eigvals(a)).max(axis=-1)
    return lam, oracle.matrix_norms(M)[1]


def _mut_squared(M):
    spec, fro = oracle.matrix_norms(M)
    return spec * spec, fro


def _mut_rms_over_all_entries(M):
    a = np.asarray(M, dtype=np.float64)
    spec, _ = oracle.matrix_norms(M)
    return spec, np.sqrt(np.mean(a * a, axis=(-2, -1)))


@pytest.mark.parametrize("mutant", [_mut_smallest, _mut_no_rank_normalisation, _mut_eigenvalue,
                                    _mut_squared, _mut_rms_over_all_entries],
                         ids=lambda m: m.__name__)
def test_norm_pins_reject_mutants(mutant):
    failed = 0
    for check in CHECKS:
        try:
            check(mutant)
        except AssertionError:
            failed += 1
    assert failed > 0, f"{mutant.__name__} passed every pin"
