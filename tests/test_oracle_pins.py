"""Pins of the CPU oracle against facts that do not come from the oracle.

Each check would fail under a plausible mistake in the oracle: a transposed
A, a dropped or misplaced affine term, an index shifted by one slot, the chain
walked in the wrong direction.  ``test_pins_reject_mutants`` runs those
mistakes (planted in Python stand-ins, on the CPU) through the same checks.

Sources of truth, all from the paper's Scan Formulation section:
  * Theorem "Bounded-Interface Backpropagation" -- recurrence
    mbar_k = J_k^T mbar_{k+1} and the product form with the product ordered
    J_k^T J_{k+1}^T ... J_{K-1}^T, empty product = identity.
  * Proposition "Scan Formulation of Backpropagation" -- suffix products,
    combine associativity.
  * torch autograd through a nonlinear region chain m_{k+1} = R_k(m_k), the
    chain rule the theorem rests on (an implementation independent of ours).
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng(20260512)


# ----------------------------------------------------------------------------
# exact rational reference: the product form, written out
# ----------------------------------------------------------------------------

def _fmat(a):
    return [[Fraction(int(v)) for v in row] for row in a]


def _fvec(v):
    return [Fraction(int(x)) for x in v]


def _matmul(X, Y):
    n, m, p = len(X), len(Y), len(Y[0])
    return [[sum((X[i][k] * Y[k][j] for k in range(m)), Fraction(0)) for j in range(p)]
            for i in range(n)]


def _matvec(X, v):
    return [sum((X[i][k] * v[k] for k in range(len(v))), Fraction(0)) for i in range(len(X))]


def _eye(r):
    return [[Fraction(int(i == j)) for j in range(r)] for i in range(r)]


def product_form(A, b, lamK):
    """lambda_j = (A_j ... A_{K-1}) lambda_K + sum_{i>=j} (A_j ... A_{i-1}) b_i, exactly.

    A[K][r][r], b[K][r] or None, lamK[r] (integers).  Returns (lam, P, c) with
    P_j, c_j the suffix composites of slot j.
    """
    K = len(A)
    r = len(lamK)
    Af = [_fmat(a) for a in A]
    bf = [_fvec(x) for x in b] if b is not None else [[Fraction(0)] * r for _ in range(K)]
    lk = _fvec(lamK)
    lam, Ps, cs = [], [], []
    for j in range(K):
        # P_j: the ordered product A_j A_{j+1} ... A_{K-1}
        P = _eye(r)
        for t in range(j, K):
            P = _matmul(P, Af[t])
        # c_j: sum over i >= j of (A_j ... A_{i-1}) b_i
        c = [Fraction(0)] * r
        for i in range(j, K):
            M = _eye(r)
            for t in range(j, i):
                M = _matmul(M, Af[t])
            c = [x + y for x, y in zip(c, _matvec(M, bf[i]))]
        lam.append([x + y for x, y in zip(_matvec(P, lk), c)])
        Ps.append(P)
        cs.append(c)
    return lam, Ps, cs


def _int_case(K, r, affine=True, lo=-3, hi=3):
    A = RNG.integers(lo, hi + 1, size=(1, K, r, r)).astype(np.float64)
    b = RNG.integers(lo, hi + 1, size=(1, K, r)).astype(np.float64) if affine else None
    lamK = RNG.integers(lo, hi + 1, size=(1, r)).astype(np.float64)
    return A, b, lamK


# ----------------------------------------------------------------------------
# the checks, written against an arbitrary candidate implementation
# ----------------------------------------------------------------------------

def check_bruteforce(fn):
    """Exact equality with the rational product form on small integer chains."""
    for K in (1, 2, 3, 4, 6):
        for r in (1, 2, 3, 4):
            for affine in (True, False):
                A, b, lamK = _int_case(K, r, affine)
                got = fn(A, b, lamK)[0]
                lam, _, _ = product_form(A[0], None if b is None else b[0], lamK[0])
                want = np.array([[float(x) for x in row] for row in lam])
                if not np.array_equal(got, want):
                    return False
    return True


def check_closed_forms(fn):
    """K = 1, 2, 3 expanded by hand from the product form (numpy matmul)."""
    for r in (2, 3, 5):
        A, b, lamK = _int_case(3, r)
        A0, A1, A2 = A[0]
        b0, b1, b2 = b[0]
        l3 = lamK[0]
        lam = fn(A, b, lamK)[0]
        want = [
            A0 @ A1 @ A2 @ l3 + A0 @ A1 @ b2 + A0 @ b1 + b0,
            A1 @ A2 @ l3 + A1 @ b2 + b1,
            A2 @ l3 + b2,
        ]
        if not all(np.array_equal(lam[j], want[j]) for j in range(3)):
            return False
        # K = 1 and K = 2 on their own
        if not np.array_equal(fn(A[:, 2:], b[:, 2:], lamK)[0][0], A2 @ l3 + b2):
            return False
        lam2 = fn(A[:, 1:], b[:, 1:], lamK)[0]
        if not np.array_equal(lam2[0], A1 @ A2 @ l3 + A1 @ b2 + b1):
            return False
    return True


def _region_chain(K, r, seed):
    """A nonlinear region chain m_{k+1} = tanh(W_k m_k + u_k) + 0.5 m_k."""
    g = torch.Generator().manual_seed(seed)
    W = torch.randn((K, r, r), generator=g, dtype=torch.float64) / np.sqrt(r)
    u = torch.randn((K, r), generator=g, dtype=torch.float64)
    m0 = torch.randn((r,), generator=g, dtype=torch.float64)
    lamK = torch.randn((r,), generator=g, dtype=torch.float64)
    bdir = torch.randn((K, r), generator=g, dtype=torch.float64)

    def region(k, m):
        return torch.tanh(W[k] @ m + u[k]) + 0.5 * m

    return W, u, m0, lamK, bdir, region


def check_autograd(fn):
    """dL/dm_j from torch autograd equals the candidate's lambda_j.

    L = lamK . m_K + sum_j bdir_j . m_j, so that dL/dm_K = lamK and each m_j
    also feeds the loss directly with gradient bdir_j (the affine term).  The
    interface Jacobians J_k = d m_{k+1}/d m_k come from
    torch.autograd.functional.jacobian; the candidate receives A_k = J_k^T.
    """
    for K, r, seed in ((1, 3, 1), (4, 5, 2), (9, 8, 3)):
        W, u, m0, lamK, bdir, region = _region_chain(K, r, seed)
        ms = [m0.clone().requires_grad_(True)]
        for k in range(K):
            mk = region(k, ms[-1])
            mk.retain_grad()
            ms.append(mk)
        L = lamK @ ms[K] + sum(bdir[j] @ ms[j] for j in range(K))
        L.backward()
        grads = np.stack([ms[j].grad.numpy() for j in range(K)])
        J = np.stack([
            torch.autograd.functional.jacobian(lambda m, k=k: region(k, m), ms[k].detach()).numpy()
            for k in range(K)
        ])  # J[k] = d m_{k+1} / d m_k, shape r x r
        A = np.ascontiguousarray(np.transpose(J, (0, 2, 1)))[None]
        got = fn(A, bdir.numpy()[None], lamK.numpy()[None])[0]
        if not np.allclose(got, grads, rtol=1e-12, atol=1e-12):
            return False
    return True


def check_identity(fn):
    """A_j = I, b = 0  =>  lambda_j = lambda_K for every j, bit for bit."""
    for K, r in ((1, 4), (7, 16), (33, 64)):
        A = np.broadcast_to(np.eye(r), (2, K, r, r)).copy()
        lamK = RNG.standard_normal((2, r))
        got = fn(A, None, lamK)
        if not np.array_equal(got, np.broadcast_to(lamK[:, None, :], got.shape)):
            return False
    return True


def check_zero_A(fn):
    """A = 0  =>  lambda_j = b_j exactly."""
    A = np.zeros((3, 5, 6, 6))
    b = RNG.standard_normal((3, 5, 6))
    lamK = RNG.standard_normal((3, 6))
    return np.array_equal(fn(A, b, lamK), b)


def check_diagonal(fn):
    """Diagonal A: r independent scalar recurrences with a closed-form sum."""
    B, K, r = 2, 12, 5
    d = RNG.uniform(-1.2, 1.2, size=(B, K, r))
    A = np.zeros((B, K, r, r))
    idx = np.arange(r)
    A[:, :, idx, idx] = d
    b = RNG.standard_normal((B, K, r))
    lamK = RNG.standard_normal((B, r))
    want = np.zeros((B, K, r))
    for j in range(K):
        prod = np.prod(d[:, j:K], axis=1)  # prod_{t=j}^{K-1} d_t
        acc = prod * lamK
        for s in range(j, K):
            acc = acc + np.prod(d[:, j:s], axis=1) * b[:, s]  # empty product = 1
        want[:, j] = acc
    return np.allclose(fn(A, b, lamK), want, rtol=1e-12, atol=1e-12)


def _haar(n, rng):
    Q, R = np.linalg.qr(rng.standard_normal((n, n)))
    return Q * np.sign(np.diag(R))


def check_orthogonal_norm(fn):
    """Orthogonal A, b = 0  =>  ||lambda_j||_2 = ||lambda_K||_2 for every j."""
    rng = np.random.default_rng(7)
    B, K, r = 2, 96, 16
    A = np.stack([np.stack([_haar(r, rng) for _ in range(K)]) for _ in range(B)])
    lamK = rng.standard_normal((B, r))
    got = fn(A, None, lamK)
    ratio = np.linalg.norm(got, axis=-1) / np.linalg.norm(lamK, axis=-1)[:, None]
    # orthogonality fails only by rounding, which drifts the norm no further
    if not np.allclose(ratio, 1.0, rtol=1e-12, atol=0):
        return False
    # and the direction does change: A is not the identity
    return not np.allclose(got[:, 0], lamK, atol=1e-3)


def check_linearity(fn):
    """Superposition in (b, lambda_K) and exact power-of-two homogeneity."""
    B, K, r = 3, 10, 7
    A = RNG.standard_normal((B, K, r, r)) / np.sqrt(r)
    b = RNG.standard_normal((B, K, r))
    lamK = RNG.standard_normal((B, r))
    full = fn(A, b, lamK)
    part = fn(A, np.zeros_like(b), lamK) + fn(A, b, np.zeros_like(lamK))
    if not np.allclose(full, part, rtol=1e-12, atol=1e-12):
        return False
    return np.array_equal(fn(A, 4.0 * b, 4.0 * lamK), 4.0 * full)


ALL_CHECKS = (check_bruteforce, check_closed_forms, check_autograd, check_identity,
              check_zero_A, check_diagonal, check_orthogonal_norm, check_linearity)


def _oracle_fn(A, b, lamK):
    return oracle.recurrence(A, b, lamK)


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_recurrence_pinned(check):
    assert check(_oracle_fn)


def _suffix_fn(A, b, lamK):
    """lambda from the oracle's suffix composites: P_j lambda_K + c_j."""
    P, c = oracle.suffix_composites(A, b)
    return np.einsum("bjik,bk->bji", P, np.asarray(lamK, dtype=np.float64)) + c


@pytest.mark.parametrize("check", (check_bruteforce, check_closed_forms, check_autograd,
                                   check_zero_A, check_linearity),
                         ids=lambda c: c.__name__)
def test_oracle_suffix_composites_pinned(check):
    assert check(_suffix_fn)


def test_suffix_composites_exact_products():
    """The oracle's P_j and c_j equal the written-out products, exactly."""
    for K, r in ((1, 3), (3, 2), (5, 3), (6, 4)):
        A, b, lamK = _int_case(K, r)
        P, c = oracle.suffix_composites(A, b)
        _, Ps, cs = product_form(A[0], b[0], lamK[0])
        for j in range(K):
            assert np.array_equal(P[0, j], np.array([[float(x) for x in row] for row in Ps[j]]))
            assert np.array_equal(c[0, j], np.array([float(x) for x in cs[j]]))


def _combine(x, y):
    """(A, b) o (A', b') = (A A', A b' + b): apply y first, then x."""
    (A, b), (A2, b2) = x, y
    return _matmul(A, A2), [s + t for s, t in zip(_matvec(A, b2), b)]


def test_combine_associative_and_identity():
    """The combine is associative and (I, 0) is a two-sided identity (exact)."""
    r = 3
    for _ in range(5):
        els = []
        for _ in range(3):
            A, b, _ = _int_case(1, r)
            els.append((_fmat(A[0, 0]), _fvec(b[0, 0])))
        x, y, z = els
        assert _combine(_combine(x, y), z) == _combine(x, _combine(y, z))
        e = (_eye(r), [Fraction(0)] * r)
        assert _combine(e, x) == x and _combine(x, e) == x


def test_chunked_composition_matches_whole_chain():
    """The composite of a whole chain is the combine of the composites of its
    two halves -- the property a blocked (two-level) scan rests on."""
    B, K, r = 2, 12, 6
    A = RNG.standard_normal((B, K, r, r)) / np.sqrt(r)
    b = RNG.standard_normal((B, K, r))
    P, c = oracle.suffix_composites(A, b)
    for m in (1, 5, 11):
        PL, cL = oracle.suffix_composites(A[:, :m], b[:, :m])
        PR, cR = oracle.suffix_composites(A[:, m:], b[:, m:])
        P0 = np.einsum("bik,bkn->bin", PL[:, 0], PR[:, 0])
        c0 = np.einsum("bik,bk->bi", PL[:, 0], cR[:, 0]) + cL[:, 0]
        np.testing.assert_allclose(P0, P[:, 0], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(c0, c[:, 0], rtol=1e-12, atol=1e-13)


def test_oracle_widens_storage_exactly():
    """fp32 and bf16 inputs are widened exactly: the same values given as
    fp64 produce the same bits."""
    B, K, r = 3, 6, 8
    A64 = RNG.standard_normal((B, K, r, r)) / np.sqrt(r)
    b64 = RNG.standard_normal((B, K, r))
    l64 = RNG.standard_normal((B, r))
    for dt in (torch.float32, torch.bfloat16):
        A = torch.from_numpy(A64).to(dt)
        b = torch.from_numpy(b64).to(dt)
        lk = torch.from_numpy(l64).to(dt)
        got = oracle.recurrence(A, b, lk)
        want = oracle.recurrence(A.double(), b.double(), lk.double())
        assert np.array_equal(got, want)


def test_oracle_thread_count_does_not_change_bits():
    B, K, r = 9, 7, 16
    A = RNG.standard_normal((B, K, r, r)) / np.sqrt(r)
    b = RNG.standard_normal((B, K, r))
    lamK = RNG.standard_normal((B, r))
    one = oracle.recurrence(A, b, lamK, nthreads=1)
    many = oracle.recurrence(A, b, lamK, nthreads=4)
    assert np.array_equal(one, many)


def test_oracle_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oracle.recurrence(np.zeros((2, 3, 4, 5)), None, np.zeros((2, 4)))
    with pytest.raises(ValueError):
        oracle.recurrence(np.zeros((2, 3, 4, 4)), None, np.zeros((2, 5)))
    with pytest.raises(ValueError):
        oracle.recurrence(np.zeros((2, 3, 4, 4)), np.zeros((2, 3, 5)), np.zeros((2, 4)))


# ----------------------------------------------------------------------------
# the pins catch plausible mistakes (planted in CPU stand-ins, never on a GPU)
# ----------------------------------------------------------------------------

def _mut_transposed(A, b, lamK):
    return oracle.recurrence(np.ascontiguousarray(np.swapaxes(A, -1, -2)), b, lamK)


def _mut_dropped_b(A, b, lamK):
    return oracle.recurrence(A, None, lamK)


def _mut_b_inside(A, b, lamK):
    # lambda_j = A_j (lambda_{j+1} + b_j): the affine term on the wrong side
    A = np.asarray(A, dtype=np.float64)
    lam = np.asarray(lamK, dtype=np.float64).copy()
    out = np.zeros(A.shape[:3])
    for j in range(A.shape[1] - 1, -1, -1):
        x = lam + (0 if b is None else np.asarray(b)[:, j])
        lam = np.einsum("bik,bk->bi", A[:, j], x)
        out[:, j] = lam
    return out


def _mut_shifted(A, b, lamK):
    # output slot j holds lambda_{j+1} (an off-by-one in the store)
    full = oracle.recurrence(A, b, lamK)
    out = np.empty_like(full)
    out[:, :-1] = full[:, 1:]
    out[:, -1] = np.asarray(lamK, dtype=np.float64)
    return out


def _mut_forward(A, b, lamK):
    # walks the chain from slot 0 upwards instead of from slot K-1 down
    return oracle.recurrence(np.ascontiguousarray(np.asarray(A)[:, ::-1]),
                             None if b is None else np.ascontiguousarray(np.asarray(b)[:, ::-1]),
                             lamK)[:, ::-1]


@pytest.mark.parametrize("mutant", (_mut_transposed, _mut_dropped_b, _mut_b_inside,
                                    _mut_shifted, _mut_forward),
                         ids=lambda f: f.__name__)
def test_pins_reject_mutants(mutant):
    failed = [c.__name__ for c in ALL_CHECKS if not c(mutant)]
    assert failed, f"no pin catches {mutant.__name__}"
    # the two strongest pins catch every planted mistake on their own
    assert "check_bruteforce" in failed or "check_autograd" in failed
