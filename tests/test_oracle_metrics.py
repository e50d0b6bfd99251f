"""Pins of the oracle's error metrics, the checker behind every parity test.

``oracle.rel_frobenius(x, ref)`` is ||x - ref||_F / ||ref||_F over the whole
compared output (the absolute error ||x - ref||_F when ref is all zero), and
``oracle.per_chain_rel_frobenius`` is the same per chain (leading axis).
These definitions are the relative-Frobenius parity metric stated for the
scan.  The values below are worked by hand from Pythagorean triples, so none
of them restates the code: a swapped ratio, a missing square root, a sum over
the wrong axis or a maximum in place of the norm each fails one of them
(``test_metric_pins_reject_mutants`` plants those mistakes in stand-ins).
"""
import numpy as np
import pytest

import oracle


# ----------------------------------------------------------------------------
# the checks, each taking (rel, per_chain) implementations
# ----------------------------------------------------------------------------

def check_three_four_five(rel, per):
    # ref = (6, 8): norm 10; x - ref = (3, 4): norm 5; ratio 1/2
    assert rel(np.array([9.0, 12.0]), np.array([6.0, 8.0])) == pytest.approx(0.5, rel=1e-15)
    # ref = (5, 12): norm 13; x - ref = (-5, 0): norm 5; ratio 5/13
    assert rel(np.array([0.0, 12.0]), np.array([5.0, 12.0])) == pytest.approx(5.0 / 13.0,
                                                                                rel=1e-15)


def check_matrix_shape_is_flattened(rel, per):
    # a 2 x 2 x 2 block: ref entries 1 (norm sqrt(8)), error 1 in two entries
    # (norm sqrt(2)): ratio sqrt(2) / sqrt(8) = 1/2
    ref = np.ones((2, 2, 2))
    x = ref.copy()
    x[0, 1, 0] += 1.0
    x[1, 0, 1] -= 1.0
    assert rel(x, ref) == pytest.approx(0.5, rel=1e-15)


def check_zero_reference_is_absolute(rel, per):
    # ||ref|| = 0: the absolute error, here ||(3, 4)|| = 5
    assert rel(np.array([3.0, 4.0]), np.zeros(2)) == pytest.approx(5.0, rel=1e-15)
    assert rel(np.zeros(3), np.zeros(3)) == 0.0


def check_exact_match_is_zero(rel, per):
    ref = np.array([[1.5, -2.0], [7.0, 0.25]])
    assert rel(ref.copy(), ref) == 0.0
    assert np.all(per(ref.copy(), ref) == 0.0)


def check_per_chain_values_and_axis(rel, per):
    # chain 0: ref (6, 8, 0, 0), error (3, 4, 0, 0) -> 1/2
    # chain 1: ref (0, 0, 5, 12), error (0, 0, 0, 0) -> 0
    # chain 2: ref (1, 0, 0, 0) (norm 1), error (0, 0, 8, 15) (norm 17) -> 17
    ref = np.array([[6.0, 8.0, 0.0, 0.0], [0.0, 0.0, 5.0, 12.0], [1.0, 0.0, 0.0, 0.0]])
    err = np.array([[3.0, 4.0, 0.0, 0.0], [0.0, 0.0, 0.0, 0.0], [0.0, 0.0, 8.0, 15.0]])
    got = per(ref + err, ref)
    assert got.shape == (3,)
    np.testing.assert_allclose(got, [0.5, 0.0, 17.0], rtol=1e-15, atol=0)
    # the whole-output figure is not the mean of the chains: sqrt(25 + 289) /
    # sqrt(100 + 169 + 1)
    assert rel(ref + err, ref) == pytest.approx(np.sqrt(314.0 / 270.0), rel=1e-15)


def check_per_chain_multidim_and_zero_chain(rel, per):
    # chains of shape (2, 2): chain 0 ref all 2 (norm 4), error one entry 2 ->
    # 1/2; chain 1 ref zero, error (0, 3; 4, 0) -> absolute 5
    ref = np.zeros((2, 2, 2))
    ref[0] = 2.0
    x = ref.copy()
    x[0, 1, 1] += 2.0
    x[1, 0, 1] = 3.0
    x[1, 1, 0] = 4.0
    np.testing.assert_allclose(per(x, ref), [0.5, 5.0], rtol=1e-15, atol=0)


CHECKS = [check_three_four_five, check_matrix_shape_is_flattened,
          check_zero_reference_is_absolute, check_exact_match_is_zero,
          check_per_chain_values_and_axis, check_per_chain_multidim_and_zero_chain]


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_oracle_metrics_pinned(check):
    check(oracle.rel_frobenius, oracle.per_chain_rel_frobenius)


def test_metrics_accept_float32_and_lists():
    # inputs are widened to float64 before the norms
    x = np.array([9.0, 12.0], dtype=np.float32)
    assert oracle.rel_frobenius(x, np.array([6.0, 8.0])) == pytest.approx(0.5, rel=1e-15)
    assert oracle.rel_frobenius([9.0, 12.0], [6.0, 8.0]) == pytest.approx(0.5, rel=1e-15)


# ----------------------------------------------------------------------------
# plausible mistakes, planted in stand-ins; every one must fail a check
# ----------------------------------------------------------------------------

def _norm(a):
    return float(np.sqrt(np.sum(np.asarray(a, dtype=np.float64) ** 2)))


def _rel_swapped(x, ref):
    num, den = _norm(np.asarray(x) - np.asarray(ref)), _norm(ref)
    return den / num if num > 0 else den


def _rel_no_sqrt(x, ref):
    num = float(np.sum((np.asarray(x) - np.asarray(ref)) ** 2))
    den = float(np.sum(np.asarray(ref) ** 2))
    return num / den if den > 0 else num


def _rel_max(x, ref):
    num = float(np.max(np.abs(np.asarray(x) - np.asarray(ref))))
    den = float(np.max(np.abs(np.asarray(ref))))
    return num / den if den > 0 else num


def _rel_relative_to_x(x, ref):
    num, den = _norm(np.asarray(x) - np.asarray(ref)), _norm(x)
    return num / den if den > 0 else num


def _rel_zero_ref_nan(x, ref):
    num, den = _norm(np.asarray(x) - np.asarray(ref)), _norm(ref)
    return num / den if den > 0 else float("nan")


def _per_wrong_axis(x, ref):
    x = np.asarray(x, dtype=np.float64).reshape(x.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    num = np.linalg.norm(x - ref, axis=0)
    den = np.linalg.norm(ref, axis=0)
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), num)


def _per_last_axis_only(x, ref):
    # norms over the last axis, then the first row of each chain
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.linalg.norm(x - ref, axis=-1)
    den = np.linalg.norm(ref, axis=-1)
    out = np.where(den > 0, num / np.where(den > 0, den, 1.0), num)
    return out.reshape(x.shape[0], -1)[:, 0]


def _per_mean_of_rows(x, ref):
    x = np.asarray(x, dtype=np.float64).reshape(x.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    return np.abs(x - ref).mean(axis=1) / np.maximum(np.abs(ref).mean(axis=1), 1e-300)


MUTANTS = [
    (_rel_swapped, oracle.per_chain_rel_frobenius),
    (_rel_no_sqrt, oracle.per_chain_rel_frobenius),
    (_rel_max, oracle.per_chain_rel_frobenius),
    (_rel_relative_to_x, oracle.per_chain_rel_frobenius),
    (_rel_zero_ref_nan, oracle.per_chain_rel_frobenius),
    (oracle.rel_frobenius, _per_wrong_axis),
    (oracle.rel_frobenius, _per_last_axis_only),
    (oracle.rel_frobenius, _per_mean_of_rows),
]


@pytest.mark.parametrize("rel,per", MUTANTS,
                         ids=[f"{a.__name__}-{b.__name__}" for a, b in MUTANTS])
def test_metric_pins_reject_mutants(rel, per):
    failed = []
    for check in CHECKS:
        try:
            check(rel, per)
        except (AssertionError, ValueError, IndexError):
            failed.append(check.__name__)
    assert failed, "no pin catches this mutant"
