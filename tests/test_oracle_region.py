"""Pins of the oracle's Phase 1 (region-Jacobian construction for the synthetic
bounded-interface region map of Eq. "concrete-region-arch") that do not go
through torch autograd: central finite differences, the closed-form
LayerNorm Jacobian, LayerNorm's invariants, and a closed form of the whole
Jacobian when the region MLP is switched off.
"""
from __future__ import annotations

import copy
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import synth

WL = synth.RegionWorkload("pin", B=2, K=2, L=16, D=32, X=48, r=16, seed=9)


def _inputs(**override):
    x = synth.generate_region(WL)
    p = {k: v.clone() for k, v in x.params.items()}
    for name, val in override.items():
        p[name] = val
    return p, x.x_embed, x.m


def _silu(t):
    return t / (1.0 + np.exp(-t))


def _dsilu(t):
    s = 1.0 / (1.0 + np.exp(-t))
    return s * (1.0 + t * (1.0 - s))


def _ln_jacobian(z, gamma):
    """d LN(z) / dz = diag(gamma) / sigma (I - 11^T / r - zhat zhat^T / r)."""
    r = z.shape[0]
    mu = z.mean()
    sig = math.sqrt(((z - mu) ** 2).mean() + oracle.LN_EPS)
    zh = (z - mu) / sig
    return (gamma[:, None] / sig) * (np.eye(r) - 1.0 / r - np.outer(zh, zh) / r)


def check_finite_differences(fn_jac):
    p, x, m = _inputs()
    J, _ = fn_jac(p, x, m)
    h = 1e-5
    for b in range(WL.B):
        for k in range(WL.K):
            m0 = m[b, k].to(torch.float64)
            fd = np.empty((WL.r, WL.r))
            for j in range(WL.r):
                e = torch.zeros(WL.r, dtype=torch.float64)
                e[j] = h
                up = oracle.region_forward(p, k, x[b], m0 + e).numpy()
                dn = oracle.region_forward(p, k, x[b], m0 - e).numpy()
                fd[:, j] = (up - dn) / (2 * h)
            assert np.abs(fd - J[b, k]).max() <= 1e-7 * max(1.0, np.abs(fd).max())


def check_alpha_zero_is_layernorm(fn_jac):
    """alpha = 0: the region only renormalises m, J = the LayerNorm Jacobian at m."""
    p, x, m = _inputs(alpha=torch.zeros(WL.K))
    J, mn = fn_jac(p, x, m)
    for b in range(WL.B):
        for k in range(WL.K):
            z = m[b, k].double().numpy()
            g = p["gamma"][k].double().numpy()
            assert np.abs(J[b, k] - _ln_jacobian(z, g)).max() <= 1e-12
            mu, sig = z.mean(), math.sqrt(z.var() + oracle.LN_EPS)
            want = g * (z - mu) / sig + p["beta"][k].double().numpy()
            assert np.abs(mn[b, k] - want).max() <= 1e-12


def check_layernorm_invariants(fn_jac):
    """LN's output (minus beta, over gamma) has zero mean whatever z is, so for
    every column j: sum_i J_ij / gamma_i = 0.  (Its norm is fixed only with a
    zero epsilon; the alpha = 0 closed form pins that part.)"""
    p, x, m = _inputs()
    J, _ = fn_jac(p, x, m)
    for b in range(WL.B):
        for k in range(WL.K):
            g = p["gamma"][k].double().numpy()
            Jg = J[b, k] / g[:, None]
            assert np.abs(Jg.sum(axis=0)).max() <= 1e-11


def check_mlp_off_closed_form(fn_jac):
    """W1 = 0 (Phi = identity): pool(Phi(x_embed + d)) = mean(x_embed) + d, so
    J = LN'(z) (I + alpha W_e2 diag(silu'(e)) W_e1 W_d2 diag(silu'(a)) W_d1)."""
    p, x, m = _inputs()
    p["W1"] = torch.zeros_like(p["W1"])
    J, _ = fn_jac(p, x, m)
    f = {n: v.double().numpy() for n, v in p.items()}
    for b in range(WL.B):
        for k in range(WL.K):
            mm = m[b, k].double().numpy()
            a = f["W_d1"][k] @ mm + f["b_d1"][k]
            d = f["W_d2"][k] @ _silu(a) + f["b_d2"][k]
            pool = x[b].double().numpy().mean(axis=0) + d
            e = f["W_e1"][k] @ pool + f["b_e1"][k]
            z = mm + f["alpha"][k] * (f["W_e2"][k] @ _silu(e) + f["b_e2"][k])
            jdec = f["W_d2"][k] @ (_dsilu(a)[:, None] * f["W_d1"][k])
            jenc = f["W_e2"][k] @ (_dsilu(e)[:, None] * (f["W_e1"][k] @ jdec))
            want = _ln_jacobian(z, f["gamma"][k]) @ (np.eye(WL.r) + f["alpha"][k] * jenc)
            assert np.abs(J[b, k] - want).max() <= 1e-11


CHECKS = [check_finite_differences, check_alpha_zero_is_layernorm, check_layernorm_invariants,
          check_mlp_off_closed_form]


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_oracle_region_jacobians_pinned(check):
    check(oracle.region_jacobians)


# --- plausible mistakes each check set must reject ---------------------------

def _mut_transposed(p, x, m):
    J, mn = oracle.region_jacobians(p, x, m)
    return np.swapaxes(J, -1, -2), mn


def _mut_no_residual(p, x, m):
    """m_{k+1} = LN(alpha Enc(...)) (the skip of m_k dropped)."""
    J, mn = oracle.region_jacobians(p, x, m)
    r = m.shape[-1]
    out = np.empty_like(J)
    for b in range(m.shape[0]):
        for k in range(m.shape[1]):
            z = m[b, k].double().numpy()
            out[b, k] = J[b, k] - _ln_jacobian(z, p["gamma"][k].double().numpy()) @ np.eye(r)
    return out, mn


def _mut_sum_pool(p, x, m):
    """pool = sum over tokens instead of the mean."""
    q = copy.copy(p)
    L = x.shape[1]
    q["W2"] = p["W2"] * L
    xs = x.double() * L
    return oracle.region_jacobians(q, xs, m)


def _mut_no_layernorm_scale(p, x, m):
    J, mn = oracle.region_jacobians(p, x, m)
    return J * 1.5, mn


@pytest.mark.parametrize("mutant", [_mut_transposed, _mut_no_residual, _mut_sum_pool,
                                    _mut_no_layernorm_scale], ids=lambda m: m.__name__)
def test_region_pins_reject_mutants(mutant):
    failed = 0
    for check in CHECKS:
        try:
            check(mutant)
        except AssertionError:
            failed += 1
    assert failed > 0, f"{mutant.__name__} passed every pin"
