"""Pins of the oracle's Phase 1 (region-Jacobian construction for the synthetic
bounded-interface region map of Eq. "concrete-region-arch") that do not go
through torch autograd: central finite differences, the closed-form
LayerNorm Jacobian, LayerNorm's invariants, a closed form of the whole
Jacobian when the region MLP is switched off, a closed form of the whole
Jacobian with the region MLP on (written out in numpy), a one-token region
whose forward value is worked by hand from literal SiLU values, and the
invariance of the mean pool under a permutation of the tokens.

Each check takes a candidate (jac, fwd): ``jac(params, x_embed, m)`` returns
(J, m_next) and ``fwd(params, k, x_b, m_bk)`` is the forward it
differentiates.  The oracle is (oracle.region_jacobians,
oracle.region_forward); the planted mistakes below are candidates whose
forward or Jacobian is wrong in one place, and each must fail some check.
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


def check_finite_differences(jac, fwd):
    p, x, m = _inputs()
    J, _ = jac(p, x, m)
    h = 1e-5
    for b in range(WL.B):
        for k in range(WL.K):
            m0 = m[b, k].to(torch.float64)
            fd = np.empty((WL.r, WL.r))
            for j in range(WL.r):
                e = torch.zeros(WL.r, dtype=torch.float64)
                e[j] = h
                up = fwd(p, k, x[b], m0 + e).numpy()
                dn = fwd(p, k, x[b], m0 - e).numpy()
                fd[:, j] = (up - dn) / (2 * h)
            assert np.abs(fd - J[b, k]).max() <= 1e-7 * max(1.0, np.abs(fd).max())


def check_alpha_zero_is_layernorm(jac, fwd):
    """alpha = 0: the region only renormalises m, J = the LayerNorm Jacobian at m."""
    p, x, m = _inputs(alpha=torch.zeros(WL.K))
    J, mn = jac(p, x, m)
    for b in range(WL.B):
        for k in range(WL.K):
            z = m[b, k].double().numpy()
            g = p["gamma"][k].double().numpy()
            assert np.abs(J[b, k] - _ln_jacobian(z, g)).max() <= 1e-12
            mu, sig = z.mean(), math.sqrt(z.var() + oracle.LN_EPS)
            want = g * (z - mu) / sig + p["beta"][k].double().numpy()
            assert np.abs(mn[b, k] - want).max() <= 1e-12


def check_layernorm_invariants(jac, fwd):
    """LN's output (minus beta, over gamma) has zero mean whatever z is, so for
    every column j: sum_i J_ij / gamma_i = 0.  (Its norm is fixed only with a
    zero epsilon; the alpha = 0 closed form pins that part.)"""
    p, x, m = _inputs()
    J, _ = jac(p, x, m)
    for b in range(WL.B):
        for k in range(WL.K):
            g = p["gamma"][k].double().numpy()
            Jg = J[b, k] / g[:, None]
            assert np.abs(Jg.sum(axis=0)).max() <= 1e-11


def _closed_form(f, k, xb, mm):
    """(J, m_next) of region k for one sequence, written out in numpy.

    With a = W_d1 m + b_d1 and d = W_d2 silu(a) + b_d2, every token enters the
    region MLP as x_l = x_embed_l + d, so d x_l / dm = Jdec = W_d2
    diag(silu'(a)) W_d1 for every l.  Phi(x) = x + W2 silu(W1 x) has the
    differential I + W2 diag(silu'(W1 x)) W1, and the mean pool averages it
    over the tokens: dp = Jdec + W2 diag(mean_l silu'(h_l)) W1 Jdec with
    h_l = W1 x_l.  Then e = W_e1 p + b_e1, z = m + alpha (W_e2 silu(e) +
    b_e2), and J = LN'(z) (I + alpha W_e2 diag(silu'(e)) W_e1 dp).
    """
    a = f["W_d1"][k] @ mm + f["b_d1"][k]
    d = f["W_d2"][k] @ _silu(a) + f["b_d2"][k]
    xl = xb + d[None, :]
    h = xl @ f["W1"][k].T
    phi = xl + _silu(h) @ f["W2"][k].T
    pool = phi.mean(axis=0)
    jdec = f["W_d2"][k] @ (_dsilu(a)[:, None] * f["W_d1"][k])
    dp = jdec + f["W2"][k] @ (_dsilu(h).mean(axis=0)[:, None] * (f["W1"][k] @ jdec))
    e = f["W_e1"][k] @ pool + f["b_e1"][k]
    z = mm + f["alpha"][k] * (f["W_e2"][k] @ _silu(e) + f["b_e2"][k])
    jenc = f["W_e2"][k] @ (_dsilu(e)[:, None] * (f["W_e1"][k] @ dp))
    r = mm.shape[0]
    J = _ln_jacobian(z, f["gamma"][k]) @ (np.eye(r) + f["alpha"][k] * jenc)
    mu, sig = z.mean(), math.sqrt(z.var() + oracle.LN_EPS)
    return J, f["gamma"][k] * (z - mu) / sig + f["beta"][k]


def check_mlp_off_closed_form(jac, fwd):
    """W1 = 0 (Phi = identity): pool(Phi(x_embed + d)) = mean(x_embed) + d, so
    J = LN'(z) (I + alpha W_e2 diag(silu'(e)) W_e1 W_d2 diag(silu'(a)) W_d1)."""
    p, x, m = _inputs()
    p["W1"] = torch.zeros_like(p["W1"])
    J, _ = jac(p, x, m)
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


def check_mlp_on_closed_form(jac, fwd):
    """The region MLP on (W1 != 0, the generated weights): J and m_next equal
    the closed form of ``_closed_form``."""
    p, x, m = _inputs()
    assert float(p["W1"].abs().max()) > 0
    J, mn = jac(p, x, m)
    f = {n: v.double().numpy() for n, v in p.items()}
    for b in range(WL.B):
        xb = x[b].double().numpy()
        for k in range(WL.K):
            Jw, mw = _closed_form(f, k, xb, m[b, k].double().numpy())
            assert np.abs(J[b, k] - Jw).max() <= 1e-11 * max(1.0, np.abs(Jw).max())
            assert np.abs(mn[b, k] - mw).max() <= 1e-12 * max(1.0, np.abs(mw).max())


def check_one_token_by_hand(jac, fwd):
    """A one-token region (r = D = X = 2, L = 1) whose output is worked by hand.

    Dec is switched off (W_d1 = W_d2 = 0, biases 0: silu(0) = 0, so d = 0) and
    the token is x = (1, -1).  Phi: h = W1 x = (1, -2) with W1 = diag(1, 2),
    silu(1) = 0.7310585786300049 and silu(-2) = -0.2384058440442351 (the
    values of t / (1 + e^-t)), W2 = I, so Phi(x) = x + silu(h) =
    (1.7310585786300049, -1.2384058440442351), which is also the pool of
    one token.  Enc is the identity in double precision: b_e1 = 40 puts e =
    p + 40 where silu(e) = e exactly (the logistic of e rounds to 1), and
    b_e2 = -40 takes the shift back off with W_e1 = W_e2 = I.  With alpha = 1
    and m = (1/2, -1/4), z = m + Phi(x); LayerNorm over two features (gamma
    1, beta 0) maps z to (delta, -delta) / sqrt(delta^2 + eps) with delta =
    (z_0 - z_1) / 2.
    """
    t = lambda v: torch.tensor(v, dtype=torch.float64)  # noqa: E731
    p = {"W_d1": t([[[0.0, 0.0], [0.0, 0.0]]]), "b_d1": t([[0.0, 0.0]]),
         "W_d2": t([[[0.0, 0.0], [0.0, 0.0]]]), "b_d2": t([[0.0, 0.0]]),
         "W1": t([[[1.0, 0.0], [0.0, 2.0]]]), "W2": t([[[1.0, 0.0], [0.0, 1.0]]]),
         "W_e1": t([[[1.0, 0.0], [0.0, 1.0]]]), "b_e1": t([[40.0, 40.0]]),
         "W_e2": t([[[1.0, 0.0], [0.0, 1.0]]]), "b_e2": t([[-40.0, -40.0]]),
         "alpha": t([1.0]), "gamma": t([[1.0, 1.0]]), "beta": t([[0.0, 0.0]])}
    x = t([[[1.0, -1.0]]])
    m = t([[[0.5, -0.25]]])
    _, mn = jac(p, x, m)
    phi = np.array([1.0 + 0.7310585786300049, -1.0 - 0.2384058440442351])
    z = np.array([0.5, -0.25]) + phi
    delta = (z[0] - z[1]) / 2.0
    want = np.array([delta, -delta]) / math.sqrt(delta * delta + oracle.LN_EPS)
    assert np.abs(mn[0, 0] - want).max() <= 1e-13


def check_token_permutation_invariance(jac, fwd):
    """The mean pool does not see the order of the tokens: permuting
    x_embed's tokens leaves J and m_next unchanged (to rounding)."""
    p, x, m = _inputs()
    J, mn = jac(p, x, m)
    perm = torch.randperm(WL.L, generator=torch.Generator().manual_seed(3))
    Jp, mnp = jac(p, x[:, perm], m)
    assert np.abs(Jp - J).max() <= 1e-12 * max(1.0, np.abs(J).max())
    assert np.abs(mnp - mn).max() <= 1e-12


CHECKS = [check_finite_differences, check_alpha_zero_is_layernorm, check_layernorm_invariants,
          check_mlp_off_closed_form, check_mlp_on_closed_form, check_one_token_by_hand,
          check_token_permutation_invariance]

ORACLE = (oracle.region_jacobians, oracle.region_forward)


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_oracle_region_jacobians_pinned(check):
    check(*ORACLE)


def test_closed_form_helper_against_finite_differences():
    """The numpy closed form itself, against central differences of its own
    m_next (so that a slip in it cannot hide behind the oracle)."""
    p, x, m = _inputs()
    f = {n: v.double().numpy() for n, v in p.items()}
    xb, mm = x[0].double().numpy(), m[0, 1].double().numpy()
    J, _ = _closed_form(f, 1, xb, mm)
    h = 1e-6
    for j in range(WL.r):
        e = np.zeros(WL.r)
        e[j] = h
        fd = (_closed_form(f, 1, xb, mm + e)[1] - _closed_form(f, 1, xb, mm - e)[1]) / (2 * h)
        assert np.abs(fd - J[:, j]).max() <= 1e-7 * max(1.0, np.abs(J).max())


# --- plausible mistakes each check set must reject ---------------------------

def _jac_of(fwd):
    """Jacobians of a (mistaken) forward by autograd, as the oracle takes them."""
    def jac(p, x, m):
        B, K, r = m.shape
        J = np.empty((B, K, r, r))
        mn = np.empty((B, K, r))
        for b in range(B):
            for k in range(K):
                m0 = m[b, k].detach().to(torch.float64)
                fn = lambda mm: fwd(p, k, x[b], mm)  # noqa: E731
                J[b, k] = torch.autograd.functional.jacobian(fn, m0, vectorize=True).numpy()
                mn[b, k] = fn(m0).detach().numpy()
        return J, mn
    return jac


def _forward_with(phi_act=None, phi_residual=True, pool="mean"):
    """The region forward with one part changed: Phi's activation, Phi's
    residual, or the pool."""
    def fwd(params, k, x_embed_b, m_bk):
        f = {n: v[k].to(torch.float64) for n, v in params.items()}
        xb = x_embed_b.to(torch.float64)
        m = m_bk.to(torch.float64)
        silu = lambda t: t * torch.sigmoid(t)  # noqa: E731
        d = f["W_d2"] @ silu(f["W_d1"] @ m + f["b_d1"]) + f["b_d2"]
        x_in = xb + d
        act = phi_act or silu
        phi = (x_in if phi_residual else 0.0) + act(x_in @ f["W1"].T) @ f["W2"].T
        pooled = phi.mean(dim=0) if pool == "mean" else phi[-1]
        enc = f["W_e2"] @ silu(f["W_e1"] @ pooled + f["b_e1"]) + f["b_e2"]
        z = m + f["alpha"] * enc
        mu = z.mean()
        var = ((z - mu) ** 2).mean()
        return f["gamma"] * (z - mu) / torch.sqrt(var + oracle.LN_EPS) + f["beta"]
    return fwd


def _cand(fwd):
    return _jac_of(fwd), fwd


def _dsilu_t(t):
    s = torch.sigmoid(t)
    return s * (1.0 + t * (1.0 - s))


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


MUTANTS = {
    "transposed": (_mut_transposed, oracle.region_forward),
    "no_residual": (_mut_no_residual, oracle.region_forward),
    "sum_pool": (_mut_sum_pool, oracle.region_forward),
    "no_layernorm_scale": (_mut_no_layernorm_scale, oracle.region_forward),
    # Phi's activation replaced by its derivative, by tanh, or by the
    # logistic function; Phi's residual dropped; the last token in place of
    # the mean pool.  Each is a consistent forward: finite differences of it
    # match its own Jacobian, so only the closed forms, the hand-worked
    # token and the permutation invariance can catch it.
    "phi_silu_derivative": _cand(_forward_with(phi_act=_dsilu_t)),
    "phi_tanh": _cand(_forward_with(phi_act=torch.tanh)),
    "phi_sigmoid": _cand(_forward_with(phi_act=torch.sigmoid)),
    "phi_no_residual": _cand(_forward_with(phi_residual=False)),
    "pool_last_token": _cand(_forward_with(pool="last")),
}


def test_mistaken_forwards_are_self_consistent():
    """The planted forwards differ from the oracle's only where intended: the
    unchanged forward built the same way reproduces the oracle."""
    p, x, m = _inputs()
    same = _jac_of(_forward_with())
    J0, mn0 = oracle.region_jacobians(p, x, m)
    J1, mn1 = same(p, x, m)
    assert np.abs(J1 - J0).max() <= 1e-12 and np.abs(mn1 - mn0).max() <= 1e-12


@pytest.mark.parametrize("name", list(MUTANTS))
def test_region_pins_reject_mutants(name):
    jac, fwd = MUTANTS[name]
    failed = 0
    for check in CHECKS:
        try:
            check(jac, fwd)
        except AssertionError:
            failed += 1
    assert failed > 0, f"{name} passed every pin"


@pytest.mark.parametrize("name", ["phi_silu_derivative", "phi_tanh", "phi_sigmoid",
                                  "phi_no_residual"])
def test_phi_mutants_fail_the_phi_pins(name):
    """Each planted mistake inside Phi fails the closed form with the MLP on
    and the hand-worked token, not only some unrelated pin."""
    jac, fwd = MUTANTS[name]
    for check in (check_mlp_on_closed_form, check_one_token_by_hand):
        with pytest.raises(AssertionError):
            check(jac, fwd)
