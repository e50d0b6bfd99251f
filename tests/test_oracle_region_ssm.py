"""Pins of the oracle's token-mixing region block (``phi="ssm"``) that do not
go through the oracle's own code path: the causal recurrence against its
closed-form sum, its special decays, the whole region Jacobian against the
chain rule written out by hand in numpy (with the recurrence's tangent in
closed form), central finite differences, and the decay-one limit, where the
block passes its input through unchanged.  Planted mistakes (each a forward
that is wrong in one place) must each fail some pin.

The block (the architecture section lists SSMs among the region
transformations): s_l = a * s_{l-1} + (1 - a) * x_l from s_0 = 0 over the L
tokens of a sequence, and Phi(x)_l = x_l + (W2 silu(W1 s_l)) * silu(s_l).
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import synth

WL = synth.RegionWorkload("pin_ssm", B=2, K=2, L=12, D=32, X=48, r=16, seed=19)


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
    r = z.shape[0]
    mu = z.mean()
    sig = math.sqrt(((z - mu) ** 2).mean() + oracle.LN_EPS)
    zh = (z - mu) / sig
    return (gamma[:, None] / sig) * (np.eye(r) - 1.0 / r - np.outer(zh, zh) / r)


# ---- the recurrence -------------------------------------------------------------

def _states_closed_form(x, a):
    """s_l = sum_{i <= l} a^(l - i) (1 - a) x_i (tokens 1-based), in numpy."""
    L = x.shape[0]
    s = np.zeros_like(x)
    for l in range(L):
        w = a[None, :] ** (l - np.arange(l + 1))[:, None]  # [l + 1, D]
        s[l] = ((1.0 - a)[None, :] * w * x[:l + 1]).sum(axis=0)
    return s


def test_states_match_the_closed_form_sum():
    g = np.random.default_rng(3)
    x = g.standard_normal((9, 5))
    a = g.uniform(0.0, 1.0, 5)
    got = oracle.ssm_states(torch.from_numpy(x), torch.from_numpy(a)).numpy()
    assert np.abs(got - _states_closed_form(x, a)).max() <= 1e-14


def test_states_special_decays():
    g = np.random.default_rng(4)
    x = torch.from_numpy(g.standard_normal((7, 4)))
    # a = 0: the state is the token itself; a = 1: nothing enters
    assert torch.equal(oracle.ssm_states(x, torch.zeros(4, dtype=torch.float64)), x)
    assert not oracle.ssm_states(x, torch.ones(4, dtype=torch.float64)).any()
    # a constant input c reaches (1 - a^l) c after l tokens
    a = torch.tensor([0.5, 0.9, 0.25, 0.75], dtype=torch.float64)
    c = torch.tensor([1.0, -2.0, 3.0, 0.5], dtype=torch.float64)
    s = oracle.ssm_states(c.expand(7, 4).clone(), a)
    for l in range(1, 8):
        assert torch.allclose(s[l - 1], (1 - a ** l) * c, rtol=0, atol=1e-15)


def test_states_are_causal():
    """d s_l / d x_t = 0 for t > l (and a^(l - t) (1 - a) on the diagonal
    blocks otherwise)."""
    g = np.random.default_rng(5)
    x = torch.from_numpy(g.standard_normal((6, 3)))
    a = torch.tensor([0.3, 0.6, 0.9], dtype=torch.float64)
    J = torch.autograd.functional.jacobian(lambda t: oracle.ssm_states(t, a), x)  # [6,3,6,3]
    for l in range(6):
        for t in range(6):
            blk = J[l, :, t, :]
            want = torch.diag((1 - a) * a ** (l - t)) if t <= l else torch.zeros(3, 3)
            assert torch.allclose(blk, want.to(blk.dtype), rtol=0, atol=1e-15)


# ---- the whole region -----------------------------------------------------------

def _closed_form_ssm(f, k, xb, mm):
    """(J, m_next) of region k with the token-mixing block, in numpy.

    Every token enters as x_l = x_embed_l + d, so dx_l / dm = Jdec for every l;
    the state's tangent is then ds_l = (1 - a^l) Jdec (the recurrence of a
    constant).  With u_l = W1 s_l, y_l = W2 silu(u_l) and z_l = silu(s_l),
    Phi_l = x_l + y_l z_l has the tangent
      Jdec + diag(z_l) W2 diag(silu'(u_l)) W1 ds_l + diag(y_l silu'(s_l)) ds_l,
    averaged over the tokens by the pool; then Enc and the LayerNorm as in the
    token-wise block.
    """
    a = f["W_d1"][k] @ mm + f["b_d1"][k]
    d = f["W_d2"][k] @ _silu(a) + f["b_d2"][k]
    dec = f["decay"][k]
    xl = xb + d[None, :]
    s = _states_closed_form(xl, dec)
    u = s @ f["W1"][k].T
    y = _silu(u) @ f["W2"][k].T
    pool = (xl + y * _silu(s)).mean(axis=0)
    jdec = f["W_d2"][k] @ (_dsilu(a)[:, None] * f["W_d1"][k])
    L = xb.shape[0]
    dp = jdec.copy()
    for l in range(L):
        ds = (1.0 - dec ** (l + 1))[:, None] * jdec
        inner = f["W2"][k] @ (_dsilu(u[l])[:, None] * (f["W1"][k] @ ds))
        dp += (_silu(s[l])[:, None] * inner + (y[l] * _dsilu(s[l]))[:, None] * ds) / L
    e = f["W_e1"][k] @ pool + f["b_e1"][k]
    z = mm + f["alpha"][k] * (f["W_e2"][k] @ _silu(e) + f["b_e2"][k])
    jenc = f["W_e2"][k] @ (_dsilu(e)[:, None] * (f["W_e1"][k] @ dp))
    r = mm.shape[0]
    J = _ln_jacobian(z, f["gamma"][k]) @ (np.eye(r) + f["alpha"][k] * jenc)
    mu, sig = z.mean(), math.sqrt(z.var() + oracle.LN_EPS)
    return J, f["gamma"][k] * (z - mu) / sig + f["beta"][k]


def _jac_of(fwd):
    def jac(p, x, m):
        B, K, r = m.shape
        J = np.empty((B, K, r, r))
        mn = np.empty((B, K, r))
        for b in range(B):
            for k in range(K):
                m0 = m[b, k].to(torch.float64)
                fn = lambda mm: fwd(p, k, x[b], mm)  # noqa: E731
                J[b, k] = torch.autograd.functional.jacobian(fn, m0).numpy()
                mn[b, k] = fn(m0).detach().numpy()
        return J, mn
    return jac


def _oracle_fwd(p, k, xb, mm):
    return oracle.region_forward(p, k, xb, mm, "ssm")


def _oracle_jac(p, x, m):
    return oracle.region_jacobians(p, x, m, phi="ssm")


def check_closed_form(jac, fwd):
    p, x, m = _inputs()
    J, mn = jac(p, x, m)
    f = {n: v.double().numpy() for n, v in p.items()}
    for b in range(WL.B):
        xb = x[b].double().numpy()
        for k in range(WL.K):
            Jc, mc = _closed_form_ssm(f, k, xb, m[b, k].double().numpy())
            assert np.abs(J[b, k] - Jc).max() <= 1e-11 * max(1.0, np.abs(Jc).max())
            assert np.abs(mn[b, k] - mc).max() <= 1e-11


def check_finite_differences(jac, fwd):
    p, x, m = _inputs()
    J, _ = jac(p, x, m)
    h = 1e-5
    b, k = 1, 0
    m0 = m[b, k].to(torch.float64)
    fd = np.empty((WL.r, WL.r))
    for j in range(WL.r):
        e = torch.zeros(WL.r, dtype=torch.float64)
        e[j] = h
        fd[:, j] = (fwd(p, k, x[b], m0 + e).numpy() - fwd(p, k, x[b], m0 - e).numpy()) / (2 * h)
    assert np.abs(fd - J[b, k]).max() <= 1e-7 * max(1.0, np.abs(fd).max())


def check_decay_one_passes_the_input(jac, fwd):
    """a = 1: no token enters the state (s = 0), silu(0) = 0 closes the gate,
    so Phi(x) = x and the region is the token-wise region with W1 = 0, whose
    Jacobian is LN'(z) (I + alpha Jenc Jdec) with p = mean(x_embed) + d."""
    p, x, m = _inputs()
    p["decay"] = torch.ones_like(p["decay"])
    J, mn = jac(p, x, m)
    f = {n: v.double().numpy() for n, v in p.items()}
    for b in range(WL.B):
        xb = x[b].double().numpy()
        for k in range(WL.K):
            mm = m[b, k].double().numpy()
            a = f["W_d1"][k] @ mm + f["b_d1"][k]
            d = f["W_d2"][k] @ _silu(a) + f["b_d2"][k]
            pool = xb.mean(axis=0) + d
            jdec = f["W_d2"][k] @ (_dsilu(a)[:, None] * f["W_d1"][k])
            e = f["W_e1"][k] @ pool + f["b_e1"][k]
            z = mm + f["alpha"][k] * (f["W_e2"][k] @ _silu(e) + f["b_e2"][k])
            jenc = f["W_e2"][k] @ (_dsilu(e)[:, None] * (f["W_e1"][k] @ jdec))
            Jc = _ln_jacobian(z, f["gamma"][k]) @ (np.eye(WL.r) + f["alpha"][k] * jenc)
            assert np.abs(J[b, k] - Jc).max() <= 1e-12 * max(1.0, np.abs(Jc).max())


CHECKS = [check_closed_form, check_finite_differences, check_decay_one_passes_the_input]


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_oracle_ssm_region_pinned(check):
    check(_oracle_jac, _oracle_fwd)


def test_jacobian_columns_equal_the_full_jacobian():
    """Forward-mode columns (one JVP per basis vector) equal the reverse-mode
    Jacobian, for both blocks."""
    p, x, m = _inputs()
    for phi in ("mlp", "ssm"):
        J, mn = oracle.region_jacobians(p, x, m, pairs=[(1, 1)], phi=phi)
        cols, mc = oracle.region_jacobian_columns(p, x, m, 1, 1, [0, 5, 15], phi=phi)
        assert np.abs(cols - J[1, 1][:, [0, 5, 15]].T).max() <= 1e-12
        assert np.abs(mc - mn[1, 1]).max() <= 1e-14


def test_blocks_differ():
    """The token-mixing block is not the token-wise one (a sanity check that
    the phi argument reaches the forward)."""
    p, x, m = _inputs()
    a = oracle.region_forward(p, 0, x[0], m[0, 0].double(), "mlp")
    b = oracle.region_forward(p, 0, x[0], m[0, 0].double(), "ssm")
    assert (a - b).abs().max() > 1e-3


# ---- planted mistakes -----------------------------------------------------------

def _silu_t(t):
    return t * torch.sigmoid(t)


def _mutant(kind):
    def fwd(params, k, x_embed_b, m_bk):
        f = {n: v[k].to(torch.float64) for n, v in params.items()}
        xb = x_embed_b.to(torch.float64)
        m = m_bk.to(torch.float64)
        d = f["W_d2"] @ _silu_t(f["W_d1"] @ m + f["b_d1"]) + f["b_d2"]
        xin = xb + d
        a = f["decay"]
        if kind == "anticausal":
            s = oracle.ssm_states(xin.flip(0), a).flip(0)
        elif kind == "no_input_gain":
            out, prev = [], torch.zeros_like(xin[0])
            for t in range(xin.shape[0]):
                prev = a * prev + xin[t]
                out.append(prev)
            s = torch.stack(out)
        else:
            s = oracle.ssm_states(xin, a)
        mlp = _silu_t(s @ f["W1"].T) @ f["W2"].T
        if kind == "no_gate":
            phi = xin + mlp
        elif kind == "gate_on_input":
            phi = xin + mlp * _silu_t(xin)
        elif kind == "no_residual":
            phi = mlp * _silu_t(s)
        else:
            phi = xin + mlp * _silu_t(s)
        pool = phi.mean(dim=0)
        enc = f["W_e2"] @ _silu_t(f["W_e1"] @ pool + f["b_e1"]) + f["b_e2"]
        z = m + f["alpha"] * enc
        mu = z.mean()
        var = ((z - mu) ** 2).mean()
        return f["gamma"] * (z - mu) / torch.sqrt(var + oracle.LN_EPS) + f["beta"]
    return fwd


MUTANTS = ["anticausal", "no_input_gain", "no_gate", "gate_on_input", "no_residual"]


def test_unmutated_twin_passes():
    """The mutant template with no mistake passes every pin (so a failure of a
    mutant comes from its mistake)."""
    fwd = _mutant("none")
    for check in CHECKS:
        check(_jac_of(fwd), fwd)


@pytest.mark.parametrize("kind", MUTANTS)
def test_pins_reject_mutants(kind):
    fwd = _mutant(kind)
    failed = []
    for check in CHECKS:
        try:
            check(_jac_of(fwd), fwd)
        except AssertionError:
            failed.append(check.__name__)
    assert failed, f"mutant {kind} passed every pin"
