"""CPU oracle for the interface-adjoint scan -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never calls it and
shares no code with it.

What it computes (paper: "LBI: Parallel Scan Backpropagation via Latent
Bounded Interfaces"):

* ``recurrence`` -- Theorem "Bounded-Interface Backpropagation":
  mbar_k = J_k^T mbar_{k+1} for k = K-1..0, extended with the affine term b_k
  (the direct gradient of loss terms that read m_k):
  ``lambda_j = A_j lambda_{j+1} + b_j`` with ``A_j = J_j^T``.  This is the plain
  definition of what the scan returns; fp64, inputs widened exactly.
* ``suffix_composites`` -- Proposition "Scan Formulation of Backpropagation":
  the suffix products ``P_j = A_j ... A_{K-1}`` (empty product I) and offsets
  ``c_j``, obtained by folding the combine (A, b) o (A', b') = (AA', Ab' + b)
  from the right end of the chain.  fp64.
* ``matrix_norms`` -- the statistics of the appendix "Interface Jacobian
  Structure": spectral norm (largest singular value, from an fp64 SVD) and
  Frobenius norm / sqrt(r) of each matrix of a stack.
* ``region_forward`` / ``region_jacobians`` -- Phase 1 of Algorithm
  "Bounded-Interface Backpropagation" for the concrete region map of Eq.
  "concrete-region-arch", m_{k+1} = LN(m_k + alpha_k Enc_k(pool(Phi_k(x_embed +
  Dec_k(m_k))))), with the readings of the synthetic map (2-layer SiLU MLPs
  for Dec and Enc, a token-wise residual SiLU MLP for Phi, mean pooling over
  tokens, LayerNorm over the r interface features with eps 1e-5): the forward
  written out in fp64 torch ops and J_k = dR_k(m_k) from torch autograd
  (Eq. "jacobian-identity-construction": the differential applied to I_r).
  With ``phi="ssm"`` Phi_k mixes the tokens (the SSM-style region block of the
  architecture section, "e.g. attention, SSM, MLP"): a causal diagonal linear
  recurrence s_l = a_k * s_{l-1} + (1 - a_k) * x_l from s_0 = 0, then
  Phi_k(x)_l = x_l + (W2 silu(W1 s_l)) * silu(s_l).  ``ssm_states`` is that
  recurrence on its own; ``region_jacobian_columns`` gives chosen columns of
  J_k by forward-mode AD (Eq. "basis-JVP": dR_k(m_k) e_j), for large regions.

Every function here is pinned by the CPU tests against closed forms, exact
rational brute force, invariants and torch autograd (see tests/test_oracle_*).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lbi_oracle.c")
_LIBDIR = os.path.join(_HERE, "_lib")
_LIB = os.path.join(_LIBDIR, "liblbi_oracle.so")

_F64, _F32, _BF16 = 0, 1, 2

_lib = None


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (-O2 -ffp-contract=off -fopenmp)."""
    if not force and os.path.exists(_LIB):
        return _LIB
    os.makedirs(_LIBDIR, exist_ok=True)
    tmp = _LIB + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", tmp, _SRC]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        vp, i64, i32, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int
        lib.lbi_oracle_recurrence.argtypes = [vp, vp, vp, vp, i64, i64, i32, ci, ci]
        lib.lbi_oracle_recurrence.restype = ci
        lib.lbi_oracle_suffix_composites.argtypes = [vp, vp, vp, vp, i64, i64, i32, ci]
        lib.lbi_oracle_suffix_composites.restype = ci
        lib.lbi_oracle_threads.argtypes = [ci]
        lib.lbi_oracle_threads.restype = ci
        _lib = lib
    return _lib


def _host_array(x) -> Tuple[object, int]:
    """A C-contiguous host buffer for x (torch tensor or numpy) + its dtype code.

    The returned object keeps the buffer alive; bf16 is passed as raw bits.
    """
    try:
        import torch
    except ImportError:  # pragma: no cover - torch is always present here
        torch = None
    if torch is not None and isinstance(x, torch.Tensor):
        t = x.detach().to("cpu").contiguous()
        if t.dtype == torch.float64:
            return t, _F64
        if t.dtype == torch.float32:
            return t, _F32
        if t.dtype == torch.bfloat16:
            return t, _BF16
        raise TypeError(f"unsupported oracle input dtype {t.dtype}")
    a = np.ascontiguousarray(x)
    if a.dtype == np.float64:
        return a, _F64
    if a.dtype == np.float32:
        return a, _F32
    raise TypeError(f"unsupported oracle input dtype {a.dtype}")


def _ptr(obj) -> int:
    if isinstance(obj, np.ndarray):
        return obj.ctypes.data
    return obj.data_ptr()


def threads(nthreads: int = 0) -> int:
    """Threads the recurrence runs on for ``nthreads`` (<= 0: OpenMP default)."""
    return int(_load().lbi_oracle_threads(int(nthreads)))


def recurrence(A, b, lamK, nthreads: int = 0) -> np.ndarray:
    """lambda[B, K, r] (float64) from A[B, K, r, r], b[B, K, r] or None, lamK[B, r]."""
    lib = _load()
    a_buf, dt = _host_array(A)
    l_buf, dt_l = _host_array(lamK)
    if dt_l != dt:
        raise TypeError("A and lamK must share a dtype")
    shape = tuple(a_buf.shape)
    if len(shape) != 4 or shape[2] != shape[3]:
        raise ValueError(f"A must be [B, K, r, r], got {shape}")
    B, K, r, _ = shape
    if tuple(l_buf.shape) != (B, r):
        raise ValueError("lamK must be [B, r]")
    b_ptr = None
    b_buf = None
    if b is not None:
        b_buf, dt_b = _host_array(b)
        if dt_b != dt or tuple(b_buf.shape) != (B, K, r):
            raise ValueError("b must be [B, K, r] in A's dtype")
        b_ptr = _ptr(b_buf)
    out = np.empty((B, K, r), dtype=np.float64)
    if B == 0:
        return out
    rc = lib.lbi_oracle_recurrence(_ptr(a_buf), b_ptr, _ptr(l_buf), out.ctypes.data,
                                   B, K, r, dt, int(nthreads))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return out


def suffix_composites(A, b) -> Tuple[np.ndarray, np.ndarray]:
    """(P[B, K, r, r], c[B, K, r]) in float64: the inclusive suffix scan."""
    lib = _load()
    a_buf, dt = _host_array(A)
    B, K, r, _ = a_buf.shape
    b_ptr = None
    b_buf = None
    if b is not None:
        b_buf, dt_b = _host_array(b)
        if dt_b != dt or tuple(b_buf.shape) != (B, K, r):
            raise ValueError("b must be [B, K, r] in A's dtype")
        b_ptr = _ptr(b_buf)
    P = np.empty((B, K, r, r), dtype=np.float64)
    c = np.empty((B, K, r), dtype=np.float64)
    if B == 0:
        return P, c
    rc = lib.lbi_oracle_suffix_composites(_ptr(a_buf), b_ptr, P.ctypes.data, c.ctypes.data,
                                          B, K, r, dt)
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return P, c


def rel_frobenius(x: np.ndarray, ref: np.ndarray) -> float:
    """||x - ref||_F / ||ref||_F (the absolute error when ||ref||_F = 0)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = float(np.linalg.norm((x - ref).ravel()))
    den = float(np.linalg.norm(ref.ravel()))
    return num / den if den > 0 else num


def per_chain_rel_frobenius(x: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Relative Frobenius error of each chain (leading axis)."""
    x = np.asarray(x, dtype=np.float64).reshape(x.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(ref.shape[0], -1)
    num = np.linalg.norm(x - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), num)


def matrix_norms(M) -> Tuple[np.ndarray, np.ndarray]:
    """(||M_i||_2, ||M_i||_F / sqrt(r)) in float64 for M[..., r, r].

    The spectral norm is the largest singular value (LAPACK SVD in fp64 on the
    exactly widened input); the Frobenius norm is the square root of the sum
    of squares.  r is the tile width (the last axis).
    """
    buf, dt = _host_array(M)
    if dt == _BF16:
        a = buf.to(dtype=__import__("torch").float64).numpy()
    else:
        a = np.asarray(buf if isinstance(buf, np.ndarray) else buf.numpy(), dtype=np.float64)
    if a.ndim < 2 or a.shape[-1] != a.shape[-2]:
        raise ValueError(f"M must be [..., r, r], got {a.shape}")
    r = a.shape[-1]
    lead = a.shape[:-2]
    flat = a.reshape((-1, r, r))
    spec = np.empty(flat.shape[0], dtype=np.float64)
    fro = np.empty(flat.shape[0], dtype=np.float64)
    for i in range(flat.shape[0]):
        spec[i] = np.linalg.svd(flat[i], compute_uv=False)[0]
        fro[i] = np.sqrt(np.sum(flat[i] * flat[i])) / np.sqrt(r)
    return spec.reshape(lead), fro.reshape(lead)


LN_EPS = 1e-5


def _silu(t):
    return t * (1.0 / (1.0 + (-t).exp()))


def ssm_states(x, a):
    """The causal diagonal linear recurrence over the tokens of one sequence:
    s_l = a * s_{l-1} + (1 - a) * x_l for l = 1..L, s_0 = 0; x [L, D], a [D]
    (torch, any float dtype).  Returns s [L, D]."""
    import torch
    out = []
    prev = torch.zeros_like(x[0])
    for t in range(x.shape[0]):
        prev = a * prev + (1.0 - a) * x[t]
        out.append(prev)
    return torch.stack(out)


def region_forward(params: dict, k: int, x_embed_b, m_bk, phi: str = "mlp"):
    """R_k(m) for one sequence in float64: x_embed_b [L, D], m_bk [r] (torch).
    phi: "mlp" (token-wise residual MLP) or "ssm" (causal recurrence over the
    tokens, then the MLP gated by silu of the state; needs params["decay"])."""
    import torch
    f = {n: v[k].to(torch.float64) for n, v in params.items()}
    x_embed_b = x_embed_b.to(torch.float64)
    m = m_bk.to(torch.float64)
    # Dec_k: injects the interface state into the region (Eq. "concrete-region-injection")
    d = f["W_d2"] @ _silu(f["W_d1"] @ m + f["b_d1"]) + f["b_d2"]
    x_in = x_embed_b + d                               # [L, D]
    if phi == "mlp":
        # Phi_k: token-wise residual MLP
        phi_out = x_in + _silu(x_in @ f["W1"].T) @ f["W2"].T   # [L, D]
    elif phi == "ssm":
        # Phi_k: the state s_l of the causal recurrence, the MLP on s_l gated
        # by silu(s_l), plus the token's input
        s = ssm_states(x_in, f["decay"])
        phi_out = x_in + (_silu(s @ f["W1"].T) @ f["W2"].T) * _silu(s)
    else:
        raise ValueError(f"phi must be 'mlp' or 'ssm', got {phi!r}")
    phi = phi_out
    # pool: mean over the L tokens
    p = phi.mean(dim=0)
    # Enc_k projects into the interface space
    enc = f["W_e2"] @ _silu(f["W_e1"] @ p + f["b_e1"]) + f["b_e2"]
    z = m + f["alpha"] * enc
    mu = z.mean()
    var = ((z - mu) ** 2).mean()
    return f["gamma"] * (z - mu) / torch.sqrt(var + LN_EPS) + f["beta"]


def region_jacobians(params: dict, x_embed, m, pairs=None,
                     phi: str = "mlp") -> Tuple[np.ndarray, np.ndarray]:
    """(J [B, K, r, r], m_next [B, K, r]) in float64: J[b, k] = d m_{k+1} / d m_k
    of region k at m[b, k] (rows: outputs), and m_next[b, k] = R_k(m[b, k]).
    With ``pairs`` (a list of (b, k)), only those entries are computed (the
    rest are NaN).  ``phi`` selects the region block (``region_forward``)."""
    import torch
    B, K, r = m.shape
    J = np.full((B, K, r, r), np.nan)
    mn = np.full((B, K, r), np.nan)
    todo = pairs if pairs is not None else [(b, k) for b in range(B) for k in range(K)]
    for b, k in todo:
        m0 = m[b, k].detach().to("cpu", torch.float64)
        xb = x_embed[b].detach().to("cpu")
        fn = lambda mm: region_forward(params, k, xb, mm, phi)  # noqa: E731
        J[b, k] = torch.autograd.functional.jacobian(fn, m0, vectorize=True).numpy()
        mn[b, k] = fn(m0).detach().numpy()
    return J, mn


def region_jacobian_columns(params: dict, x_embed, m, b: int, k: int, cols,
                            phi: str = "mlp") -> Tuple[np.ndarray, np.ndarray]:
    """(columns [len(cols), r], m_next [r]) in float64: row i is column
    cols[i] of J_k at m[b, k], dR_k(m_k) e_j by forward-mode AD (one
    Jacobian-vector product per column, Eq. "basis-JVP")."""
    import torch
    m0 = m[b, k].detach().to("cpu", torch.float64)
    xb = x_embed[b].detach().to("cpu")
    fn = lambda mm: region_forward(params, k, xb, mm, phi)  # noqa: E731
    out = []
    val = None
    for j in cols:
        e = torch.zeros_like(m0)
        e[j] = 1.0
        val, tan = torch.func.jvp(fn, (m0,), (e,))
        out.append(tan.detach().numpy())
    mn = (val if val is not None else fn(m0)).detach().numpy()
    return np.stack(out) if out else np.zeros((0, m0.shape[0])), mn
