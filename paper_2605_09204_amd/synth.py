"""Seeded synthetic inputs for the interface-adjoint scan and its Phase 1.

This module draws operands and nothing else: the stack of interface-Jacobian
transposes ``A[B, K, R, R]``, the affine terms ``b[B, K, R]`` and the terminal
adjoints ``lambda_K[B, R]`` of the scan; the weights, token embeddings and
interface states of a synthetic region map (Phase 1); and the compact packing
of ragged tiles.  It contains none of the method's arithmetic, so the HIP path
and the CPU oracle can both consume what it makes without sharing any of it.

Layout (row-major, C-contiguous):
  * ``A[beta, j]`` is the transpose of the interface Jacobian
    ``J_j = d m_{j+1} / d m_j`` (Section "Implementation Details" defines J_j as
    an r_{j+1} x r_j matrix), so it has r_j rows and r_{j+1} columns.  Widths
    below the tile width R are zero-padded.
  * ``b[beta, j]`` has r_j meaningful entries, ``lambda_K[beta]`` has r_K.

Recipes (each a workload of the paper's r = 64 setting or its variants):
  * ``uniform``: A = Q1 diag(s) Q2 with Q1, Q2 Haar-orthogonal (the Q of the
    QR factorisation of a Gaussian matrix with positive diag(R), Mezzadri 2007) and
    s ~ U[0.9, 1.1].
  * ``concentrated``: the same factors with a spectrum shaped like the trained
    Mamba-3 interface Jacobians of the spectral-structure appendix (leading
    singular value about 2.5 x the RMS singular value): r-1 values log-uniform
    on [0.3, 1.0], s_1 = 2.5 * RMS(s) (RMS over all r values), then all values
    scaled by min(1, 1.05 / s_1) so that ||A||_2 <= 1.05.
  * rectangular blocks (mixed widths): Q1[:, :k] diag(s) Q2[:k, :] with
    k = min(r_j, r_{j+1}).
  * b_j ~ N(0, 1/r_j) (variance 1/r_j), lambda_K ~ N(0, 1).

Values are produced in float64, rounded to float32 (round-to-nearest-even) and,
for bf16 workloads, rounded once more to bfloat16.  Draws come from a
``torch.Generator`` seeded per chunk of ``CHUNK`` chains, on the device that
generates; a CPU and a GPU generator give different (equally distributed)
streams, so tests always hand the *same* stored bits to both sides.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence, Tuple

import torch

CHUNK = 16  # chains drawn per generator seed

STORAGE = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic scan workload: B independent chains of K slots."""

    name: str
    B: int
    K: int
    r: int  # tile width R (largest interface width)
    dtype: str  # storage dtype of A, b, lambda_K: "f32" | "bf16"
    seed: int
    spectrum: str = "uniform"  # "uniform" | "concentrated" | "orthogonal"
    affine: bool = True  # False: b is absent (the caller passes NULL)
    widths: Optional[Tuple[int, ...]] = None  # r_0..r_K, None: all equal r

    def interface_widths(self) -> Tuple[int, ...]:
        if self.widths is None:
            return (self.r,) * (self.K + 1)
        return self.widths

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def cyclic_widths(K: int, cycle: Sequence[int] = (32, 64, 128)) -> Tuple[int, ...]:
    """r_k = cycle[k mod len(cycle)] for k = 0..K (K+1 interfaces)."""
    return tuple(cycle[k % len(cycle)] for k in range(K + 1))


# The five workloads of the paper's r = 64 setting and its variants.
WORKLOADS = {
    # B=4 sequences, K=8 regions, r=16, fp32: small enough for exact checks.
    "tiny": Workload("tiny", B=4, K=8, r=16, dtype="f32", seed=0),
    # B=256, K=32, r=64, fp32: the paper's interface width.
    "paper_width": Workload("paper_width", B=256, K=32, r=64, dtype="f32", seed=1),
    # B=4096 token positions, K=32, r=64, bf16 storage, b = 0 (loss at the
    # last region only, the paper's own setting).
    "bf16_tokens": Workload("bf16_tokens", B=4096, K=32, r=64, dtype="bf16", seed=2,
                            affine=False),
    # B=512, K=512, r=64, fp32, spectrally concentrated Jacobians.
    "long_chain": Workload("long_chain", B=512, K=512, r=64, dtype="f32", seed=3,
                           spectrum="concentrated"),
    # B=1024, K=64, r_k cycling 32/64/128 padded to 128, bf16 storage.
    "mixed_widths": Workload("mixed_widths", B=1024, K=64, r=128, dtype="bf16", seed=4,
                             widths=cyclic_widths(64)),
}

WORKLOAD_ORDER = ("tiny", "paper_width", "bf16_tokens", "long_chain", "mixed_widths")


@dataclasses.dataclass
class Inputs:
    """Operands of one scan call, in storage dtype on one device."""

    A: torch.Tensor  # [B, K, R, R]
    b: Optional[torch.Tensor]  # [B, K, R] or None
    lamK: torch.Tensor  # [B, R]
    widths: Tuple[int, ...]  # r_0..r_K
    workload: Workload

    def to(self, device) -> "Inputs":
        return Inputs(self.A.to(device), None if self.b is None else self.b.to(device),
                      self.lamK.to(device), self.widths, self.workload)

    def chains(self, idx) -> "Inputs":
        """The sub-batch of chains ``idx`` (a LongTensor or slice)."""
        A = self.A[idx]
        b = None if self.b is None else self.b[idx]
        lamK = self.lamK[idx]
        wl = self.workload.with_(B=A.shape[0])
        return Inputs(A.contiguous(), None if b is None else b.contiguous(),
                      lamK.contiguous(), self.widths, wl)


def _chunk_seed(seed: int, chunk: int) -> int:
    # Distinct, reproducible 63-bit seeds per (workload seed, chunk index).
    return (seed * 1_000_003 + chunk * 7_919 + 12_345) % (2**63 - 1)


def _haar(n: int, d: int, gen: torch.Generator, device) -> torch.Tensor:
    """n Haar-distributed d x d orthogonal matrices (float64).

    The Q of the QR factorisation G = QR of a Gaussian G with diag(R) > 0,
    which is unique and Haar-distributed (Mezzadri 2007).  On the CPU it comes
    from LAPACK's QR with the signs of diag(R) folded into Q; on a GPU from
    classical Gram-Schmidt with one re-orthogonalisation pass (CGS2), which
    produces the same positive-diagonal factor as batched matrix products.
    """
    G = torch.randn((n, d, d), generator=gen, device=device, dtype=torch.float64)
    if G.device.type == "cpu":
        Q, R = torch.linalg.qr(G)
        sgn = torch.sign(torch.diagonal(R, dim1=-2, dim2=-1))
        sgn = torch.where(sgn == 0, torch.ones_like(sgn), sgn)
        return Q * sgn.unsqueeze(-2)
    Q = torch.empty_like(G)
    for k in range(d):
        v = G[:, :, k:k + 1].clone()
        if k > 0:
            Qk = Q[:, :, :k]
            QkT = Qk.transpose(1, 2).contiguous()
            for _ in range(2):
                v = v - torch.bmm(Qk, torch.bmm(QkT, v))
        Q[:, :, k:k + 1] = v / torch.linalg.vector_norm(v, dim=1, keepdim=True)
    return Q


def _spectrum(n: int, k: int, kind: str, gen: torch.Generator, device) -> torch.Tensor:
    if kind == "uniform":
        return 0.9 + 0.2 * torch.rand((n, k), generator=gen, device=device, dtype=torch.float64)
    if kind == "orthogonal":
        return torch.ones((n, k), device=device, dtype=torch.float64)
    if kind == "concentrated":
        u = torch.rand((n, k - 1), generator=gen, device=device, dtype=torch.float64)
        rest = torch.exp(math.log(0.3) + u * (math.log(1.0) - math.log(0.3)))
        # s_1 = 2.5 * sqrt((s_1^2 + sum rest^2) / k)  =>  closed form below.
        s1 = torch.sqrt(6.25 * (rest * rest).sum(-1) / (k - 6.25))
        s = torch.cat([s1.unsqueeze(-1), rest], dim=-1)
        scale = torch.clamp(1.05 / s1, max=1.0).unsqueeze(-1)
        return s * scale
    raise ValueError(f"unknown spectrum {kind!r}")


def _round_storage(x: torch.Tensor, dtype: str) -> torch.Tensor:
    x = x.to(torch.float32)
    if dtype == "bf16":
        x = x.to(torch.bfloat16)
    return x


def generate(wl: Workload, device="cpu") -> Inputs:
    """Draw the operands of workload ``wl`` on ``device`` (seeded, chunked)."""
    device = torch.device(device)
    B, K, R = wl.B, wl.K, wl.r
    widths = wl.interface_widths()
    if len(widths) != K + 1 or max(widths) > R or min(widths) < 1:
        raise ValueError("widths must hold K+1 entries in [1, R]")
    sd = STORAGE[wl.dtype]
    A = torch.zeros((B, K, R, R), dtype=sd, device=device)
    b = torch.zeros((B, K, R), dtype=sd, device=device) if wl.affine else None
    lamK = torch.zeros((B, R), dtype=sd, device=device)
    # slots grouped by (r_j, r_{j+1}) so each group is one batched draw
    groups = {}
    for j in range(K):
        groups.setdefault((widths[j], widths[j + 1]), []).append(j)
    for c0 in range(0, B, CHUNK):
        c1 = min(B, c0 + CHUNK)
        n = c1 - c0
        gen = torch.Generator(device=device)
        gen.manual_seed(_chunk_seed(wl.seed, c0 // CHUNK))
        for (rj, rj1), slots in sorted(groups.items()):
            m = n * len(slots)
            kk = min(rj, rj1)
            Q1 = _haar(m, rj, gen, device)
            s = _spectrum(m, kk, wl.spectrum, gen, device)
            Q2 = _haar(m, rj1, gen, device)
            blk = (Q1[:, :, :kk] * s.unsqueeze(-2)) @ Q2[:, :kk, :]
            blk = _round_storage(blk, wl.dtype).view(n, len(slots), rj, rj1)
            sl = torch.tensor(slots, device=device)
            A[c0:c1, sl, :rj, :rj1] = blk
        if wl.affine:
            for j in range(K):
                rj = widths[j]
                bj = torch.randn((n, rj), generator=gen, device=device,
                                 dtype=torch.float64) / math.sqrt(rj)
                b[c0:c1, j, :rj] = _round_storage(bj, wl.dtype)
        rK = widths[K]
        lk = torch.randn((n, rK), generator=gen, device=device, dtype=torch.float64)
        lamK[c0:c1, :rK] = _round_storage(lk, wl.dtype)
    return Inputs(A, b, lamK, widths, wl)


# ----------------------------------------------------------------------------
# Structured inputs for edge cases and exactness checks.
# ----------------------------------------------------------------------------

def random_chain(B: int, K: int, r: int, dtype: str = "f32", seed: int = 0,
                 spectrum: str = "uniform", affine: bool = True,
                 widths: Optional[Tuple[int, ...]] = None, device="cpu") -> Inputs:
    """A random workload of arbitrary shape (same recipes as ``generate``)."""
    wl = Workload(f"random_B{B}_K{K}_r{r}", B=B, K=K, r=r, dtype=dtype, seed=seed,
                  spectrum=spectrum, affine=affine, widths=widths)
    return generate(wl, device)


def identity_chain(B: int, K: int, r: int, dtype: str = "f32", seed: int = 0,
                   device="cpu") -> Inputs:
    """A_j = I, no affine term, lambda_K ~ N(0, 1)."""
    sd = STORAGE[dtype]
    eye = torch.eye(r, dtype=torch.float32)
    A = eye.expand(B, K, r, r).to(sd).contiguous().to(device)
    gen = torch.Generator().manual_seed(_chunk_seed(seed, 999))
    lamK = _round_storage(torch.randn((B, r), generator=gen, dtype=torch.float64), dtype)
    wl = Workload(f"identity_B{B}_K{K}_r{r}", B, K, r, dtype, seed, "orthogonal", False)
    return Inputs(A, None, lamK.to(device), (r,) * (K + 1), wl)


def permutation_chain(B: int, K: int, r: int, dtype: str = "f32", seed: int = 0,
                      affine: bool = True, device="cpu") -> Inputs:
    """A_j random permutation matrices, b_j and lambda_K small integers.

    Every product, sum and output is an integer of magnitude below 2^8 * (K+1),
    so all of them are exact in float32 and the inputs are exact in bfloat16.
    """
    sd = STORAGE[dtype]
    gen = torch.Generator().manual_seed(_chunk_seed(seed, 4242))
    perm = torch.argsort(torch.rand((B, K, r), generator=gen), dim=-1)
    A = torch.zeros((B, K, r, r), dtype=torch.float32)
    A.scatter_(-1, perm.unsqueeze(-1), 1.0)
    b = None
    if affine:
        b = torch.randint(-8, 9, (B, K, r), generator=gen).to(torch.float32).to(sd).to(device)
    lamK = torch.randint(-8, 9, (B, r), generator=gen).to(torch.float32).to(sd).to(device)
    wl = Workload(f"perm_B{B}_K{K}_r{r}", B, K, r, dtype, seed, "orthogonal", affine)
    return Inputs(A.to(sd).to(device), b, lamK, (r,) * (K + 1), wl)


# ----------------------------------------------------------------------------
# compact (ragged) storage: layout only, no arithmetic
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class RaggedInputs:
    """The operands of ``Inputs`` with every tile cut to its true shape and the
    slots of a chain stored back to back: A [B, sum r_j r_{j+1}],
    b [B, sum r_j] or None, lamK [B, r_K] (the layout of the library's ragged
    entry point)."""

    A: torch.Tensor
    b: Optional[torch.Tensor]
    lamK: torch.Tensor
    widths: Tuple[int, ...]


def pack_ragged(x: Inputs) -> RaggedInputs:
    """Cut the zero-padded tiles of ``x`` to r_j x r_{j+1} and pack them."""
    w = x.widths
    K = len(w) - 1
    B = x.A.shape[0]
    A = torch.cat([x.A[:, j, :w[j], :w[j + 1]].reshape(B, -1) for j in range(K)], dim=1)
    b = None
    if x.b is not None:
        b = torch.cat([x.b[:, j, :w[j]] for j in range(K)], dim=1).contiguous()
    return RaggedInputs(A.contiguous(), b, x.lamK[:, :w[K]].contiguous(), tuple(w))


def unpack_ragged(lam: torch.Tensor, widths: Sequence[int], R: int) -> torch.Tensor:
    """lambda [B, sum r_j] in compact layout -> [B, K, R], zero-padded rows."""
    K = len(widths) - 1
    B = lam.shape[0]
    out = torch.zeros((B, K, R), dtype=lam.dtype, device=lam.device)
    o = 0
    for j in range(K):
        out[:, j, :widths[j]] = lam[:, o:o + widths[j]]
        o += widths[j]
    return out


# ----------------------------------------------------------------------------
# Phase 1 inputs: a synthetic bounded-interface region map with random weights
# ----------------------------------------------------------------------------
#
# Region k maps the interface state m_k (r values per sequence) to
#   m_{k+1} = LN(m_k + alpha_k Enc_k(pool(Phi_k(x_embed + Dec_k(m_k)))))
# (Eq. "concrete-region-arch").  The parameters drawn here, per region k:
#   Dec_k = 2-layer MLP r -> D -> D:  W_d1 [D, r], b_d1 [D], W_d2 [D, D], b_d2 [D]
#   Phi_k = token-wise residual MLP D -> X -> D:  W1 [X, D], W2 [D, X]
#   Enc_k = 2-layer MLP D -> D -> r:  W_e1 [D, D], b_e1 [D], W_e2 [r, D], b_e2 [r]
#   alpha_k (scalar), LN gain gamma [r] and shift beta [r];
#   decay a_k [D] for the token-mixing block (Phi_k with a causal recurrence
#   s_l = a_k s_{l-1} + (1 - a_k) x_l over the tokens, then
#   Phi_k(x)_l = x_l + (W2 silu(W1 s_l)) silu(s_l)), unused by the token-wise one.
# Matrices ~ N(0, 1/fan_in), rounded to bf16; biases ~ N(0, 0.01) and the
# rest in fp32.  x_embed [B, L, D] ~ N(0, 1) in bf16; m [B, K, r] ~ N(0, 1) in
# fp32 (each region's Jacobian depends only on its own m_k and x_embed).

@dataclasses.dataclass(frozen=True)
class RegionWorkload:
    name: str
    B: int  # sequences
    K: int  # regions
    L: int  # tokens per sequence
    D: int  # model width
    X: int  # width of the region MLP
    r: int  # interface width
    seed: int


REGION_WORKLOADS = {
    # The illustrative configuration of the paper's cost analysis (about 1B
    # parameters): B=8, L=2048, D=768, X=3072 (Transformer MLP width), r=64,
    # K=16 (32 layers at 2 layers per region).
    "region_paper": RegionWorkload("region_paper", B=8, K=16, L=2048, D=768, X=3072, r=64,
                                   seed=5),
    # small enough for the fp64 autograd oracle in seconds
    "region_small": RegionWorkload("region_small", B=2, K=3, L=256, D=128, X=256, r=32, seed=6),
}

REGION_MATRICES = ("W_d1", "W_d2", "W1", "W2", "W_e1", "W_e2")
REGION_VECTORS = ("b_d1", "b_d2", "b_e1", "b_e2", "alpha", "gamma", "beta")


@dataclasses.dataclass
class RegionInputs:
    params: dict  # name -> tensor, stacked over the K regions
    x_embed: torch.Tensor  # [B, L, D] bf16
    m: torch.Tensor  # [B, K, r] fp32
    workload: RegionWorkload

    def to(self, device) -> "RegionInputs":
        return RegionInputs({k: v.to(device) for k, v in self.params.items()},
                            self.x_embed.to(device), self.m.to(device), self.workload)


def generate_region(wl: RegionWorkload, device="cpu") -> RegionInputs:
    """Draw the region parameters, x_embed and m of ``wl`` (seeded)."""
    device = torch.device(device)
    gen = torch.Generator(device=device)
    gen.manual_seed(_chunk_seed(wl.seed, 777))
    K, D, X, r = wl.K, wl.D, wl.X, wl.r

    def mat(rows, cols):
        w = torch.randn((K, rows, cols), generator=gen, device=device, dtype=torch.float64)
        return (w / math.sqrt(cols)).to(torch.float32).to(torch.bfloat16)

    def vec(n, scale=0.1):
        v = torch.randn((K, n), generator=gen, device=device, dtype=torch.float64) * scale
        return v.to(torch.float32)

    p = {"W_d1": mat(D, r), "b_d1": vec(D), "W_d2": mat(D, D), "b_d2": vec(D),
         "W1": mat(X, D), "W2": mat(D, X),
         "W_e1": mat(D, D), "b_e1": vec(D), "W_e2": mat(r, D), "b_e2": vec(r)}
    p["alpha"] = (0.5 + 0.5 * torch.rand((K,), generator=gen, device=device,
                                         dtype=torch.float64)).to(torch.float32)
    p["gamma"] = (1.0 + vec(r)).contiguous()
    p["beta"] = vec(r)
    x = torch.randn((wl.B, wl.L, D), generator=gen, device=device, dtype=torch.float64)
    m = torch.randn((wl.B, K, r), generator=gen, device=device, dtype=torch.float64)
    # the token-mixing block's per-channel state decay a_k in [0.9, 0.999]
    # (1 - a log-uniform over [1e-3, 1e-1]: memories of about 10 to 1000
    # tokens), drawn last so that the other parameters do not depend on it
    u = torch.rand((K, D), generator=gen, device=device, dtype=torch.float64)
    p["decay"] = (1.0 - 10.0 ** (-3.0 + 2.0 * u)).to(torch.float32)
    return RegionInputs(p, x.to(torch.float32).to(torch.bfloat16), m.to(torch.float32), wl)
