"""Python binding of the C-ABI in ``include/lbi.h`` (argument marshalling only).

Every function has the name of the C entry point it calls.  Tensors are torch
tensors on the current GPU; torch provides device memory and the stream (the
current torch stream unless one is given).  All arithmetic runs in the HIP
library; if the library is not built, the first call raises ``RuntimeError``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "liblbi.so")

LBI_F32 = 0
LBI_BF16 = 1
LBI_OK = 0
LBI_MAX_HINT_K = 2047
LBI_MATH_DEFAULT = 0
LBI_MATH_F32_MFMA = 1
LBI_MATH_F32_SPLIT = 2
LBI_MATH_BF16_SINGLE = 3
LBI_ALGO_AUTO = 0
LBI_ALGO_CHAIN = 1
LBI_ALGO_TWO_LEVEL = 2
LBI_ALGO_CHAIN_WAVE = 3
LBI_ALGO_CHAIN_SPLITK = 4
LBI_ALGO_TREE = 5
LBI_ALGO_CHAIN_RING = 6
LBI_ERR_SCRATCH = 9
LBI_BF16_SINGLE_MAX_K = 64
LBI_NOALLOC_SCRATCH_BYTES = 64 << 20

_DTYPES = {torch.float32: LBI_F32, torch.bfloat16: LBI_BF16}

# lbi_region_params, in declaration order: (name, dtype, shape given K, D, X, r)
REGION_PARAM_FIELDS = (
    ("W_d1", torch.bfloat16, lambda K, D, X, r: (K, D, r)),
    ("b_d1", torch.float32, lambda K, D, X, r: (K, D)),
    ("W_d2", torch.bfloat16, lambda K, D, X, r: (K, D, D)),
    ("b_d2", torch.float32, lambda K, D, X, r: (K, D)),
    ("W1", torch.bfloat16, lambda K, D, X, r: (K, X, D)),
    ("W2", torch.bfloat16, lambda K, D, X, r: (K, D, X)),
    ("W_e1", torch.bfloat16, lambda K, D, X, r: (K, D, D)),
    ("b_e1", torch.float32, lambda K, D, X, r: (K, D)),
    ("W_e2", torch.bfloat16, lambda K, D, X, r: (K, r, D)),
    ("b_e2", torch.float32, lambda K, D, X, r: (K, r)),
    ("alpha", torch.float32, lambda K, D, X, r: (K,)),
    ("gamma", torch.float32, lambda K, D, X, r: (K, r)),
    ("beta", torch.float32, lambda K, D, X, r: (K, r)),
)


class RegionParams(ctypes.Structure):
    """lbi_region_params: device pointers of the K regions' parameters."""
    _fields_ = [(name, ctypes.c_void_p) for name, _, _ in REGION_PARAM_FIELDS]

_lib = None


class LbiError(RuntimeError):
    """A non-OK lbi_status from the library."""

    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


def library_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Load the HIP library (raises RuntimeError when it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(
            f"HIP library not built: {_LIB_PATH} is missing "
            "(run `python -m paper_2605_09204_amd.build`)")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    lib.lbi_scan_backward_workspace_bytes.argtypes = [i64, i64, i32, ctypes.c_int]
    lib.lbi_scan_backward_workspace_bytes.restype = sz
    lib.lbi_scan_backward_workspace_bytes_ex.argtypes = [i64, i64, i32, ctypes.c_int,
                                                         ctypes.c_int]
    lib.lbi_scan_backward_workspace_bytes_ex.restype = sz
    lib.lbi_scan_backward.argtypes = [vp, vp, vp, vp, i64, i64, i32, ctypes.c_int, vp, sz, vp]
    lib.lbi_scan_backward.restype = ctypes.c_int
    lib.lbi_scan_backward_widths.argtypes = [vp, vp, vp, vp, i64, i64, i32, ctypes.c_int, vp,
                                             sz, vp, ctypes.POINTER(ctypes.c_int32)]
    lib.lbi_scan_backward_widths.restype = ctypes.c_int
    lib.lbi_scan_backward_ex.argtypes = [vp, vp, vp, vp, i64, i64, i32, ctypes.c_int, vp, sz,
                                         vp, ctypes.POINTER(ctypes.c_int32), ctypes.c_int,
                                         ctypes.c_int]
    lib.lbi_scan_backward_ex.restype = ctypes.c_int
    lib.lbi_scan_suffix_products.argtypes = [vp, vp, vp, vp, i64, i64, i32, ctypes.c_int, vp,
                                             ctypes.POINTER(ctypes.c_int32), ctypes.c_int]
    lib.lbi_scan_suffix_products.restype = ctypes.c_int
    lib.lbi_scan_backward_streaming.argtypes = [vp, vp, vp, vp, i64, i64, i32, ctypes.c_int, vp,
                                                ctypes.POINTER(ctypes.c_int32), ctypes.c_int,
                                                vp, i32, vp]
    lib.lbi_scan_backward_streaming.restype = ctypes.c_int
    lib.lbi_wait_progress.argtypes = [vp, i64, ctypes.c_uint32, i64, vp, vp, vp]
    lib.lbi_wait_progress.restype = ctypes.c_int
    lib.lbi_scan_backward_noalloc.argtypes = [vp, vp, vp, vp, i64, i64, i32, ctypes.c_int, vp,
                                              ctypes.POINTER(ctypes.c_int32), ctypes.c_int,
                                              ctypes.c_int]
    lib.lbi_scan_backward_noalloc.restype = ctypes.c_int
    lib.lbi_scan_backward_ragged.argtypes = [vp, vp, vp, vp, i64, i64,
                                             ctypes.POINTER(ctypes.c_int32), ctypes.c_int, vp,
                                             ctypes.c_int]
    lib.lbi_scan_backward_ragged.restype = ctypes.c_int
    lib.lbi_region_jacobians_workspace_bytes.argtypes = [i64, i64, i64, i32, i32, i32]
    lib.lbi_region_jacobians_workspace_bytes.restype = sz
    lib.lbi_region_jacobians.argtypes = [ctypes.POINTER(RegionParams), vp, vp, vp, vp, i64, i64,
                                         i64, i32, i32, i32, vp, sz, vp]
    lib.lbi_region_jacobians.restype = ctypes.c_int
    lib.lbi_region_jacobians_ssm_workspace_bytes.argtypes = [i64, i64, i64, i32, i32, i32]
    lib.lbi_region_jacobians_ssm_workspace_bytes.restype = sz
    lib.lbi_region_jacobians_ssm.argtypes = [ctypes.POINTER(RegionParams), vp, vp, vp, vp, vp,
                                             i64, i64, i64, i32, i32, i32, vp, sz, vp]
    lib.lbi_region_jacobians_ssm.restype = ctypes.c_int
    lib.lbi_matrix_norms.argtypes = [vp, i64, i32, ctypes.c_int, vp, vp, vp]
    lib.lbi_matrix_norms.restype = ctypes.c_int
    lib.lbi_status_string.argtypes = [ctypes.c_int]
    lib.lbi_status_string.restype = ctypes.c_char_p
    lib.lbi_abi_version.argtypes = []
    lib.lbi_abi_version.restype = ctypes.c_int
    _lib = lib
    return lib


def lbi_status_string(status: int) -> str:
    return load().lbi_status_string(int(status)).decode()


def lbi_abi_version() -> int:
    return int(load().lbi_abi_version())


def lbi_scan_backward_workspace_bytes(B: int, K: int, r: int, dt: int) -> int:
    return int(load().lbi_scan_backward_workspace_bytes(int(B), int(K), int(r), int(dt)))


def lbi_scan_backward_workspace_bytes_ex(B: int, K: int, r: int, dt: int, algo: int) -> int:
    return int(load().lbi_scan_backward_workspace_bytes_ex(int(B), int(K), int(r), int(dt),
                                                            int(algo)))


def _check(status: int) -> None:
    if status != LBI_OK:
        raise LbiError(status, lbi_status_string(status))


def _stream_ptr(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _marshal(A: torch.Tensor, b: Optional[torch.Tensor], lambda_K: torch.Tensor,
             lam: Optional[torch.Tensor], workspace: Optional[torch.Tensor], stream,
             algo: int = LBI_ALGO_AUTO):
    if A.dim() != 4 or A.shape[2] != A.shape[3]:
        raise ValueError(f"A must be [B, K, r, r], got {tuple(A.shape)}")
    B, K, r = int(A.shape[0]), int(A.shape[1]), int(A.shape[2])
    if A.dtype not in _DTYPES:
        raise TypeError(f"A must be float32 or bfloat16, got {A.dtype}")
    dt = _DTYPES[A.dtype]
    for name, t, shape in (("b", b, (B, K, r)), ("lambda_K", lambda_K, (B, r))):
        if t is None:
            continue
        if tuple(t.shape) != shape or t.dtype != A.dtype or t.device != A.device:
            raise ValueError(f"{name} must be {shape} {A.dtype} on {A.device}")
    tensors = [A, lambda_K] + ([b] if b is not None else [])
    if not A.is_cuda:
        raise ValueError("tensors must be on a GPU device")
    if not all(t.is_contiguous() for t in tensors):
        raise ValueError("tensors must be contiguous")
    if lam is None:
        lam = torch.empty((B, K, r), dtype=torch.float32, device=A.device)
    elif tuple(lam.shape) != (B, K, r) or lam.dtype != torch.float32 or not lam.is_contiguous() \
            or lam.device != A.device:
        raise ValueError("lambda must be a contiguous float32 [B, K, r] tensor on A's device")
    need = lbi_scan_backward_workspace_bytes_ex(B, K, r, dt, algo)
    if workspace is None and need > 0:
        workspace = torch.empty((need,), dtype=torch.uint8, device=A.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    s_ptr = _stream_ptr(stream, A.device)
    args = (A.data_ptr(), b.data_ptr() if b is not None else None, lambda_K.data_ptr(),
            lam.data_ptr(), B, K, r, dt, ws_ptr, ws_bytes, s_ptr)
    return lam, args


def lbi_scan_backward(A: torch.Tensor, b: Optional[torch.Tensor], lambda_K: torch.Tensor,
                      lam: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """lambda[B, K, r] (float32) = every interface adjoint; see include/lbi.h."""
    lam, args = _marshal(A, b, lambda_K, lam, workspace, stream)
    _check(load().lbi_scan_backward(*args))
    return lam


def _widths_arg(widths, K):
    if widths is None:
        return None, None
    if len(widths) != K + 1:
        raise ValueError("widths must hold K+1 entries")
    warr = (ctypes.c_int32 * len(widths))(*[int(x) for x in widths])
    return warr, ctypes.cast(warr, ctypes.POINTER(ctypes.c_int32))


def lbi_scan_backward_widths(A: torch.Tensor, b: Optional[torch.Tensor],
                             lambda_K: torch.Tensor, widths: Optional[Sequence[int]],
                             lam: Optional[torch.Tensor] = None,
                             workspace: Optional[torch.Tensor] = None,
                             stream=None) -> torch.Tensor:
    """As lbi_scan_backward with the interface widths r_0..r_K as a hint."""
    lam, args = _marshal(A, b, lambda_K, lam, workspace, stream)
    warr, wptr = _widths_arg(widths, int(A.shape[1]))
    _check(load().lbi_scan_backward_widths(*args, wptr))
    return lam


def lbi_scan_backward_ex(A: torch.Tensor, b: Optional[torch.Tensor], lambda_K: torch.Tensor,
                         widths: Optional[Sequence[int]] = None, math: int = LBI_MATH_DEFAULT,
                         algo: int = LBI_ALGO_AUTO, lam: Optional[torch.Tensor] = None,
                         workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """As lbi_scan_backward_widths, with the arithmetic chosen by ``math``
    and the scan by ``algo``."""
    lam, args = _marshal(A, b, lambda_K, lam, workspace, stream, algo)
    warr, wptr = _widths_arg(widths, int(A.shape[1]))
    _check(load().lbi_scan_backward_ex(*args, wptr, int(math), int(algo)))
    return lam


def lbi_scan_backward_noalloc(A: torch.Tensor, b: Optional[torch.Tensor],
                              lambda_K: torch.Tensor, widths: Optional[Sequence[int]] = None,
                              math: int = LBI_MATH_DEFAULT, algo: int = LBI_ALGO_AUTO,
                              lam: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """As lbi_scan_backward_ex, with the library's static scratch array in
    place of a workspace (the call itself allocates nothing; ``lam`` may be
    passed to keep the binding from allocating the output)."""
    lam, args = _marshal(A, b, lambda_K, lam, None, stream, LBI_ALGO_CHAIN)
    Aptr, bptr, lkptr, lamptr, B_, K, r, dt, _ws, _wsb, sptr = args
    warr, wptr = _widths_arg(widths, int(A.shape[1]))
    _check(load().lbi_scan_backward_noalloc(Aptr, bptr, lkptr, lamptr, B_, K, r, dt, sptr, wptr,
                                            int(math), int(algo)))
    return lam


def lbi_scan_suffix_products(A: torch.Tensor, b: Optional[torch.Tensor],
                             widths: Optional[Sequence[int]] = None,
                             math: int = LBI_MATH_DEFAULT, P: Optional[torch.Tensor] = None,
                             c: Optional[torch.Tensor] = None, want_c: bool = True,
                             stream=None):
    """(P[B, K, r, r], c[B, K, r] or None), float32: the suffix composites."""
    if A.dim() != 4 or A.shape[2] != A.shape[3] or A.dtype not in _DTYPES or not A.is_cuda:
        raise ValueError("A must be a [B, K, r, r] float32/bfloat16 GPU tensor")
    if not A.is_contiguous() or (b is not None and not b.is_contiguous()):
        raise ValueError("tensors must be contiguous")
    B, K, r = int(A.shape[0]), int(A.shape[1]), int(A.shape[2])
    if b is not None and (tuple(b.shape) != (B, K, r) or b.dtype != A.dtype
                          or b.device != A.device):
        raise ValueError(f"b must be {(B, K, r)} {A.dtype} on {A.device}")
    if P is None:
        P = torch.empty((B, K, r, r), dtype=torch.float32, device=A.device)
    if want_c and c is None:
        c = torch.empty((B, K, r), dtype=torch.float32, device=A.device)
    for name, t, shape in (("P", P, (B, K, r, r)), ("c", c, (B, K, r))):
        if t is not None and (tuple(t.shape) != shape or t.dtype != torch.float32
                              or not t.is_contiguous() or t.device != A.device):
            raise ValueError(f"{name} must be a contiguous float32 {shape} tensor on A's device")
    warr, wptr = _widths_arg(widths, K)
    _check(load().lbi_scan_suffix_products(
        A.data_ptr(), b.data_ptr() if b is not None else None, P.data_ptr(),
        c.data_ptr() if c is not None else None, B, K, r, _DTYPES[A.dtype],
        _stream_ptr(stream, A.device), wptr, int(math)))
    return P, c


def lbi_scan_backward_streaming(A: torch.Tensor, b: Optional[torch.Tensor],
                                lambda_K: torch.Tensor, progress: torch.Tensor, chunk: int,
                                widths: Optional[Sequence[int]] = None,
                                math: int = LBI_MATH_DEFAULT, lam: Optional[torch.Tensor] = None,
                                stream=None,
                                publish_clock: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The chain scan, raising progress[beta] (int32/uint32 [B] GPU tensor, zeroed by
    the caller) to the count of final adjoints every ``chunk`` slots; with
    ``publish_clock`` (int64 [B, ceil(K / chunk)] GPU tensor) the real-time
    counter of each publication is recorded there."""
    lam, args = _marshal(A, b, lambda_K, lam, None, stream, LBI_ALGO_CHAIN)
    B = int(A.shape[0])
    if (progress.dim() != 1 or progress.shape[0] != B or progress.dtype not in
            (torch.int32, torch.uint32) or not progress.is_contiguous()
            or progress.device != A.device):
        raise ValueError(f"progress must be a contiguous 32-bit [{B}] tensor on A's device")
    warr, wptr = _widths_arg(widths, int(A.shape[1]))
    Aptr, bptr, lkptr, lamptr, B_, K, r, dt, _ws, _wsb, sptr = args
    cptr = None
    if publish_clock is not None:
        npub = -(-int(A.shape[1]) // int(chunk)) if int(chunk) > 0 else 0
        if (publish_clock.dtype not in (torch.int64, torch.uint64)
                or tuple(publish_clock.shape) != (B, npub)
                or not publish_clock.is_contiguous() or publish_clock.device != A.device):
            raise ValueError(f"publish_clock must be a contiguous 64-bit [{B}, {npub}] tensor "
                             "on A's device")
        cptr = publish_clock.data_ptr()
    _check(load().lbi_scan_backward_streaming(Aptr, bptr, lkptr, lamptr, B_, K, r, dt, sptr,
                                              wptr, int(math), progress.data_ptr(),
                                              int(chunk), cptr))
    return lam


def lbi_wait_progress(progress: torch.Tensor, target: int, max_polls: int,
                      released: Optional[torch.Tensor] = None,
                      release_clock: Optional[torch.Tensor] = None, stream=None) -> None:
    """Enqueue on ``stream`` (default: the current stream) a wait until every
    progress[beta] >= target, giving up after ``max_polls`` polls.  ``released``
    (32-bit [1] GPU tensor) receives 1 / 0 (satisfied / gave up),
    ``release_clock`` (64-bit [1] GPU tensor) the real-time counter at the end."""
    if (progress.dim() != 1 or progress.dtype not in (torch.int32, torch.uint32)
            or not progress.is_contiguous() or not progress.is_cuda):
        raise ValueError("progress must be a contiguous 32-bit [B] GPU tensor")
    for t, dts, name in ((released, (torch.int32, torch.uint32), "released"),
                         (release_clock, (torch.int64, torch.uint64), "release_clock")):
        if t is not None and (t.dtype not in dts or t.numel() < 1 or not t.is_cuda
                              or t.device != progress.device):
            raise ValueError(f"{name} must be a GPU tensor of {dts} on progress's device")
    _check(load().lbi_wait_progress(
        progress.data_ptr(), int(progress.shape[0]), int(target) & 0xFFFFFFFF, int(max_polls),
        None if released is None else released.data_ptr(),
        None if release_clock is None else release_clock.data_ptr(),
        _stream_ptr(stream, progress.device)))


def lbi_matrix_norms(M: torch.Tensor, want_spec: bool = True, want_fro: bool = True,
                     spec: Optional[torch.Tensor] = None, fro: Optional[torch.Tensor] = None,
                     stream=None):
    """(||M_i||_2, ||M_i||_F / sqrt(r)) as float32 tensors of M's leading shape
    (None where not wanted) for a [..., r, r] float32/bfloat16 GPU tensor M."""
    if M.dim() < 2 or M.shape[-1] != M.shape[-2] or M.dtype not in _DTYPES or not M.is_cuda:
        raise ValueError("M must be a [..., r, r] float32/bfloat16 GPU tensor")
    if not M.is_contiguous():
        raise ValueError("M must be contiguous")
    lead = tuple(M.shape[:-2])
    r = int(M.shape[-1])
    n = 1
    for d in lead:
        n *= int(d)
    if want_spec and spec is None:
        spec = torch.empty(lead, dtype=torch.float32, device=M.device)
    if want_fro and fro is None:
        fro = torch.empty(lead, dtype=torch.float32, device=M.device)
    for name, t in (("spec", spec), ("fro", fro)):
        if t is not None and (tuple(t.shape) != lead or t.dtype != torch.float32
                              or not t.is_contiguous() or t.device != M.device):
            raise ValueError(f"{name} must be a contiguous float32 {lead} tensor on M's device")
    _check(load().lbi_matrix_norms(
        M.data_ptr(), n, r, _DTYPES[M.dtype], spec.data_ptr() if spec is not None else None,
        fro.data_ptr() if fro is not None else None, _stream_ptr(stream, M.device)))
    return spec, fro


def lbi_scan_backward_ragged(A: torch.Tensor, b: Optional[torch.Tensor], lambda_K: torch.Tensor,
                             widths: Sequence[int], math: int = LBI_MATH_DEFAULT,
                             lam: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """lambda [B, SR] (float32) from compact ragged storage: A [B, SA], b [B, SR] or None,
    lambda_K [B, r_K], with SA = sum r_j r_{j+1} and SR = sum r_j over j < K."""
    K = len(widths) - 1
    if K < 1:
        raise ValueError("widths must hold K+1 >= 2 entries")
    SA = sum(int(widths[j]) * int(widths[j + 1]) for j in range(K))
    SR = sum(int(widths[j]) for j in range(K))
    if A.dim() != 2 or A.shape[1] != SA or A.dtype not in _DTYPES or not A.is_cuda:
        raise ValueError(f"A must be a [B, {SA}] float32/bfloat16 GPU tensor")
    B = int(A.shape[0])
    for name, t, shape in (("b", b, (B, SR)), ("lambda_K", lambda_K, (B, int(widths[K])))):
        if t is not None and (tuple(t.shape) != shape or t.dtype != A.dtype
                              or t.device != A.device):
            raise ValueError(f"{name} must be {shape} {A.dtype} on {A.device}")
    if not all(t.is_contiguous() for t in (A, lambda_K) + ((b,) if b is not None else ())):
        raise ValueError("tensors must be contiguous")
    if lam is None:
        lam = torch.empty((B, SR), dtype=torch.float32, device=A.device)
    elif (tuple(lam.shape) != (B, SR) or lam.dtype != torch.float32 or not lam.is_contiguous()
          or lam.device != A.device):
        raise ValueError(f"lambda must be a contiguous float32 [B, {SR}] tensor on A's device")
    warr, wptr = _widths_arg(widths, K)
    _check(load().lbi_scan_backward_ragged(
        A.data_ptr(), b.data_ptr() if b is not None else None, lambda_K.data_ptr(),
        lam.data_ptr(), B, K, wptr, _DTYPES[A.dtype], _stream_ptr(stream, A.device),
        int(math)))
    return lam


def lbi_region_jacobians_workspace_bytes(B: int, K: int, L: int, D: int, X: int, r: int) -> int:
    return int(load().lbi_region_jacobians_workspace_bytes(int(B), int(K), int(L), int(D),
                                                            int(X), int(r)))


def lbi_region_jacobians_ssm_workspace_bytes(B: int, K: int, L: int, D: int, X: int,
                                             r: int) -> int:
    return int(load().lbi_region_jacobians_ssm_workspace_bytes(int(B), int(K), int(L), int(D),
                                                                int(X), int(r)))


def lbi_region_jacobians_ssm(params: dict, x_embed: torch.Tensor, m: torch.Tensor,
                             A: Optional[torch.Tensor] = None,
                             m_next: Optional[torch.Tensor] = None, want_m_next: bool = True,
                             workspace: Optional[torch.Tensor] = None, stream=None):
    """As ``lbi_region_jacobians`` for the token-mixing region block, whose
    per-channel decay is params["decay"] ([K, D] float32)."""
    return lbi_region_jacobians(params, x_embed, m, A, m_next, want_m_next, workspace, stream,
                                _ssm=True)


def lbi_region_jacobians(params: dict, x_embed: torch.Tensor, m: torch.Tensor,
                         A: Optional[torch.Tensor] = None, m_next: Optional[torch.Tensor] = None,
                         want_m_next: bool = True, workspace: Optional[torch.Tensor] = None,
                         stream=None, _ssm: bool = False):
    """(A [B, K, r, r] = J_k^T, m_next [B, K, r] or None), float32: Phase 1 for the
    synthetic region map (include/lbi.h), from the parameter dict of
    ``REGION_PARAM_FIELDS``, x_embed [B, L, D] bf16 and m [B, K, r] float32."""
    if x_embed.dim() != 3 or x_embed.dtype != torch.bfloat16 or not x_embed.is_cuda:
        raise ValueError("x_embed must be a [B, L, D] bfloat16 GPU tensor")
    B, L, D = (int(v) for v in x_embed.shape)
    if m.dim() != 3 or m.shape[0] != B or m.dtype != torch.float32 or m.device != x_embed.device:
        raise ValueError("m must be a [B, K, r] float32 tensor on x_embed's device")
    K, r = int(m.shape[1]), int(m.shape[2])
    X = int(params["W1"].shape[1])
    ptrs = []
    for name, dt, shape in REGION_PARAM_FIELDS:
        t = params[name]
        if (tuple(t.shape) != shape(K, D, X, r) or t.dtype != dt or not t.is_contiguous()
                or t.device != x_embed.device):
            raise ValueError(f"{name} must be a contiguous {dt} {shape(K, D, X, r)} tensor "
                             "on x_embed's device")
        ptrs.append(t.data_ptr())
    if not (x_embed.is_contiguous() and m.is_contiguous()):
        raise ValueError("tensors must be contiguous")
    if A is None:
        A = torch.empty((B, K, r, r), dtype=torch.float32, device=x_embed.device)
    if want_m_next and m_next is None:
        m_next = torch.empty((B, K, r), dtype=torch.float32, device=x_embed.device)
    rp = RegionParams(*ptrs)
    tail = (m.data_ptr(), A.data_ptr(), m_next.data_ptr() if m_next is not None else None,
            B, K, L, D, X, r)
    if _ssm:
        dec = params["decay"]
        if (tuple(dec.shape) != (K, D) or dec.dtype != torch.float32 or not dec.is_contiguous()
                or dec.device != x_embed.device):
            raise ValueError(f"decay must be a contiguous float32 {(K, D)} tensor on x_embed's "
                             "device")
        need = lbi_region_jacobians_ssm_workspace_bytes(B, K, L, D, X, r)
    else:
        need = lbi_region_jacobians_workspace_bytes(B, K, L, D, X, r)
    if workspace is None and need > 0:
        workspace = torch.empty((need,), dtype=torch.uint8, device=x_embed.device)
    ws = (workspace.data_ptr() if workspace is not None else None,
          workspace.numel() if workspace is not None else 0, _stream_ptr(stream, x_embed.device))
    if _ssm:
        _check(load().lbi_region_jacobians_ssm(ctypes.byref(rp), dec.data_ptr(),
                                               x_embed.data_ptr(), *tail, *ws))
    else:
        _check(load().lbi_region_jacobians(ctypes.byref(rp), x_embed.data_ptr(), *tail, *ws))
    return A, m_next
