"""The C-ABI library loads, exports what include/lbi.h declares, and rejects
bad arguments before touching the GPU (runs without a GPU: no call here
reaches a HIP API)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2605_09204_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lbi.h")

pytestmark = pytest.mark.skipif(not os.path.exists(binding.library_path()),
                                reason="library not built")

# fake device addresses: never dereferenced, only validated
PA, PB, PL, POUT = 0x10000000, 0x20000000, 0x30000000, 0x40000000


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lbi_[a-z_]+)\s*\(", text)))


def test_header_declares_entry_points():
    names = declared_functions()
    assert names == sorted(["lbi_scan_backward_workspace_bytes",
                            "lbi_scan_backward_workspace_bytes_ex", "lbi_scan_backward",
                            "lbi_scan_backward_widths", "lbi_scan_backward_ex",
                            "lbi_scan_suffix_products", "lbi_scan_backward_streaming",
                            "lbi_matrix_norms", "lbi_scan_backward_ragged",
                            "lbi_region_jacobians_workspace_bytes", "lbi_region_jacobians",
                            "lbi_region_jacobians_ssm_workspace_bytes",
                            "lbi_region_jacobians_ssm", "lbi_wait_progress", "lbi_scan_backward_noalloc",
                            "lbi_status_string", "lbi_abi_version"])


def test_library_exports_every_declared_symbol():
    lib = binding.load()
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", binding.library_path()],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\b(lbi_[a-z_]+)\b", out))
    assert set(declared_functions()) <= exported


def test_header_compiles_as_c():
    src = '#include "lbi.h"\nint main(void){return lbi_abi_version()==LBI_ABI_VERSION?0:1;}\n'
    res = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-fsyntax-only",
                          f"-I{os.path.join(ROOT, 'include')}", "-x", "c", "-"],
                         input=src, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr


def test_version_and_status_strings():
    assert binding.lbi_abi_version() == 12
    assert binding.lbi_status_string(0) == "LBI_OK"
    for code in range(1, 10):
        assert binding.lbi_status_string(code).startswith("LBI_ERR_")
    assert "unknown" in binding.lbi_status_string(99)


def call(A=PA, b=PB, L=PL, out=POUT, B=2, K=3, r=64, dt=0, ws=None, wsb=0, widths=None,
         math=None, algo=0):
    lib = binding.load()
    if math is not None or algo:
        return lib.lbi_scan_backward_ex(A, b, L, out, B, K, r, dt, ws, wsb, None, None,
                                        math or 0, algo)
    if widths is None:
        return lib.lbi_scan_backward(A, b, L, out, B, K, r, dt, ws, wsb, None)
    arr = (ctypes.c_int32 * len(widths))(*widths)
    return lib.lbi_scan_backward_widths(A, b, L, out, B, K, r, dt, ws, wsb, None,
                                        ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)))


def test_argument_errors():
    assert call(dt=7) == 3                      # LBI_ERR_DTYPE
    assert call(math=4) == 3 and call(math=-1) == 3 and call(dt=1, math=9) == 3
    for r in (0, 8, 48, 96, 256):
        assert call(r=r) == 4                   # LBI_ERR_UNSUPPORTED_R
    assert call(K=0) == 2 and call(B=-1) == 2   # LBI_ERR_SHAPE
    assert call(B=2**40, K=2**20) == 2          # size overflow
    assert call(A=None) == 1 and call(L=None) == 1 and call(out=None) == 1
    assert call(A=PA + 4) == 7 and call(out=POUT + 8) == 7 and call(b=PB + 2) == 7
    # lambda overlapping A / b / lambda_K
    assert call(out=PA + 256) == 8
    assert call(out=PB) == 8
    assert call(out=PL - 16) == 8
    # widths out of range
    assert call(widths=[64, 64, 0, 64]) == 2
    assert call(widths=[64, 65, 64, 64]) == 2


def test_empty_batch_is_a_noop():
    # B = 0 succeeds without touching pointers or the GPU
    assert call(B=0, A=None, L=None, out=None) == 0


def test_workspace_query():
    for r in (16, 32, 64, 128):
        for dt in (0, 1):
            # short chains: the chain scan, no workspace
            assert binding.lbi_scan_backward_workspace_bytes(4, 8, r, dt) == 0
            # many chains: the chain scan fills the GPU by itself
            assert binding.lbi_scan_backward_workspace_bytes(4096, 512, r, dt) == 0
            assert binding.lbi_scan_backward_workspace_bytes_ex(4096, 64, r, dt, 1) == 0
            # few long chains: the two-level scan keeps composites and carries
            need = binding.lbi_scan_backward_workspace_bytes(2, 512, r, dt)
            assert need >= 2 * 512 * r * (r + 1) * 4
            assert binding.lbi_scan_backward_workspace_bytes_ex(2, 512, r, dt, 2) == need
            assert binding.lbi_scan_backward_workspace_bytes_ex(2, 512, r, dt, 1) == 0
            assert need <= 2 * 512 * r * (r + 1) * 4 + 2 * 64 * r * 4 + 3 * 256
    assert binding.lbi_scan_backward_workspace_bytes_ex(2, 512, 64, 0, 7) == 0
    assert binding.lbi_scan_backward_workspace_bytes(2, 512, 48, 0) == 0


def test_two_level_needs_workspace():
    # the two-level path checks its workspace before touching the GPU
    assert call(B=2, K=512, algo=2) == 5                 # LBI_ERR_WORKSPACE
    need = binding.lbi_scan_backward_workspace_bytes_ex(2, 512, 64, 0, 2)
    assert call(B=2, K=512, algo=2, ws=0x50000000, wsb=need - 1) == 5
    assert call(B=2, K=512, algo=2, ws=0x50000008, wsb=need) == 7  # misaligned
    # workspace overlapping an input
    assert call(B=2, K=512, algo=2, ws=PA + 64, wsb=need) == 8
    assert call(B=2, K=512, algo=9) == 3


def test_chain_wave_argument_errors():
    # one wavefront per chain: bf16 storage and r <= 64 only, no workspace;
    # rejected before any pointer is touched
    assert call(algo=3) == 3                    # fp32 storage: LBI_ERR_DTYPE
    assert call(dt=1, r=128, algo=3) == 4       # LBI_ERR_UNSUPPORTED_R
    assert call(dt=1, r=64, algo=3, A=None) == 1
    for r in (16, 32, 64):
        assert binding.lbi_scan_backward_workspace_bytes_ex(4096, 32, r, 1, 3) == 0
        assert binding.lbi_scan_backward_workspace_bytes_ex(2, 512, r, 1, 3) == 0


def test_chain_splitk_argument_errors():
    # eight waves per chain: fp32 storage in the split arithmetic, r = 64
    # only, no workspace; rejected before any pointer is touched
    assert call(dt=1, algo=4) == 3              # bf16 storage: LBI_ERR_DTYPE
    assert call(math=1, algo=4) == 3            # fp32 matrix cores: LBI_ERR_DTYPE
    assert call(r=32, algo=4) == 4              # LBI_ERR_UNSUPPORTED_R
    assert call(r=128, algo=4) == 4
    assert call(algo=4, A=None) == 1
    assert call(algo=7) == 3                    # not an lbi_algo
    assert binding.lbi_scan_backward_workspace_bytes_ex(256, 32, 64, 0, 4) == 0
    assert binding.lbi_scan_backward_workspace_bytes_ex(2, 512, 64, 0, 4) == 0


def test_tree_argument_errors():
    # the log-depth scan: split arithmetic (the default) only, r <= 64
    assert call(algo=5, r=128) == 4             # LBI_ERR_UNSUPPORTED_R
    assert call(algo=5, math=1) == 3            # fp32 matrix cores: LBI_ERR_DTYPE
    assert call(dt=1, algo=5, math=3) == 3      # single rounding: LBI_ERR_DTYPE
    assert call(algo=5, A=None) == 1
    assert call(algo=5, math=2, A=None) == 1
    assert call(dt=1, algo=5, A=None) == 1
    assert call(algo=7) == 3                    # not an lbi_algo
    ws = binding.lbi_scan_backward_workspace_bytes_ex
    assert ws(2, 8, 64, 0, 5) == 0              # one chunk: no workspace
    assert ws(2, 16, 32, 1, 5) == 0
    # K = 100 at r = 64: levels of 13 and 2 aggregates (P, c, carries)
    lev = [13, 2]
    want = sum(-(-(2 * n * x) // 256) * 256 for n in lev for x in (64 * 64 * 4, 64 * 4, 64 * 4))
    assert ws(2, 100, 64, 0, 5) == want
    assert ws(2, 100, 128, 0, 5) == 0           # unsupported r


def call_ex(widths, A=PA, B=2, r=128, dt=1, math=0, algo=6):
    K = len(widths) - 1
    arr = (ctypes.c_int32 * len(widths))(*widths)
    return binding.load().lbi_scan_backward_ex(
        A, PB, PL, POUT, B, K, r, dt, None, 0, None,
        ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)), math, algo)


def test_chain_ring_argument_errors():
    # the LDS-ring chain kernel: bf16 storage, default arithmetic, r in {64,
    # 128}, widths 32/64/128 with r_K = 64, three tiles within the ring;
    # rejected before any pointer is touched (A=None reaches LBI_ERR_NULL
    # only for shapes it takes)
    assert call(algo=6) == 3                    # fp32 storage: LBI_ERR_DTYPE
    assert call(dt=1, math=3, algo=6) == 3      # single rounding: LBI_ERR_DTYPE
    assert call(dt=1, r=64, algo=6, A=None) == 1
    assert call(dt=1, r=32, algo=6) == 2        # storage width 32: LBI_ERR_SHAPE
    assert call(dt=1, r=128, algo=6) == 2       # uniform 128: r_K != 64
    assert call_ex([32, 64, 128, 32, 64], A=None) == 1
    assert call_ex([32, 64, 128, 32, 64], r=64) == 2     # a width past r
    assert call_ex([48, 64, 128, 32, 64]) == 2           # 48 not taken
    assert call_ex([32, 64, 128, 32, 128]) == 2          # r_K = 128
    assert call_ex([128, 128, 64, 64]) == 2              # a 128 x 128 tile
    assert call_ex([64] * 2049, r=64) == 2               # K past the hint
    assert call_ex([64] * 2048, r=64, A=None) == 1
    assert call_ex([32, 64, 128, 32, 64], math=1, A=None) == 1  # fp32 choice acts as default
    assert binding.lbi_scan_backward_workspace_bytes_ex(1024, 64, 128, 1, 6) == 0
    assert binding.lbi_scan_backward_workspace_bytes_ex(4096, 32, 64, 1, 6) == 0


def test_bf16_single_argument_errors():
    # single-rounding arithmetic: bf16 storage only, not on the wavefront-per-
    # chain scan; rejected before any pointer is touched
    assert call(math=3) == 3                    # fp32 storage: LBI_ERR_DTYPE
    assert call(dt=1, r=32, math=3, algo=3) == 3
    assert call(dt=1, r=32, math=3, A=None) == 1
    assert call(dt=1, r=32, math=3, algo=1, A=None) == 1
    f = binding.load().lbi_scan_suffix_products
    assert f(PA, PB, POUT, PL, 2, 3, 64, 0, None, None, 3) == 3
    assert f(None, PB, POUT, PL, 2, 3, 64, 1, None, None, 3) == 1
    # chains longer than LBI_BF16_SINGLE_MAX_K (64): LBI_ERR_SHAPE, in every
    # entry point that takes the arithmetic
    assert call(dt=1, K=65, math=3) == 2
    assert call(dt=1, K=65, math=3, algo=1) == 2
    assert call(dt=1, K=65, math=3, algo=2) == 2
    assert call(dt=1, K=64, math=3, A=None) == 1
    assert call(dt=1, K=65, math=0, A=None) == 1
    assert f(PA, PB, POUT, PL, 2, 65, 64, 1, None, None, 3) == 2
    g = binding.load().lbi_scan_backward_streaming
    assert g(PA, PB, PL, POUT, 2, 65, 64, 1, None, None, 3, 0x60000000, 4, None) == 2
    h = binding.load().lbi_scan_backward_ragged
    w65 = (ctypes.c_int32 * 66)(*([64] * 66))
    assert h(PA, PB, PL, POUT, 2, 65, w65, 1, None, 3) == 2
    assert h(None, PB, PL, POUT, 2, 64, w65, 1, None, 3) == 1


def test_suffix_products_argument_errors():
    lib = binding.load()
    f = lib.lbi_scan_suffix_products
    assert f(PA, PB, POUT, PL, 2, 3, 64, 7, None, None, 0) == 3
    assert f(PA, PB, POUT, PL, 2, 3, 48, 0, None, None, 0) == 4
    assert f(PA, PB, POUT, PL, 2, 0, 64, 0, None, None, 0) == 2
    assert f(None, PB, POUT, PL, 2, 3, 64, 0, None, None, 0) == 1
    assert f(PA, PB, None, PL, 2, 3, 64, 0, None, None, 0) == 1
    assert f(PA, PB, POUT + 4, PL, 2, 3, 64, 0, None, None, 0) == 7
    assert f(PA, PB, PA + 64, PL, 2, 3, 64, 0, None, None, 0) == 8
    assert f(None, None, None, None, 0, 3, 64, 0, None, None, 0) == 0


def test_streaming_argument_errors():
    f = binding.load().lbi_scan_backward_streaming
    PP = 0x60000000
    assert f(PA, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, PP, 0, None) == 2     # chunk < 1
    assert f(PA, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, None, 4, None) == 1   # no progress
    assert f(PA, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, PP + 2, 4, None) == 7
    assert f(PA, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, PA + 64, 4, None) == 8
    assert f(PA, PB, PL, POUT, 2, 3, 64, 3, None, None, 0, PP, 4, None) == 3
    assert f(None, None, None, None, 0, 3, 64, 0, None, None, 0, None, 4, None) == 0


def test_streaming_clock_argument_errors():
    f = binding.load().lbi_scan_backward_streaming
    PP, PC = 0x60000000, 0x68000000
    assert f(PA, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, PP, 4, PC + 4) == 7   # 8-byte
    assert f(PA, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, PP, 4, PP) == 8       # on progress
    assert f(PA, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, PP, 4, POUT + 8) == 8
    assert f(None, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, PP, 4, PC) == 1
    assert f(PA, PB, PL, POUT, 1, 2**32, 16, 0, None, None, 0, PP, 4, PC) == 2   # 32-bit counts


def test_wait_progress_argument_errors():
    f = binding.load().lbi_wait_progress
    PP, PR, PC = 0x60000000, 0x64000000, 0x68000000
    assert f(PP, -1, 1, 10, PR, PC, None) == 2              # B < 0
    assert f(PP, 2, 1, 0, PR, PC, None) == 2                # max_polls < 1
    assert f(None, 2, 1, 10, PR, PC, None) == 1
    assert f(PP + 2, 2, 1, 10, PR, PC, None) == 7
    assert f(PP, 2, 1, 10, PR + 2, PC, None) == 7
    assert f(PP, 2, 1, 10, PR, PC + 4, None) == 7
    assert f(PP, 2, 1, 10, PP + 4, PC, None) == 8           # released on progress
    assert f(PP, 2, 1, 10, PR, PR, None) == 8               # outputs overlap


def test_noalloc_argument_errors():
    f = binding.load().lbi_scan_backward_noalloc
    # the argument checks of lbi_scan_backward_ex
    assert f(PA, PB, PL, POUT, 2, 3, 64, 7, None, None, 0, 0) == 3
    assert f(PA, PB, PL, POUT, 2, 3, 48, 0, None, None, 0, 0) == 4
    assert f(None, PB, PL, POUT, 2, 3, 64, 0, None, None, 0, 0) == 1
    assert f(PA, PB, PL, POUT + 4, 2, 3, 64, 0, None, None, 0, 0) == 7
    assert f(PA, PB, PL, PA + 64, 2, 3, 64, 0, None, None, 0, 0) == 8
    assert f(None, None, None, None, 0, 3, 64, 0, None, None, 0, 0) == 0
    # 2048 chains of 2048 slots at r = 128, two-level: even the segment
    # aggregates (64 segments of 64 KB per chain, 8.6 GB) pass the 64 MiB
    # array; refused before anything is enqueued (far-apart fake addresses)
    QA, QL, QO = 1 << 44, 1 << 45, 1 << 46
    assert f(QA, None, QL, QO, 2048, 2048, 128, 0, None, None, 0, 2) == 9
    assert "LBI_NOALLOC_SCRATCH_BYTES" in binding.lbi_status_string(9)


def test_matrix_norms_argument_errors():
    f = binding.load().lbi_matrix_norms
    PS, PF = 0x70000000, 0x78000000
    assert f(PA, 5, 64, 7, PS, PF, None) == 3                  # dtype
    assert f(PA, 5, 48, 0, PS, PF, None) == 4                  # r
    assert f(PA, -1, 64, 0, PS, PF, None) == 2                 # n < 0
    assert f(PA, 2**40, 128, 0, PS, PF, None) == 2             # size overflow
    assert f(None, 5, 64, 0, PS, PF, None) == 1
    assert f(PA, 5, 64, 0, None, None, None) == 1              # no output
    assert f(PA + 4, 5, 64, 0, PS, PF, None) == 7
    assert f(PA, 5, 64, 0, PS + 4, None, None) == 7
    assert f(PA, 5, 64, 0, PA + 256, None, None) == 8          # output inside M
    assert f(PA, 5, 64, 0, PS, PS + 16, None) == 8             # outputs overlap
    assert f(None, 0, 64, 0, None, None, None) == 0            # n = 0: no-op


def test_ragged_argument_errors():
    f = binding.load().lbi_scan_backward_ragged

    def w(vals):
        arr = (ctypes.c_int32 * len(vals))(*vals)
        return ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)), arr

    good, _g = w([32, 64, 128, 64])
    assert f(PA, PB, PL, POUT, 2, 3, good, 7, None, 0) == 3           # dtype
    assert f(PA, PB, PL, POUT, 2, 3, good, 0, None, 7) == 3           # math
    assert f(PA, PB, PL, POUT, 2, 3, None, 0, None, 0) == 1           # no widths
    for bad in ([32, 60, 128, 64], [32, 64, 144, 64], [0, 64, 128, 64], [8, 16, 16, 16]):
        p, _a = w(bad)
        assert f(PA, PB, PL, POUT, 2, 3, p, 0, None, 0) == 2, bad     # not 16..128 step 16
    long_w, _l = w([64] * 2049)
    assert f(PA, PB, PL, POUT, 2, 2048, long_w, 0, None, 0) == 2      # K above the hint limit
    assert f(PA, PB, PL, POUT, 2, 0, good, 0, None, 0) == 2           # K = 0
    assert f(None, PB, PL, POUT, 2, 3, good, 0, None, 0) == 1
    assert f(PA, PB, PL, POUT + 4, 2, 3, good, 0, None, 0) == 7
    assert f(PA, PB, PL, PA + 64, 2, 3, good, 0, None, 0) == 8        # output inside A
    assert f(None, None, None, None, 0, 3, good, 0, None, 0) == 0     # B = 0: no-op


def test_region_argument_errors():
    f = binding.load().lbi_region_jacobians
    wsb = binding.lbi_region_jacobians_workspace_bytes
    assert wsb(8, 16, 2048, 768, 3072, 64) > 0
    assert wsb(8, 16, 2048, 760, 3072, 64) == 0      # D not a multiple of 64
    assert wsb(8, 16, 2048, 768, 3000, 64) == 0      # X not a multiple of 128
    assert wsb(8, 16, 2048, 768, 3072, 48) == 0      # r
    assert wsb(8, 0, 2048, 768, 3072, 64) == 0       # K = 0
    base = 0x10000000
    good = binding.RegionParams(*[base + 0x01000000 * i for i in range(13)])
    XE, M, A, MN, WS = 0x30000000, 0x31000000, 0x32000000, 0x33000000, 0x40000000
    need = wsb(2, 3, 256, 128, 256, 32)

    def call(params=good, xe=XE, m=M, a=A, mn=MN, B=2, K=3, L=256, D=128, X=256, r=32, ws=WS,
             nws=None):
        return f(ctypes.byref(params) if params is not None else None, xe, m, a, mn, B, K, L, D,
                 X, r, ws, need if nws is None else nws, None)

    assert call(r=48) == 4                           # unsupported r
    assert call(D=100) == 2 and call(X=200) == 2 and call(L=0) == 2 and call(K=0) == 2
    assert call(params=None) == 1
    assert call(xe=None) == 1 and call(m=None) == 1 and call(a=None) == 1
    bad = binding.RegionParams(*[base + 0x01000000 * i for i in range(13)])
    bad.W1 = None
    assert call(params=bad) == 1
    bad.W1 = base + 8                                # misaligned weight
    assert call(params=bad) == 7
    assert call(ws=None) == 5 and call(nws=need - 1) == 5
    assert call(a=XE + 256) == 8                     # A inside x_embed
    assert call(mn=WS + 1024) == 8                   # m_next inside the workspace
    assert call(B=0, xe=None, m=None, a=None) == 0   # B = 0: no-op


def test_region_ssm_argument_errors():
    # the token-mixing block: the token-wise block's checks, a decay pointer,
    # and L r / 128 row tiles within a launch's y
    f = binding.load().lbi_region_jacobians_ssm
    wsb = binding.lbi_region_jacobians_ssm_workspace_bytes
    paper = wsb(8, 16, 2048, 768, 3072, 64)
    # past the token-wise block's workspace: a group of pairs' tangent products
    assert paper > binding.lbi_region_jacobians_workspace_bytes(8, 16, 2048, 768, 3072, 64)
    assert paper < (8 << 30)
    assert wsb(8, 16, 2048, 760, 3072, 64) == 0
    assert wsb(1, 1, 65535 * 128 // 64 + 1, 64, 128, 64) == 0   # L r / 128 past 65535
    assert wsb(1, 1, 65535 * 128 // 64, 64, 128, 64) > 0
    base = 0x10000000
    good = binding.RegionParams(*[base + 0x01000000 * i for i in range(13)])
    DEC, XE, M, A, MN, WS = 0x2f000000, 0x30000000, 0x31000000, 0x32000000, 0x33000000, 0x40000000
    need = wsb(2, 3, 256, 128, 256, 32)
    assert need > 0

    def call(params=good, dec=DEC, xe=XE, m=M, a=A, mn=MN, B=2, K=3, L=256, D=128, X=256, r=32,
             ws=WS, nws=None):
        return f(ctypes.byref(params) if params is not None else None, dec, xe, m, a, mn, B, K,
                 L, D, X, r, ws, need if nws is None else nws, None)

    assert call(r=48) == 4
    assert call(D=100) == 2 and call(L=0) == 2
    assert call(L=65535 * 128 // 32 + 1) == 2
    assert call(params=None) == 1 and call(dec=None) == 1
    assert call(dec=DEC + 4) == 7                    # misaligned decay
    assert call(ws=None) == 5 and call(nws=need - 1) == 5
    assert call(a=DEC) == 8                          # A over the decay vectors
    assert call(B=0, dec=None, xe=None, m=None, a=None) == 0
