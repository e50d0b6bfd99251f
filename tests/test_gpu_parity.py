"""Parity of the HIP scan with the CPU oracle, through the C-ABI (needs a GPU).

Tolerances (relative Frobenius over the compared output):
  * float32 storage: 1e-5; bf16 storage with fp32 accumulation: 2e-2.
  * bf16 runs also check 1e-3, well above what the hi/lo feedback of the
    composite leaves (about 1e-5), to catch a lost low part.
  * chains whose products do not contract (orthogonal A over many slots)
    carry fp32 rounding as a random walk: relative error ~ c sqrt(K r) u with
    u = 2^-24; the norm-carry test bounds it by 8 sqrt(K r) u, and over
    K = 512 both arithmetics also meet the flat 1e-5.
Integer/permutation inputs, where every intermediate is exact in fp32, must
match bit for bit.

float32 inputs run under both arithmetic modes of the library: products on the
fp32 matrix cores (LBI_MATH_F32_MFMA) and products from exact three-part bf16
splits on the bf16 matrix cores (LBI_MATH_F32_SPLIT, the default); both must
meet the fp32 tolerance.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import binding, synth

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
BF16_EXPECTED = 1e-3
U32 = 2.0 ** -24


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


MATH = {"split": binding.LBI_MATH_F32_SPLIT, "mfma": binding.LBI_MATH_F32_MFMA}
# (storage dtype, float32 arithmetic) pairs every shape test runs under
MODES = [("f32", "split"), ("f32", "mfma"), ("bf16", None)]
MODE_IDS = ["f32-split", "f32-mfma", "bf16"]


ALGO = {"auto": binding.LBI_ALGO_AUTO, "chain": binding.LBI_ALGO_CHAIN,
        "two_level": binding.LBI_ALGO_TWO_LEVEL, "chain_wave": binding.LBI_ALGO_CHAIN_WAVE,
        "chain_splitk": binding.LBI_ALGO_CHAIN_SPLITK}


def run_gpu(x: synth.Inputs, widths=None, stream=None, math=None, algo=None):
    dev = torch.device("cuda:0")
    A = x.A.to(dev)
    b = None if x.b is None else x.b.to(dev)
    lk = x.lamK.to(dev)
    if math is not None or algo is not None:
        lam = binding.lbi_scan_backward_ex(A, b, lk, widths, MATH[math] if math else 0,
                                           ALGO[algo or "auto"], stream=stream)
    elif widths is None:
        lam = binding.lbi_scan_backward(A, b, lk, stream=stream)
    else:
        lam = binding.lbi_scan_backward_widths(A, b, lk, widths, stream=stream)
    torch.cuda.synchronize()
    return lam


def ref(x: synth.Inputs, idx=None):
    if idx is not None:
        x = x.chains(idx)
    return oracle.recurrence(x.A, x.b, x.lamK)


def assert_close(got, want, tol, what=""):
    got = np.asarray(got, dtype=np.float64)
    err = oracle.rel_frobenius(got, want)
    per = oracle.per_chain_rel_frobenius(got, want)
    _say(f"  {what}: rel-Frobenius {err:.3e}, worst chain {per.max():.3e}")
    assert err <= tol, f"{what}: relative Frobenius error {err:.3e} > {tol:.1e}"
    # element by element: no entry off by more than tol x the chain's max
    scale = np.abs(want).reshape(want.shape[0], -1).max(axis=1)
    diff = np.abs(got - want).reshape(want.shape[0], -1).max(axis=1)
    bad = diff > 4 * tol * np.maximum(scale, 1e-30)
    assert not bad.any(), f"{what}: elementwise error in chains {np.nonzero(bad)[0][:8]}"
    return err


def sample_chains(B, n=48, seed=0):
    if B <= n:
        return torch.arange(B)
    g = torch.Generator().manual_seed(seed)
    mid = torch.randperm(B - 2, generator=g)[: n - 2] + 1
    return torch.cat([torch.tensor([0, B - 1]), mid]).sort().values


# ----------------------------------------------------------------------------
# the five workloads at full size, in the launch configuration of the bench
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_parity_full_size(name):
    wl = synth.WORKLOADS[name]
    _say(f"[parity] workload {name}: B={wl.B} K={wl.K} r={wl.r} {wl.dtype}")
    x = synth.generate(wl, device="cuda:0")
    hint = wl.widths
    lam = run_gpu(x, widths=hint)
    if wl.dtype == "f32":
        # the default arithmetic is the split one; the fp32 matrix cores agree
        native = run_gpu(x, widths=hint, math="mfma")
        assert torch.equal(lam, run_gpu(x, widths=hint, math="split"))
        idx0 = sample_chains(wl.B)
        assert_close(native[idx0.to(native.device)].cpu().numpy(),
                     ref(x.to("cpu"), idx0), TOL["f32"], f"{name} fp32 MFMA")
    idx = sample_chains(wl.B)
    xh = x.to("cpu")
    want = ref(xh, idx)
    got = lam[idx.to(lam.device)].cpu().numpy()
    err = assert_close(got, want, TOL[wl.dtype], name)
    if wl.dtype == "bf16":
        assert err <= BF16_EXPECTED
    if hint is not None:
        # padded output lanes are exactly zero
        for j in range(wl.K):
            if hint[j] < wl.r:
                assert float(lam[:, j, hint[j]:].abs().max()) == 0.0


# ----------------------------------------------------------------------------
# shapes off the workload grid: ragged K, single chains, every tile width
# ----------------------------------------------------------------------------

STRESS = [(B, K, r) for r in (16, 32, 64, 128) for (B, K) in
          ((1, 1), (3, 2), (2, 3), (5, 31), (4, 33), (1, 130))]


@pytest.mark.parametrize("algo", ["chain", "two_level"])
@pytest.mark.parametrize("dtype,arith", MODES, ids=MODE_IDS)
@pytest.mark.parametrize("B,K,r", STRESS)
def test_stress_shapes(B, K, r, dtype, arith, algo):
    _say(f"[stress] B={B} K={K} r={r} {dtype} {arith} {algo}")
    for affine in (True, False):
        x = synth.random_chain(B, K, r, dtype=dtype, seed=K * 7 + r, affine=affine)
        lam = run_gpu(x, math=arith, algo=algo)
        assert_close(lam.cpu().numpy(), ref(x), TOL[dtype] if dtype == "f32" else BF16_EXPECTED,
                     f"B{B} K{K} r{r} {dtype} {arith} {algo} affine={affine}")


@pytest.mark.parametrize("r", [16, 32, 64])
@pytest.mark.parametrize("B,K", [(1, 1), (3, 2), (2, 3), (5, 31), (4, 33), (1, 130), (70, 9)])
def test_chain_wave_shapes(B, K, r):
    """One wavefront per chain (bf16 storage, r <= 64), ragged K and B, with
    and without b, against the oracle; with a widths hint it is unchanged."""
    _say(f"[wave] B={B} K={K} r={r}")
    for affine in (True, False):
        x = synth.random_chain(B, K, r, dtype="bf16", seed=K * 11 + r, affine=affine)
        lam = run_gpu(x, algo="chain_wave")
        assert_close(lam.cpu().numpy(), ref(x), BF16_EXPECTED,
                     f"wave B{B} K{K} r{r} affine={affine}")
        hinted = run_gpu(x, widths=[r] * (K + 1), algo="chain_wave")
        assert torch.equal(lam, hinted)


@pytest.mark.parametrize("r", [16, 32, 64])
def test_chain_wave_permutation_exact(r):
    for K in (1, 7, 40):
        x = synth.permutation_chain(3, K, r, dtype="bf16", seed=K + r)
        got = run_gpu(x, algo="chain_wave").cpu().numpy().astype(np.float64)
        assert np.array_equal(got, ref(x)), f"K={K}"


def test_chain_wave_token_batches_and_auto():
    """Token batches (K = 32, b = NULL, bf16): at r = 32 AUTO runs the
    wavefront-per-chain scan, which equals the explicit call bit for bit and
    meets the oracle on sampled chains; at r = 64 (the bf16_tokens workload)
    AUTO keeps the workgroup kernel, and the wave kernel agrees with it to the
    bf16 tolerance."""
    x = synth.random_chain(3000, 32, 32, dtype="bf16", seed=21, affine=False, device="cuda:0")
    auto = run_gpu(x)
    wave = run_gpu(x, algo="chain_wave")
    assert torch.equal(auto, wave)
    idx = sample_chains(3000, seed=5)
    assert_close(wave[idx.to(wave.device)].cpu().numpy(), ref(x.to("cpu"), idx), BF16_EXPECTED,
                 "r32 token batch wave")
    wl = synth.WORKLOADS["bf16_tokens"]
    y = synth.generate(wl, device="cuda:0")
    auto = run_gpu(y)
    assert torch.equal(auto, run_gpu(y, algo="chain"))
    wave = run_gpu(y, algo="chain_wave")
    idx = sample_chains(wl.B, seed=6)
    assert_close(wave[idx.to(wave.device)].cpu().numpy(), ref(y.to("cpu"), idx), BF16_EXPECTED,
                 "bf16_tokens wave")
    assert oracle.rel_frobenius(wave.cpu().double().numpy(), auto.cpu().double().numpy()) < 1e-4


def test_chain_wave_offsets_past_4gib():
    """2048 bf16 chains of 256 slots at r = 64: A spans 4.3 GB, so the last
    chains sit past 2^32 bytes (64-bit chain bases, 32-bit per-tile offsets).
    Tiles are I + N(0, 0.02^2) noise drawn on the GPU; sampled chains, the
    last among them, are held to the oracle."""
    B, K, r = 2048, 256, 64
    _say(f"[wave] B={B} K={K} r={r} (A = {B * K * r * r * 2 / 1e9:.1f} GB)")
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(97)
    A = torch.empty((B, K, r, r), dtype=torch.bfloat16, device=dev)
    eye = torch.eye(r, device=dev)
    for c in range(0, B, 256):
        A[c:c + 256] = (eye + 0.02 * torch.randn((256, K, r, r), generator=g, device=dev)).bfloat16()
    b = (0.1 * torch.randn((B, K, r), generator=g, device=dev)).bfloat16()
    lamK = torch.randn((B, r), generator=g, device=dev).bfloat16()
    wl = synth.Workload("wave_4gib", B, K, r, "bf16", 0, "uniform", True)
    x = synth.Inputs(A, b, lamK, (r,) * (K + 1), wl)
    lam = run_gpu(x, algo="chain_wave")
    idx = torch.tensor([0, 1, 1023, 1500, B - 2, B - 1])
    sub = x.chains(idx.to(dev)).to("cpu")
    assert_close(lam[idx.to(dev)].cpu().numpy(), oracle.recurrence(sub.A, sub.b, sub.lamK),
                 BF16_EXPECTED, "wave past 4 GiB")
    del A, b, lam


@pytest.mark.parametrize("B,K", [(1, 1), (3, 2), (2, 3), (5, 31), (4, 33), (1, 130), (70, 9),
                                 (300, 5)])
def test_chain_splitk_shapes(B, K):
    """The small-batch chain kernel (fp32 storage, split arithmetic, r = 64),
    ragged K and B (B = 300: more chains than CUs), with and without b,
    against the oracle.  A widths hint of full widths changes nothing."""
    _say(f"[splitk] B={B} K={K}")
    for affine in (True, False):
        x = synth.random_chain(B, K, 64, dtype="f32", seed=K * 13 + B, affine=affine)
        lam = run_gpu(x, algo="chain_splitk")
        assert_close(lam.cpu().numpy(), ref(x), TOL["f32"], f"splitk B{B} K{K} affine={affine}")
        hinted = run_gpu(x, widths=[64] * (K + 1), algo="chain_splitk")
        assert torch.equal(lam, hinted)


@pytest.mark.parametrize("B", [3, 300])
def test_chain_splitk_permutation_exact(B):
    for K in (1, 2, 7, 40):
        x = synth.permutation_chain(B, K, 64, dtype="f32", seed=K + B)
        got = run_gpu(x, algo="chain_splitk").cpu().numpy().astype(np.float64)
        assert np.array_equal(got, ref(x)), f"B={B} K={K}"


@pytest.mark.parametrize("name", ["paper_width", "long_chain"])
def test_chain_splitk_full_size(name):
    """The fp32 r = 64 workloads at full size through the small-batch kernel,
    sampled chains against the oracle, and the whole output against the
    workgroup chain kernel."""
    wl = synth.WORKLOADS[name]
    _say(f"[splitk] {name} B={wl.B} K={wl.K}")
    x = synth.generate(wl, device="cuda:0")
    lam = run_gpu(x, algo="chain_splitk")
    idx = sample_chains(wl.B, n=24, seed=17)
    assert_close(lam[idx.to(lam.device)].cpu().numpy(), ref(x.to("cpu"), idx), TOL["f32"],
                 f"{name} splitk")
    base = run_gpu(x, algo="chain")
    assert oracle.rel_frobenius(lam.cpu().double().numpy(), base.cpu().double().numpy()) < 2e-6


@pytest.mark.parametrize("B", [4])
@pytest.mark.parametrize("spectrum,affine", [("uniform", False), ("uniform", True),
                                             ("orthogonal", False)])
def test_chain_splitk_long_undamped_chain(spectrum, affine, B):
    K, r = 512, 64
    _say(f"[splitk] {spectrum} affine={affine} K=512 B={B}")
    x = synth.random_chain(B, K, r, dtype="f32", seed=7, spectrum=spectrum, affine=affine)
    lam = run_gpu(x, algo="chain_splitk").cpu().numpy().astype(np.float64)
    assert_close(lam, ref(x), TOL["f32"], f"splitk {spectrum} K512 B{B}")


@pytest.mark.parametrize("algo", ["chain", "two_level"])
@pytest.mark.parametrize("arith", ["split", "mfma"])
def test_long_contracting_chain_r16(arith, algo):
    x = synth.random_chain(2, 2049, 16, dtype="f32", seed=3, spectrum="concentrated")
    _say(f"[stress] K=2049 r=16 concentrated {arith} {algo}")
    assert_close(run_gpu(x, math=arith, algo=algo).cpu().numpy(), ref(x), TOL["f32"], "K2049")


@pytest.mark.parametrize("algo", ["chain", "two_level"])
@pytest.mark.parametrize("r", [16, 32, 64, 128])
@pytest.mark.parametrize("dtype,arith", MODES, ids=MODE_IDS)
def test_permutation_chains_bit_exact(r, dtype, arith, algo):
    _say(f"[exact] permutation r={r} {dtype} {arith} {algo}")
    for K in (1, 7, 40):
        x = synth.permutation_chain(3, K, r, dtype=dtype, seed=K + r)
        got = run_gpu(x, math=arith, algo=algo).cpu().numpy().astype(np.float64)
        assert np.array_equal(got, ref(x)), f"K={K}"


@pytest.mark.parametrize("arith", ["split", "mfma"])
def test_orthogonal_long_chain_carries_norm(arith):
    """s == 1, b = 0, K = 512: nothing decays, so every slot tests the carry."""
    K, r = 512, 64
    _say(f"[stress] orthogonal K=512 r=64 {arith}")
    x = synth.random_chain(4, K, r, dtype="f32", seed=9, spectrum="orthogonal", affine=False)
    lam = run_gpu(x, math=arith, algo="chain").cpu().numpy().astype(np.float64)
    tol = 8 * math.sqrt(K * r) * U32
    assert_close(lam, ref(x), tol, "orthogonal K512")
    ratio = np.linalg.norm(lam, axis=-1) / np.linalg.norm(x.lamK.double().numpy(), axis=-1)[:, None]
    assert np.allclose(ratio, 1.0, atol=tol * 4)


@pytest.mark.parametrize("algo", ["chain", "two_level"])
@pytest.mark.parametrize("arith", ["split", "mfma"])
@pytest.mark.parametrize("spectrum,affine", [("uniform", False), ("uniform", True),
                                             ("orthogonal", False)])
def test_long_undamped_chain_meets_fp32_tolerance(arith, algo, spectrum, affine):
    """K = 512 chains whose products neither decay nor grow (s ~ U[0.9, 1.1],
    or orthogonal): every slot's rounding reaches lambda_0, so this is where a
    biased product shows.  Both float32 arithmetics meet the flat fp32
    tolerance here (a split into truncated parts does not: its dropped
    products share the sign of the value, and their bias builds up to about
    1.4e-5 over 512 slots of the uniform chain)."""
    K, r = 512, 64
    _say(f"[stress] {spectrum} affine={affine} K=512 r=64 {arith} {algo}")
    x = synth.random_chain(4, K, r, dtype="f32", seed=7, spectrum=spectrum, affine=affine)
    lam = run_gpu(x, math=arith, algo=algo).cpu().numpy().astype(np.float64)
    assert_close(lam, ref(x), TOL["f32"], f"{spectrum} K512 {arith} {algo}")


@pytest.mark.parametrize("algo", ["chain", "two_level", "chain_splitk"])
@pytest.mark.parametrize("arith", ["split", "mfma"])
def test_products_with_identity_are_exact(arith, algo):
    """A product with an identity factor must return the other factor bit for
    bit, whatever its mantissas and exponents: chains [X, I] and [I, Y] with
    full-precision random X, Y (exponents over 2^-40 .. 2^40) and one-hot
    lambda_K.  Then lambda_0 is a column of X or Y exactly, which pins the
    three-part split of both operands (A staged from memory, P carried in
    registers) to h + m + l == x."""
    if algo == "chain_splitk" and arith == "mfma":
        pytest.skip("the small-batch kernel has the split arithmetic only")
    r = 64
    gen = torch.Generator().manual_seed(83)
    n = 6
    A = torch.zeros((2 * n, 2, r, r), dtype=torch.float32)
    eye = torch.eye(r)
    for c in range(2 * n):
        mant = torch.randn((r, r), generator=gen, dtype=torch.float64)
        expo = torch.randint(-40, 41, (r, r), generator=gen).double()
        M = (mant * torch.exp2(expo)).float()
        if c < n:
            A[c, 0], A[c, 1] = M, eye           # [X, I]: X split while staged
        else:
            A[c, 0], A[c, 1] = eye, M           # [I, Y]: Y split as the carried P
    cols = torch.randint(0, r, (2 * n,), generator=gen)
    lamK = torch.zeros((2 * n, r))
    lamK[torch.arange(2 * n), cols] = 1.0
    wl = synth.Workload("identity_factor", 2 * n, 2, r, "f32", 0, "orthogonal", False)
    x = synth.Inputs(A, None, lamK, (r,) * 3, wl)
    lam = run_gpu(x, math=arith, algo=algo).cpu()
    for c in range(2 * n):
        M = A[c, 0] if c < n else A[c, 1]
        assert torch.equal(lam[c, 0], M[:, cols[c]]), f"chain {c}: lambda_0 is not the exact column"
        assert torch.equal(lam[c, 1], A[c, 1][:, cols[c]]), f"chain {c}: lambda_1"


# ----------------------------------------------------------------------------
# API behaviour
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("algo", ["chain", "two_level"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_null_b_equals_zero_b(dtype, algo):
    x = synth.random_chain(8, 20, 64, dtype=dtype, seed=1, affine=False)
    none = run_gpu(x, algo=algo)
    zero = synth.Inputs(x.A, torch.zeros(x.A.shape[:3], dtype=x.A.dtype), x.lamK, x.widths,
                        x.workload)
    assert torch.equal(none, run_gpu(zero, algo=algo))


@pytest.mark.parametrize("arith", ["split", "mfma"])
def test_bitwise_deterministic(arith):
    x = synth.generate(synth.WORKLOADS["paper_width"], device="cuda:0")
    a = run_gpu(x, math=arith)
    b = run_gpu(x, math=arith)
    assert torch.equal(a, b)
    y = synth.random_chain(3, 300, 64, dtype="f32", seed=7)
    assert torch.equal(run_gpu(y, math=arith, algo="two_level"),
                       run_gpu(y, math=arith, algo="two_level"))


def test_split_arithmetic_matches_fp32_matrix_cores():
    """Both float32 modes sit within a few fp32 roundings of each other."""
    x = synth.random_chain(16, 64, 64, dtype="f32", seed=11)
    a = run_gpu(x, math="split").cpu().numpy().astype(np.float64)
    b = run_gpu(x, math="mfma").cpu().numpy().astype(np.float64)
    want = ref(x)
    ea, eb = oracle.rel_frobenius(a, want), oracle.rel_frobenius(b, want)
    _say(f"  split {ea:.3e}, fp32 MFMA {eb:.3e}")
    assert ea <= 4 * eb + 1e-7 and eb <= 4 * ea + 1e-7


@pytest.mark.parametrize("algo", ["chain", "two_level"])
@pytest.mark.parametrize("r", [64, 128])
@pytest.mark.parametrize("dtype,arith", MODES, ids=MODE_IDS)
def test_widths_hint_matches_unhinted(dtype, arith, r, algo):
    widths = synth.cyclic_widths(23, (16, 32, 64) if r == 64 else (32, 64, 128))
    x = synth.random_chain(6, 23, r, dtype=dtype, seed=2, widths=widths)
    plain = run_gpu(x, math=arith, algo=algo)
    hinted = run_gpu(x, widths=widths, math=arith, algo=algo)
    assert torch.equal(plain, hinted)
    for j in range(23):
        if widths[j] < r:
            assert float(hinted[:, j, widths[j]:].abs().max()) == 0.0
    assert_close(hinted.cpu().numpy(), ref(x), BF16_EXPECTED if dtype == "bf16" else TOL["f32"],
                 f"hinted {dtype}")


def test_runs_on_the_given_stream():
    x = synth.generate(synth.WORKLOADS["tiny"], device="cuda:0")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        lam = binding.lbi_scan_backward(x.A, x.b, x.lamK)
    s.synchronize()
    assert_close(lam.cpu().numpy(), ref(x.to("cpu")), TOL["f32"], "side stream")


def test_empty_batch_and_argument_errors_on_gpu():
    A = torch.zeros((0, 4, 64, 64), device="cuda:0")
    lk = torch.zeros((0, 64), device="cuda:0")
    assert binding.lbi_scan_backward(A, None, lk).shape == (0, 4, 64)
    A = torch.zeros((2, 4, 48, 48), device="cuda:0")
    with pytest.raises(binding.LbiError) as e:
        binding.lbi_scan_backward(A, None, torch.zeros((2, 48), device="cuda:0"))
    assert e.value.status == 4


def test_nan_propagates():
    x = synth.random_chain(2, 6, 64, dtype="f32", seed=4)
    lk = x.lamK.clone()
    lk[1, 5] = float("nan")
    y = synth.Inputs(x.A, x.b, lk, x.widths, x.workload)
    lam = run_gpu(y).cpu()
    assert torch.isnan(lam[1]).all()
    assert torch.isfinite(lam[0]).all()


# ----------------------------------------------------------------------------
# the two-level scan (segments folded in parallel, carries, parallel apply)
# ----------------------------------------------------------------------------

TWO_LEVEL = [(1, 2, 64), (3, 17, 64), (2, 130, 16), (1, 513, 64), (2, 65, 32), (1, 40, 128)]


@pytest.mark.parametrize("dtype,arith", MODES, ids=MODE_IDS)
@pytest.mark.parametrize("B,K,r", TWO_LEVEL)
def test_two_level_parity(B, K, r, dtype, arith):
    _say(f"[two-level] B={B} K={K} r={r} {dtype} {arith}")
    for affine in (True, False):
        x = synth.random_chain(B, K, r, dtype=dtype, seed=K * 3 + r, affine=affine,
                               spectrum="concentrated" if K > 200 else "uniform")
        lam = run_gpu(x, math=arith, algo="two_level")
        assert_close(lam.cpu().numpy(), ref(x), TOL[dtype] if dtype == "f32" else BF16_EXPECTED,
                     f"two-level B{B} K{K} r{r} {dtype} {arith} affine={affine}")


@pytest.mark.parametrize("affine", [True, False])
@pytest.mark.parametrize("B", [81, 82])
def test_two_level_both_forms(B, affine):
    """At r = 64 and K = 200, B = 81 keeps every segment composite (253.1 MiB
    of fp32) and applies them in one pass; B = 82 (256.3 MiB) keeps only the
    segment aggregates and scans each segment again from its carry.  Both against the
    oracle on every chain, with and without b, and the widths hint changing
    nothing."""
    K, r = 200, 64
    _say(f"[two-level] B={B} K={K} affine={affine}")
    x = synth.random_chain(B, K, r, dtype="f32", seed=61 + B, affine=affine, device="cuda:0")
    lam = run_gpu(x, algo="two_level")
    assert_close(lam.cpu().numpy(), ref(x.to("cpu")), TOL["f32"], f"two-level B{B}")
    assert torch.equal(lam, run_gpu(x, widths=[r] * (K + 1), algo="two_level"))


@pytest.mark.parametrize("arith", ["split", "mfma"])
def test_two_level_orthogonal_long_chain(arith):
    """Nothing decays: every segment's carry and every apply must be right."""
    K, r = 512, 64
    _say(f"[two-level] orthogonal K=512 r=64 {arith}")
    x = synth.random_chain(2, K, r, dtype="f32", seed=19, spectrum="orthogonal", affine=False)
    lam = run_gpu(x, math=arith, algo="two_level").cpu().numpy().astype(np.float64)
    assert_close(lam, ref(x), 8 * math.sqrt(K * r) * U32, "two-level orthogonal K512")


def test_auto_picks_splitk_for_small_fp32_batches():
    """fp32 chains at r = 64 in the split arithmetic, at most one per CU and
    not taken by the two-level scan, run on the sixteen-wave kernel: AUTO
    equals the explicit call bit for bit (K < 16, and paper_width's B = 256,
    K = 32); the fp32 matrix cores and B = 300 keep the workgroup kernel."""
    x = synth.random_chain(5, 9, 64, dtype="f32", seed=29)
    assert torch.equal(run_gpu(x), run_gpu(x, algo="chain_splitk"))
    assert torch.equal(run_gpu(x, math="mfma", algo="auto"), run_gpu(x, math="mfma", algo="chain"))
    y = synth.generate(synth.WORKLOADS["paper_width"], device="cuda:0")
    assert torch.equal(run_gpu(y), run_gpu(y, algo="chain_splitk"))
    z = synth.random_chain(300, 9, 64, dtype="f32", seed=30)
    assert torch.equal(run_gpu(z), run_gpu(z, algo="chain"))


def test_auto_picks_two_level_for_few_long_chains():
    x = synth.random_chain(2, 96, 64, dtype="f32", seed=23)
    auto = run_gpu(x, algo="auto")
    assert torch.equal(auto, run_gpu(x, algo="two_level"))
    assert not torch.equal(auto, run_gpu(x, algo="chain"))  # a different bracketing
    many = synth.random_chain(300, 20, 64, dtype="f32", seed=24)
    assert torch.equal(run_gpu(many, algo="auto"), run_gpu(many, algo="chain"))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_two_level_widths_hint(dtype):
    widths = synth.cyclic_widths(70)
    x = synth.random_chain(2, 70, 128, dtype=dtype, seed=29, widths=widths)
    plain = run_gpu(x, algo="two_level")
    hinted = run_gpu(x, widths=widths, algo="two_level")
    assert torch.equal(plain, hinted)
    for j in range(70):
        if widths[j] < 128:
            assert float(hinted[:, j, widths[j]:].abs().max()) == 0.0
    assert_close(hinted.cpu().numpy(), ref(x), BF16_EXPECTED if dtype == "bf16" else TOL["f32"],
                 f"two-level hinted {dtype}")


@pytest.mark.parametrize("name", ["tiny", "paper_width", "mixed_widths"])
def test_two_level_workloads_full_size(name):
    wl = synth.WORKLOADS[name]
    _say(f"[two-level] workload {name}")
    x = synth.generate(wl, device="cuda:0")
    lam = run_gpu(x, widths=wl.widths, algo="two_level")
    idx = sample_chains(wl.B)
    assert_close(lam[idx.to(lam.device)].cpu().numpy(), ref(x.to("cpu"), idx), TOL[wl.dtype],
                 f"{name} two-level")


# ----------------------------------------------------------------------------
# suffix-composite export
# ----------------------------------------------------------------------------

def _rel_per_slot(got, want):
    got = np.asarray(got, dtype=np.float64)
    d = np.linalg.norm((got - want).reshape(want.shape[0], want.shape[1], -1), axis=-1)
    n = np.linalg.norm(want.reshape(want.shape[0], want.shape[1], -1), axis=-1)
    return d / np.maximum(n, 1e-300)


@pytest.mark.parametrize("dtype,arith", MODES, ids=MODE_IDS)
@pytest.mark.parametrize("r", [16, 64, 128])
def test_suffix_products_match_oracle(r, dtype, arith):
    _say(f"[export] r={r} {dtype} {arith}")
    x = synth.random_chain(3, 21, r, dtype=dtype, seed=31 + r)
    A = x.A.to("cuda:0")
    b = x.b.to("cuda:0")
    P, c = binding.lbi_scan_suffix_products(A, b, math=MATH[arith] if arith else 0)
    torch.cuda.synchronize()
    Pr, cr = oracle.suffix_composites(x.A, x.b)
    tol = TOL["f32"] if dtype == "f32" else BF16_EXPECTED
    assert _rel_per_slot(P.cpu().numpy(), Pr).max() <= tol
    assert _rel_per_slot(c.cpu().numpy()[..., None], cr[..., None]).max() <= tol
    # the composites applied to lambda_K give the adjoints (Phase 2)
    lam = np.einsum("bkij,bj->bki", P.cpu().double().numpy(), x.lamK.double().numpy()) \
        + c.cpu().double().numpy()
    assert_close(lam, ref(x), tol, f"export applied r={r} {dtype}")
    # without b: c is written as zeros, P unchanged
    P0, c0 = binding.lbi_scan_suffix_products(A, None, math=MATH[arith] if arith else 0)
    torch.cuda.synchronize()
    assert torch.equal(P0, P) and float(c0.abs().max()) == 0.0


def test_suffix_products_exact_on_permutations():
    x = synth.permutation_chain(2, 9, 64, dtype="f32", seed=37)
    P, c = binding.lbi_scan_suffix_products(x.A.to("cuda:0"), x.b.to("cuda:0"))
    torch.cuda.synchronize()
    Pr, cr = oracle.suffix_composites(x.A, x.b)
    assert np.array_equal(P.cpu().numpy().astype(np.float64), Pr)
    assert np.array_equal(c.cpu().numpy().astype(np.float64), cr)


# ----------------------------------------------------------------------------
# streaming: adjoints published while the scan runs
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,arith", MODES, ids=MODE_IDS)
@pytest.mark.parametrize("B,K,r,chunk", [(3, 40, 64, 8), (2, 33, 16, 1), (1, 130, 128, 16),
                                         (4, 7, 32, 64), (5, 96, 64, 5)])
def test_streaming_matches_oracle_and_chain_scan(B, K, r, chunk, dtype, arith):
    """The streaming scan's adjoints against the oracle (element by element, at
    the storage dtype's tolerance), equal to the chain scan's bit for bit, its
    counters at K, and one publication clock per chunk, in order."""
    _say(f"[streaming] B={B} K={K} r={r} chunk={chunk} {dtype} {arith}")
    x = synth.random_chain(B, K, r, dtype=dtype, seed=43 + K)
    dev = torch.device("cuda:0")
    progress = torch.zeros(B, dtype=torch.int32, device=dev)
    npub = -(-K // chunk)
    clock = torch.zeros((B, npub), dtype=torch.int64, device=dev)
    lam = binding.lbi_scan_backward_streaming(x.A.to(dev), x.b.to(dev), x.lamK.to(dev), progress,
                                              chunk, math=MATH[arith] if arith else 0,
                                              publish_clock=clock)
    torch.cuda.synchronize()
    err = assert_close(lam.cpu().numpy(), ref(x), TOL[dtype], f"streaming {dtype} {arith}")
    if dtype == "bf16":
        assert err <= BF16_EXPECTED
    assert torch.equal(lam, run_gpu(x, math=arith, algo="chain"))
    assert progress.tolist() == [K] * B
    c = clock.cpu()
    assert bool((c > 0).all()), "a publication recorded no clock"
    assert bool((c[:, 1:] >= c[:, :-1]).all()), "publications out of order"


def test_streaming_releases_a_consumer_before_the_scan_ends():
    """Phase 3's consumer pattern: a wait (lbi_wait_progress) is queued on a
    second stream ahead of a copy of the 1024 adjoints of the latest regions;
    the scan of 2 chains of 4096 slots runs on the first stream.  The library
    controls both sides (the publications with system-scope atomics, the
    wait's polls with system-scope acquire loads), so the test asserts:
      * the wait was satisfied, and the copy holds the final adjoints;
      * the adjoints meet the oracle (orthogonal chains: the fp32 rounding
        walk bound 8 sqrt(K r) 2^-24) and equal the chain scan's;
      * every chain published one clock per chunk, in order, spread evenly
        over the run (the middle one between 30% and 70% of the span), not
        bunched at the end;
      * the wait ended after the publication that reached 1024 and before the
        scan's last publication: the consumer started while the scan ran."""
    B, K, r, n, chunk = 2, 4096, 64, 1024, 64
    dev = torch.device("cuda:0")
    x = synth.random_chain(B, K, r, dtype="f32", seed=47, spectrum="orthogonal", device=dev)
    progress = torch.zeros(B, dtype=torch.int32, device=dev)
    npub = K // chunk
    clock = torch.zeros((B, npub), dtype=torch.int64, device=dev)
    released = torch.zeros(1, dtype=torch.int32, device=dev)
    rel_clock = torch.zeros(1, dtype=torch.int64, device=dev)
    lam = torch.empty((B, K, r), dtype=torch.float32, device=dev)
    snap = torch.empty((B, n, r), dtype=torch.float32, device=dev)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    # the consumer first: it waits (bounded) for the scan's publications
    binding.lbi_wait_progress(progress, n, 1 << 20, released=released,
                              release_clock=rel_clock, stream=s2)
    with torch.cuda.stream(s2):
        snap.copy_(lam[:, K - n:])
    binding.lbi_scan_backward_streaming(x.A, x.b, x.lamK, progress, chunk, lam=lam, stream=s1,
                                        publish_clock=clock)
    torch.cuda.synchronize()
    assert int(released.item()) == 1, "the wait gave up before the counters reached the target"
    assert progress.tolist() == [K] * B
    assert torch.equal(snap, lam[:, K - n:])
    xh = x.to("cpu")
    err = oracle.rel_frobenius(lam.cpu().numpy().astype(np.float64), ref(xh))
    _say(f"  adjoints vs oracle: {err:.3e}")
    assert err <= 8 * math.sqrt(K * r) * U32
    assert torch.equal(lam, run_gpu(xh, math="split", algo="chain"))
    c = clock.cpu().numpy().astype(np.int64)
    assert (c > 0).all() and (np.diff(c, axis=1) >= 0).all()
    span = c[:, -1] - c[:, 0]
    mid = (c[:, npub // 2] - c[:, 0]) / np.maximum(span, 1)
    t_rel = int(rel_clock.item())
    reach = c[:, n // chunk - 1].max()   # both chains had published n adjoints
    _say(f"  publications span {span.tolist()} ticks, middle at {mid.round(3).tolist()} of it; "
         f"wait released {t_rel - reach} ticks after the target publication, "
         f"{c[:, -1].max() - t_rel} ticks before the last one")
    assert (span > 0).all() and ((mid > 0.3) & (mid < 0.7)).all(), "publications not spread"
    assert reach <= t_rel < c[:, -1].max(), "the consumer was not released while the scan ran"


def test_streaming_command_processor_wait_report():
    """The same pattern with the command processor's wait
    (hipStreamWaitValue32, >=) in place of lbi_wait_progress.  How soon the
    command processor sees the counter is outside the library, so this only
    reports the lead of the copy over the scan's end; the copy must hold the
    final values."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipStreamWaitValue32.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32,
                                         ctypes.c_uint, ctypes.c_uint32]
    hip.hipStreamWaitValue32.restype = ctypes.c_int
    B, K, r, n, chunk = 2, 4096, 64, 1024, 64
    dev = torch.device("cuda:0")
    x = synth.random_chain(B, K, r, dtype="f32", seed=47, spectrum="orthogonal", device=dev)
    progress = torch.zeros(B, dtype=torch.int32, device=dev)
    lam = torch.empty((B, K, r), dtype=torch.float32, device=dev)
    snap = torch.empty((B, n, r), dtype=torch.float32, device=dev)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    done_scan = torch.cuda.Event(enable_timing=True)
    done_copy = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    binding.lbi_scan_backward_streaming(x.A, x.b, x.lamK, progress, chunk, lam=lam, stream=s1)
    done_scan.record(s1)
    for beta in range(B):
        rc = hip.hipStreamWaitValue32(s2.cuda_stream, progress.data_ptr() + 4 * beta, n, 0,
                                      0xFFFFFFFF)
        if rc != 0:
            torch.cuda.synchronize()
            pytest.skip(f"hipStreamWaitValue32 unavailable (error {rc})")
    with torch.cuda.stream(s2):
        snap.copy_(lam[:, K - n:])
        done_copy.record(s2)
    torch.cuda.synchronize()
    assert progress.tolist() == [K] * B
    assert torch.equal(snap, lam[:, K - n:])
    lead_ms = done_copy.elapsed_time(done_scan)
    _say(f"  command-processor wait: the copy of the first {n} adjoints finished "
         f"{lead_ms:.3f} ms before the scan's end (negative: after)")
