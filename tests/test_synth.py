"""Properties of the seeded input generators (CPU)."""
import math

import numpy as np
import pytest
import torch

from paper_2605_09204_amd import synth


def _svals(A):
    return torch.linalg.svdvals(A.double())


def test_workload_table():
    w = synth.WORKLOADS
    assert [w[n].B for n in synth.WORKLOAD_ORDER] == [4, 256, 4096, 512, 1024]
    assert [w[n].K for n in synth.WORKLOAD_ORDER] == [8, 32, 32, 512, 64]
    assert [w[n].r for n in synth.WORKLOAD_ORDER] == [16, 64, 64, 64, 128]
    assert [w[n].dtype for n in synth.WORKLOAD_ORDER] == ["f32", "f32", "bf16", "f32", "bf16"]
    assert w["bf16_tokens"].affine is False
    assert w["mixed_widths"].interface_widths()[:4] == (32, 64, 128, 32)
    assert w["mixed_widths"].interface_widths()[-1] == 64  # r_K = r_64


def test_deterministic_and_seed_sensitive():
    wl = synth.WORKLOADS["tiny"]
    x = synth.generate(wl)
    y = synth.generate(wl)
    assert torch.equal(x.A, y.A) and torch.equal(x.b, y.b) and torch.equal(x.lamK, y.lamK)
    z = synth.generate(wl.with_(seed=11))
    assert not torch.equal(x.A, z.A)


def test_shapes_and_dtypes():
    x = synth.generate(synth.WORKLOADS["tiny"])
    assert x.A.shape == (4, 8, 16, 16) and x.A.dtype == torch.float32
    assert x.b.shape == (4, 8, 16) and x.lamK.shape == (4, 16)
    y = synth.generate(synth.WORKLOADS["bf16_tokens"].with_(B=8))
    assert y.A.dtype == torch.bfloat16 and y.b is None and y.lamK.dtype == torch.bfloat16


def test_uniform_spectrum():
    x = synth.generate(synth.WORKLOADS["paper_width"].with_(B=2, K=4))
    s = _svals(x.A.reshape(-1, 64, 64))
    assert float(s.max()) <= 1.1 + 1e-5 and float(s.min()) >= 0.9 - 1e-5
    # not diagonal: the Haar factors mix every coordinate
    off = x.A.reshape(-1, 64, 64).abs().sum() - x.A.reshape(-1, 64, 64).diagonal(dim1=1, dim2=2).abs().sum()
    assert float(off) > 0.5 * float(x.A.abs().sum())


def test_orthogonal_spectrum_gives_orthogonal_A():
    x = synth.random_chain(2, 3, 32, spectrum="orthogonal", seed=5)
    A = x.A.double().reshape(-1, 32, 32)
    eye = torch.eye(32, dtype=torch.float64)
    assert torch.allclose(A @ A.transpose(1, 2), eye.expand_as(A), atol=1e-6)


def test_concentrated_spectrum_matches_paper_statistics():
    """Leading singular value 2.5 x the RMS singular value, ||A||_2 <= 1.05
    (spectral-structure appendix, r = 64: 1.901 / 0.749 ~ 2.5)."""
    x = synth.generate(synth.WORKLOADS["long_chain"].with_(B=2, K=16))
    s = _svals(x.A.reshape(-1, 64, 64))
    rms = torch.sqrt((s * s).mean(-1))
    ratio = s[:, 0] / rms
    assert torch.allclose(ratio, torch.full_like(ratio, 2.5), rtol=1e-4)
    assert float(s[:, 0].max()) <= 1.05 * (1 + 1e-5)
    assert float(s.min()) > 0.05


def test_mixed_width_padding_is_zero():
    wl = synth.WORKLOADS["mixed_widths"].with_(B=3, K=7, widths=synth.cyclic_widths(7))
    x = synth.generate(wl)
    w = wl.interface_widths()
    A = x.A.float()
    for j in range(wl.K):
        rj, rj1 = w[j], w[j + 1]
        assert float(A[:, j, rj:, :].abs().sum()) == 0.0
        assert float(A[:, j, :, rj1:].abs().sum()) == 0.0
        assert float(A[:, j, :rj, :rj1].abs().sum()) > 0.0
        assert float(x.b.float()[:, j, rj:].abs().sum()) == 0.0
        s = _svals(A[:, j, :rj, :rj1])
        assert float(s.max()) <= 1.1 + 1e-2 and float(s.min()) >= 0.9 - 1e-2
    assert float(x.lamK.float()[:, w[-1]:].abs().sum()) == 0.0


def test_affine_and_terminal_scales():
    x = synth.generate(synth.WORKLOADS["paper_width"].with_(B=64))
    bvar = float(x.b.double().var())
    assert abs(bvar - 1 / 64) < 0.1 / 64
    lvar = float(x.lamK.double().var())
    assert abs(lvar - 1.0) < 0.1


def test_bf16_is_rounded_from_f32():
    wl = synth.WORKLOADS["paper_width"].with_(B=2, K=2)
    f = synth.generate(wl)
    h = synth.generate(wl.with_(dtype="bf16"))
    assert torch.equal(f.A.to(torch.bfloat16), h.A)


def test_permutation_chain_is_exact():
    x = synth.permutation_chain(3, 5, 16, dtype="bf16", seed=1)
    A = x.A.float()
    assert torch.equal(A.sum(-1), torch.ones(3, 5, 16))
    assert torch.equal(A.sum(-2), torch.ones(3, 5, 16))
    assert torch.equal(x.b.float(), x.b.float().round())


def test_ragged_pack_round_trip():
    widths = synth.cyclic_widths(7, (16, 48, 32))
    x = synth.random_chain(3, 7, 64, dtype="bf16", seed=61, widths=widths)
    p = synth.pack_ragged(x)
    SA = sum(widths[j] * widths[j + 1] for j in range(7))
    SR = sum(widths[:7])
    assert tuple(p.A.shape) == (3, SA) and tuple(p.b.shape) == (3, SR)
    assert tuple(p.lamK.shape) == (3, widths[7])
    # slot 2's tile sits after slots 0 and 1, row-major at its true shape
    o = widths[0] * widths[1] + widths[1] * widths[2]
    tile = p.A[:, o:o + widths[2] * widths[3]].reshape(3, widths[2], widths[3])
    assert torch.equal(tile, x.A[:, 2, :widths[2], :widths[3]])
    # the padding that packing drops is zero, so unpacking restores b exactly
    assert torch.equal(synth.unpack_ragged(p.b, widths, 64), x.b)
