"""The C-ABI driven from plain C: tests/c/scan_from_c.c allocates device
memory with the HIP runtime API, queries and allocates the workspace, and
calls lbi_scan_backward (the library's choice of scan) and
lbi_scan_backward_ex (the chain scan), with no Python or torch in between."""

import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2605_09204_amd import binding, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c", "scan_from_c.c")


def build(out_dir) -> str:
    exe = os.path.join(str(out_dir), "scan_from_c")
    libdir = os.path.dirname(binding.library_path())
    cmd = ["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           f"-I{os.path.join(ROOT, 'include')}", SRC, "-o", exe, "-L/opt/rocm/lib", "-lamdhip64",
           f"-L{libdir}", "-llbi", f"-Wl,-rpath,{libdir}", "-Wl,-rpath,/opt/rocm/lib"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return exe


def test_c_program_builds(tmp_path):
    assert os.path.exists(build(tmp_path))


@pytest.mark.gpu
def test_scan_from_c_matches_oracle(tmp_path):
    """B = 2, K = 64, r = 64, fp32 with b: the library's choice is the
    two-level scan (so the workspace path runs), the explicit call the chain
    scan; both within the fp32 tolerance of the oracle."""
    B, K, r = 2, 64, 64
    exe = build(tmp_path)
    x = synth.random_chain(B, K, r, dtype="f32", seed=71)
    inp, out = tmp_path / "in.bin", tmp_path / "out.bin"
    np.concatenate([x.A.numpy().ravel(), x.b.numpy().ravel(), x.lamK.numpy().ravel()]).astype(
        np.float32).tofile(inp)
    res = subprocess.run([exe, str(inp), str(out), str(B), str(K), str(r)], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    assert binding.lbi_scan_backward_workspace_bytes(B, K, r, 0) > 0
    lam = np.fromfile(out, dtype=np.float32).reshape(2, B, K, r).astype(np.float64)
    want = oracle.recurrence(x.A, x.b, x.lamK)
    for got, what in ((lam[0], "library choice"), (lam[1], "chain scan")):
        err = oracle.rel_frobenius(got, want)
        assert err <= 1e-5, f"{what}: relative Frobenius error {err:.3e}"
