"""Builds the HIP library ``_lib/liblbi.so`` for gfx950 with hipcc.

Usage: ``python -m paper_2605_09204_amd.build`` (or ``build_library()``).
Cross-compiles without a GPU.  Each translation unit under ``csrc/`` (one per
arithmetic mode of the chain kernel, the carry/apply kernels, the host API) is
compiled in parallel, then linked.  Packed fp32 instructions are disabled for
all device code.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SOURCES = ["lbi_chain_f32.hip", "lbi_chain_f32x.hip", "lbi_chain_bf16.hip", "lbi_chain_bf16r1.hip",
           "lbi_chain_wave.hip",
           "lbi_chain_ksplit.hip", "lbi_tree.hip", "lbi_chain_ring.hip", "lbi_aux.hip", "lbi_norms.hip", "lbi_region.hip",
           "lbi_api.hip"]
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "liblbi.so")
ARCH = "gfx950"
# hipcc's host pass does not know the device-only feature: drop that note
_NOISE = "'-packed-fp32-ops' is not a recognized feature"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def compile_flags():
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
        "-Wall", "-Wextra", "-Wno-unused-parameter",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # MFMA accumulators in ordinary VGPRs: no copies between register
        # files around the VALU work on the running composite
        "-mllvm", "-amdgpu-mfma-vgpr-form=1",
        f"-I{INCLUDE}", f"-I{CSRC}",
    ]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if _NOISE not in l)
    return res.returncode, err


def build_library(verbose: bool = False) -> str:
    """Compile the library (always recompiles) and return its path."""
    os.makedirs(LIBDIR, exist_ok=True)
    tag = f".tmp{os.getpid()}"
    objs = [os.path.join(LIBDIR, os.path.splitext(s)[0] + ".o" + tag) for s in SOURCES]
    cmds = [[hipcc()] + compile_flags() + ["-c", os.path.join(CSRC, s), "-o", o]
            for s, o in zip(SOURCES, objs)]
    try:
        with concurrent.futures.ThreadPoolExecutor(max_workers=len(cmds)) as ex:
            results = list(ex.map(lambda c: _run(c, verbose), cmds))
        for (rc, err), src in zip(results, SOURCES):
            if rc != 0:
                raise RuntimeError(f"hipcc failed on {src} ({rc}):\n{err}")
            if verbose and err.strip():
                print(err, file=sys.stderr)
        tmp = LIB + tag
        rc, err = _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs,
                       verbose)
        if rc != 0:
            raise RuntimeError(f"hipcc link failed ({rc}):\n{err}")
        os.replace(tmp, LIB)
    finally:
        for o in objs:
            if os.path.exists(o):
                os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
