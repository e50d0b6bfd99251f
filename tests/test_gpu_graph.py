"""The library's entry points inside a HIP graph, captured through torch's
graph API on the launch stream (needs a GPU).

The calls only enqueue kernels on the caller's stream: no allocation, no
memset, no synchronisation. So a captured sequence of calls, with its
outputs and workspaces allocated beforehand, replays the same work. Each
replay is checked against the eager results bit for bit (the kernels are
deterministic), with the outputs poisoned and other eager library work run
between the replays.  The cases cover every scan algorithm's launch
sequence (one launch, the two-level scan's three, the tree scan's levels),
the LDS-ring kernel, the allocation-free entry point and both Phase 1 blocks.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2605_09204_amd import binding, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _dev(x):
    return (x.A.to(DEV), None if x.b is None else x.b.to(DEV), x.lamK.to(DEV))


CASES = [
    # (name, B, K, r, dtype, algo, widths)
    ("chain f32 split", 64, 40, 64, "f32", binding.LBI_ALGO_CHAIN, None),
    ("two-level f32", 2, 300, 32, "f32", binding.LBI_ALGO_TWO_LEVEL, None),
    ("tree one launch", 4, 16, 16, "f32", binding.LBI_ALGO_TREE, None),
    ("tree levels", 2, 100, 32, "bf16", binding.LBI_ALGO_TREE, None),
    ("wave bf16", 100, 12, 32, "bf16", binding.LBI_ALGO_CHAIN_WAVE, None),
    ("ring bf16 widths", 64, 20, 128, "bf16", binding.LBI_ALGO_CHAIN_RING,
     tuple((32, 64, 128)[k % 3] for k in range(20)) + (64,)),
]


def test_scan_calls_replay_in_a_graph():
    inputs, want, outs, wss, host = [], [], [], [], []
    for name, B, K, r, dt, algo, widths in CASES:
        x = synth.random_chain(B, K, r, dtype=dt, seed=101 + K, widths=widths)
        host.append(x)
        A, b, lk = _dev(x)
        inputs.append((A, b, lk, widths, algo))
        w = binding.lbi_scan_backward_ex(A, b, lk, None if widths is None else list(widths), 0,
                                         algo)
        want.append(w)
        outs.append(torch.empty_like(w))
        need = binding.lbi_scan_backward_workspace_bytes_ex(B, K, r, 0 if dt == "f32" else 1,
                                                             algo)
        wss.append(torch.empty((max(need, 1),), dtype=torch.uint8, device=DEV))
        _say(f"[graph] eager {name}: B={B} K={K} r={r} {dt}")
    # the allocation-free entry point on the two-level case (its scratch array
    # is resolved by an eager call first)
    A0, b0, lk0, _, _ = inputs[1]
    nw = binding.lbi_scan_backward_noalloc(A0, b0, lk0, None, 0, binding.LBI_ALGO_TWO_LEVEL)
    nout = torch.empty_like(nw)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g):
            for (A, b, lk, widths, algo), o, ws in zip(inputs, outs, wss):
                binding.lbi_scan_backward_ex(A, b, lk, None if widths is None else list(widths),
                                             0, algo, lam=o, workspace=ws)
            binding.lbi_scan_backward_noalloc(A0, b0, lk0, None, 0,
                                              binding.LBI_ALGO_TWO_LEVEL, lam=nout)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    other = synth.random_chain(8, 50, 64, dtype="f32", seed=109)
    oA, ob, olk = _dev(other)
    for rep in range(3):
        for o in outs + [nout]:
            o.fill_(float("nan"))
        # eager library work between the replays
        binding.lbi_scan_backward(oA, ob, olk)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for (name, *_), o, w in zip(CASES, outs, want):
            assert torch.equal(o, w), f"replay {rep}: {name}"
        assert torch.equal(nout, nw), f"replay {rep}: allocation-free entry point"
        _say(f"[graph] replay {rep}: {len(CASES) + 1} calls equal to the eager results")
    # and the eager results are the oracle's (the graph replays correct work)
    x = host[0]
    e = oracle.rel_frobenius(want[0].cpu().double().numpy(),
                             oracle.recurrence(x.A, x.b, x.lamK))
    assert e <= 1e-5


@pytest.mark.parametrize("phi", ["ssm", "mlp"])
def test_region_jacobians_replay_in_a_graph(phi):
    x = synth.generate_region(synth.REGION_WORKLOADS["region_small"]).to(DEV)
    wl = x.workload
    if phi == "ssm":
        call = binding.lbi_region_jacobians_ssm
        need = binding.lbi_region_jacobians_ssm_workspace_bytes(wl.B, wl.K, wl.L, wl.D, wl.X,
                                                                wl.r)
    else:
        call = binding.lbi_region_jacobians
        need = binding.lbi_region_jacobians_workspace_bytes(wl.B, wl.K, wl.L, wl.D, wl.X, wl.r)
    A_e, m_e = call(x.params, x.x_embed, x.m)
    ws = torch.empty((need,), dtype=torch.uint8, device=DEV)
    A_g = torch.empty_like(A_e)
    m_g = torch.empty_like(m_e)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g):
            call(x.params, x.x_embed, x.m, A=A_g, m_next=m_g, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for rep in range(3):
        A_g.fill_(float("nan"))
        m_g.fill_(float("nan"))
        ws.fill_(0xFF)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(A_g, A_e) and torch.equal(m_g, m_e), f"replay {rep}"
    _say(f"[graph] Phase 1 ({phi}): 3 replays equal to the eager call")
