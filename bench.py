#!/usr/bin/env python3
"""Throughput of the interface-adjoint scan on one MI355X.

One step = one ``lbi_scan_backward`` call over the whole batch of a synthetic
workload (every slot of every chain composed and applied).  Prints one JSON
line.  Default workload: ``long_chain`` (B=512 chains, K=512 regions, r=64,
fp32), the largest batched r=64 workload.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                  [--math split|mfma|bf16single] [--no-cpu-baseline] [--copy-calibration MiB]

Accounting (flop = 2 per multiply-add; the paper counts r^3 per r x r
product, i.e. one per multiply-add, in its scan-negligibility estimate):
  combine of slot j into the suffix composite S_{j+1} = (P_{j+1}, c_{j+1}):
      2 r_j r_{j+1} r_K + 2 r_j r_{j+1} + r_j flop,
  apply lambda_j = P_j lambda_K + c_j: 2 r_j r_K + r_j flop,
  algorithmic flops = B [sum_{j<K-1} combine_j + sum_j apply_j],
  algorithmic bytes = A (true-width tiles), b, lambda_K read once, lambda
  written once (fp32, padded rows included).

Roofline: the kernel's ideal time is the larger of (algorithmic bytes / HBM
peak) and (matrix-core flops it executes / the peak of the MFMA type it uses);
the larger one names the bound.  Executed matrix-core flops per combine: 2 r^3
for fp32 on the fp32 matrix cores, 4 r^3 for bf16 storage (hi + lo parts of the
composite), 12 r^3 for fp32 as three-part bf16 splits (six partial products).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2605_09204_amd", "csrc")
TRAFFIC_DIR = os.path.join(ROOT, "profiles")

METRIC = "interface combines/sec and achieved MFMA TFLOP/s (r=64, bf16/fp32), % of peak"
# Default warm-up: at least 5 launches and at least this much time.  Under a
# sustained load the GPU's clocks move for some tens of milliseconds (a
# memory-bound launch first gets faster, then up to a third slower, then
# settles), so a short warm-up times a transient rather than the steady state.
WARMUP_MIN_S = 0.25
PEAK = {  # MI355X published peaks
    "hbm_gbs": 8000.0,
    "mfma_f32_tflops": 157.3,
    "mfma_bf16_tflops": 2516.6,
}
ELEM = {"f32": 4, "bf16": 2}


# ----------------------------------------------------------------------------
# accounting
# ----------------------------------------------------------------------------


def warm_up(step, args, torch) -> int:
    """Runs the untimed launches; returns how many (recorded in args.warmup)."""
    if args.warmup is not None:
        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        return args.warmup
    # (launches back to back, as in the timed region: the GPU reaches its
    # sustained clocks under continuous load, which short bursts between
    # synchronizations do not give it; a synchronization every 256 launches
    # bounds the queue)
    n, t0 = 0, time.perf_counter()
    while n < 5 or (time.perf_counter() - t0 < WARMUP_MIN_S and n < 20000):
        step(n)
        n += 1
        if n % 256 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    args.warmup = n
    return n

def widths_of(wl):
    return wl.interface_widths()


def combines(wl) -> int:
    """Algorithmic combines: K-1 per chain (a right-to-left inclusive scan)."""
    return wl.B * (wl.K - 1)


def flops_alg(wl) -> int:
    w = widths_of(wl)
    rK = w[wl.K]
    per_chain = 0
    for j in range(wl.K):
        rj, rj1 = w[j], w[j + 1]
        if j < wl.K - 1:
            per_chain += 2 * rj * rj1 * rK + 2 * rj * rj1 + rj
        per_chain += 2 * rj * rK + rj
    return wl.B * per_chain


def flops_combines(wl) -> int:
    """The combines alone (the suffix-composite export applies nothing)."""
    w = widths_of(wl)
    rK = w[wl.K]
    return wl.B * sum(2 * w[j] * w[j + 1] * rK + 2 * w[j] * w[j + 1] + w[j]
                      for j in range(wl.K - 1))


def bytes_export(wl) -> int:
    """A, b read once; every P_j (r x r, fp32) and c_j (fp32) written once."""
    e = ELEM[wl.dtype]
    R = wl.r
    w = widths_of(wl)
    a = sum(w[j] * w[j + 1] for j in range(wl.K))
    bb = sum(w[:wl.K]) if wl.affine else 0
    return wl.B * ((a + bb) * e + wl.K * (R * R + R) * 4)


def flops_seq(wl) -> int:
    """The sequential chain of K matvecs: lambda_j = A_j lambda_{j+1} + b_j."""
    w = widths_of(wl)
    return wl.B * sum(2 * w[j] * w[j + 1] + w[j] for j in range(wl.K))


def bytes_alg(wl, padded: bool = False, compact_out: bool = False) -> int:
    """A, b, lambda_K read once at true widths (padded: whole tiles), lambda
    written once in fp32 (padded rows included, unless compact_out)."""
    w = widths_of(wl)
    e = ELEM[wl.dtype]
    R = wl.r
    if padded:
        a = wl.K * R * R
    else:
        a = sum(w[j] * w[j + 1] for j in range(wl.K))
    bb = (wl.K * R if padded else sum(w[:wl.K])) if wl.affine else 0
    lk = R if padded else w[wl.K]
    out = (sum(w[:wl.K]) if compact_out else wl.K * R) * 4
    return wl.B * ((a + bb + lk) * e + out)


def mfma_flops_executed(wl, math: str) -> int:
    """Matrix-core flops one launch executes, at the shapes the kernel runs:
    r x r tiles, or with the widths hint the slot's row and k blocks rounded
    up to 16 x a power of two and the r_K columns rounded up to 16; bf16
    products take k in blocks of 32."""
    w = widths_of(wl)
    rK = w[wl.K]
    mode = mode_of(wl, math)
    reps = {"f32-mfma": 1, "bf16": 2, "bf16-single": 1, "f32-split": 6}[mode]

    def blk(x):
        return 16 * (1 << max(0, (-(-x // 16) - 1).bit_length()))

    cols = 16 * -(-rK // 16) if wl.widths else wl.r
    per_chain = 0
    for j in range(wl.K - 1):
        rows = blk(w[j]) if wl.widths else wl.r
        ks = blk(w[j + 1]) if wl.widths else wl.r
        if mode != "f32-mfma":
            ks = 32 * -(-ks // 32)
        per_chain += 2 * rows * ks * cols
    return wl.B * per_chain * reps


def mode_of(wl, math: str) -> str:
    if wl.dtype == "bf16":
        return "bf16-single" if math == "bf16single" else "bf16"
    if math == "split" and wl.r <= 64:
        return "f32-split"
    return "f32-mfma"


def scan_payload_bytes(K: int, r: int, elem: int) -> int:
    """K interface matrices of r x r (the paper's cross-device scan payload)."""
    return K * r * r * elem


# The sources the chain-scan kernel is compiled from (its traffic counters
# stay valid while these are unchanged).
CHAIN_SOURCES = ("lbi_chain.hpp", "lbi_chain_f32.hip", "lbi_chain_f32x.hip", "lbi_chain_bf16.hip",
                 "lbi_chain_ring.hip", "lbi_device.hpp", "lbi_internal.h")


def source_hash() -> str:
    """Hash of the chain-scan kernel's sources (the PMC traffic figures hold for it only)."""
    h = hashlib.sha256()
    for name in CHAIN_SOURCES:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def _counter_rows(path):
    """(kernel name, counter name, value) per dispatch of a rocprofv3
    counter-collection CSV."""
    import csv
    rows = []
    with open(path, newline="") as f:
        for rec in csv.DictReader(f):
            name = rec.get("Kernel_Name") or rec.get("Kernel-Name") or ""
            cname = rec.get("Counter_Name") or rec.get("Counter-Name") or ""
            val = rec.get("Counter_Value") or rec.get("Counter-Value") or "nan"
            rows.append((name, cname, float(val)))
    return rows


def record_traffic(workload: str, fetch_csv: str, write_csv: str, copy_mib: int) -> dict:
    """HBM bytes per launch of the scan kernel from two rocprofv3 PMC runs
    (FETCH_SIZE, then WRITE_SIZE, in KiB per dispatch), each scaled by what the
    same counter reads for the calibration copy kernel of known size."""
    copy_bytes = float(copy_mib << 20)
    out = {"workload": workload, "source_sha256_16": source_hash(),
           "calibration_copy_bytes": copy_bytes}
    for tag, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"),
                               ("write", write_csv, "WRITE_SIZE")):
        rows = [r for r in _counter_rows(path) if r[1] == counter]
        scan = [v for n, _, v in rows if "scan_chain_kernel" in n or "scan_ring_kernel" in n]
        copy = [v for n, _, v in rows if "neg_kernel" in n]
        if not scan or not copy:
            raise SystemExit(f"{path}: no {counter} rows for the scan or the copy kernel")
        kib_scan = sum(scan) / len(scan)
        kib_copy = sum(copy) / len(copy)
        factor = copy_bytes / (kib_copy * 1024.0)
        out[f"{tag}_kib_per_dispatch"] = kib_scan
        out[f"{tag}_copy_kib_per_dispatch"] = kib_copy
        out[f"{tag}_scale"] = factor
        out[f"{tag}_bytes_per_launch"] = kib_scan * 1024.0 * factor
        out[f"{tag}_dispatches"] = len(scan)
    out["hbm_bytes_per_launch"] = out["fetch_bytes_per_launch"] + out["write_bytes_per_launch"]
    wl_bytes = None
    try:
        from paper_2605_09204_amd import synth
        wl_bytes = bytes_alg(synth.WORKLOADS[workload])
    except Exception:
        pass
    out["alg_bytes_per_launch"] = wl_bytes
    os.makedirs(TRAFFIC_DIR, exist_ok=True)
    path = os.path.join(TRAFFIC_DIR, f"traffic_{workload}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    return out


def load_traffic(workload: str):
    """Measured HBM bytes per launch from the rocprofv3 PMC runs, if they were
    taken on the current kernel source; else None."""
    path = os.path.join(TRAFFIC_DIR, f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256_16") != source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def norms_record(wl, args, total_ms, avg_launch_s, per_launch_ms, ncopy) -> dict:
    """JSON line of the --op norms run: spectral + Frobenius norms of every
    r x r tile of A.  Executed fp32 matrix-core work per matrix: the Gram
    product and 24 normalised squarings, 25 r x r x r products (50 r^3 flop);
    bytes: the A stack read twice (norms, then the Rayleigh quotient's
    matrix-vector product) and two floats written per matrix."""
    n = wl.B * wl.K
    f_exec = 50.0 * wl.r ** 3 * n
    b_alg = 2.0 * n * wl.r * wl.r * ELEM[wl.dtype] + 8.0 * n
    t_mfma = f_exec / (PEAK["mfma_f32_tflops"] * 1e12)
    t_hbm = b_alg / (PEAK["hbm_gbs"] * 1e9)
    ach = f_exec / avg_launch_s / 1e12
    return {
        "metric": "interface-Jacobian norms/sec (spectral + Frobenius, appendix statistics)",
        "value": n * args.steps / (total_ms / 1e3),
        "unit": "matrices/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": total_ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Haar-orthogonal x diag x Haar-orthogonal interface "
                "Jacobians; no dataset or checkpoint)",
        "config": {"workload": wl.name, "B": wl.B, "K": wl.K, "r": wl.r, "storage": wl.dtype,
                   "op": "norms", "parallelism": "1 GPU, one wavefront per matrix"
                   if wl.r <= 64 else "1 GPU, one workgroup per matrix"},
        "roofline": {"bound": "mfma" if t_mfma >= t_hbm else "hbm",
                     "achieved": ach if t_mfma >= t_hbm else b_alg / avg_launch_s / 1e9,
                     "peak": PEAK["mfma_f32_tflops"] if t_mfma >= t_hbm else PEAK["hbm_gbs"],
                     "unit": "TFLOP/s" if t_mfma >= t_hbm else "GB/s",
                     "frac": (ach / PEAK["mfma_f32_tflops"]) if t_mfma >= t_hbm
                     else (b_alg / avg_launch_s / 1e9) / PEAK["hbm_gbs"],
                     "traffic": None},
        "extra": {"avg_launch_ms": avg_launch_s * 1e3, "min_launch_ms": min(per_launch_ms),
                  "executed_mfma_tflops": ach, "ideal_ms_mfma": t_mfma * 1e3,
                  "ideal_ms_hbm": t_hbm * 1e3, "input_copies_rotated": ncopy},
    }


def region_flops(wl) -> float:
    """Matrix-core flops of one Phase 1 call (all B sequences, K regions): the
    token product L x D x X per sequence and region, and the tangent products
    with N = B r per region (Jdec: D x D, W1: X x D, W2: D x X, W_e1: D x D,
    W_e2: r x D)."""
    tok = 2.0 * wl.B * wl.K * wl.L * wl.D * wl.X
    tan = 2.0 * wl.K * wl.B * wl.r * (2 * wl.D * wl.D + 2 * wl.X * wl.D + wl.r * wl.D)
    return tok + tan


def region_ssm_flops(wl) -> float:
    """Matrix-core flops of one Phase 1 call with the token-mixing block: per
    sequence and region the forward's two token products (L x D x X each) and
    the tangent's two per-token products over the r directions (L r x D x X
    each), plus the products with N = B r per region (Jdec: D x D, W_e1:
    D x D, W_e2: r x D)."""
    tok = 4.0 * wl.B * wl.K * wl.L * wl.D * wl.X
    tan = 4.0 * wl.B * wl.K * wl.L * wl.r * wl.D * wl.X
    small = 2.0 * wl.K * wl.B * wl.r * (2 * wl.D * wl.D + wl.r * wl.D)
    return tok + tan + small


def bench_phase1(args) -> int:
    import torch
    from paper_2605_09204_amd import binding, synth

    if args.workload not in synth.REGION_WORKLOADS:
        args.workload = "region_paper"
    wl = synth.REGION_WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    print(f"[bench] generating {wl.name}", file=sys.stderr, flush=True)
    x = synth.generate_region(wl, device=dev)
    ssm = args.phi == "ssm"
    need = (binding.lbi_region_jacobians_ssm_workspace_bytes if ssm else
            binding.lbi_region_jacobians_workspace_bytes)(wl.B, wl.K, wl.L, wl.D, wl.X, wl.r)
    ws = torch.empty((need,), dtype=torch.uint8, device=dev)
    A = torch.empty((wl.B, wl.K, wl.r, wl.r), dtype=torch.float32, device=dev)
    mn = torch.empty((wl.B, wl.K, wl.r), dtype=torch.float32, device=dev)
    call = binding.lbi_region_jacobians_ssm if ssm else binding.lbi_region_jacobians

    def step(i):
        call(x.params, x.x_embed, x.m, A=A, m_next=mn, workspace=ws)

    warm_up(step, args, torch)
    stream = torch.cuda.current_stream(dev)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    for i in range(args.steps):
        starts[i].record(stream)
        step(i)
        ends[i].record(stream)
    torch.cuda.synchronize()
    per = [a.elapsed_time(b) for a, b in zip(starts, ends)]
    total_ms = starts[0].elapsed_time(ends[-1])
    avg_s = sum(per) / len(per) / 1e3
    f = region_ssm_flops(wl) if ssm else region_flops(wl)
    ach = f / avg_s / 1e12
    out = {
        "metric": "interface Jacobians/sec (Phase 1, synthetic region map"
                  + (", token-mixing block)" if ssm else ")"),
        "value": wl.B * wl.K * args.steps / (total_ms / 1e3),
        "unit": "jacobians/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": total_ms / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random region weights, x_embed and interface states; "
                "no dataset or checkpoint)",
        "config": {"workload": wl.name, "B": wl.B, "K": wl.K, "L": wl.L, "D": wl.D, "X": wl.X,
                   "r": wl.r, "op": "phase1", "phi": args.phi, "parallelism": "1 GPU"},
        "roofline": {"bound": "mfma", "achieved": ach, "peak": PEAK["mfma_bf16_tflops"],
                     "unit": "TFLOP/s", "frac": ach / PEAK["mfma_bf16_tflops"],
                     "traffic": None},
        "extra": {"avg_launch_ms": avg_s * 1e3, "min_launch_ms": min(per),
                  "flops_per_call": f, "workspace_bytes": need},
    }
    print(json.dumps(out), flush=True)
    return 0


# ----------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample of the same workload
# ----------------------------------------------------------------------------

def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), or the platform's."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.lower().startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def cpu_baseline(x, run_s: float = 5.0, nthreads: int = 0, runs: int = 3):
    """The fp64 oracle recurrence on the host, timed as the median of ``runs``
    runs of about ``run_s`` seconds each over a bounded sample of the same
    chains (the first n chains, n sized by a calibration run; a batch too
    small to last run_s is repeated within each run)."""
    import oracle
    import torch

    wl = x.workload
    threads = oracle.threads(nthreads)
    n_cal = min(wl.B, max(1, threads))
    host = x.chains(torch.arange(n_cal)).to("cpu")
    t0 = time.perf_counter()
    oracle.recurrence(host.A, host.b, host.lamK, nthreads)
    t_cal = max(time.perf_counter() - t0, 1e-6)
    n = int(min(wl.B, max(n_cal, n_cal * run_s / t_cal)))
    host = x.chains(torch.arange(n)).to("cpu")
    t0 = time.perf_counter()
    oracle.recurrence(host.A, host.b, host.lamK, nthreads)
    t_one = max(time.perf_counter() - t0, 1e-6)
    reps = max(1, min(4096, int(round(run_s / t_one))))
    times = []
    for _ in range(runs):
        t0 = time.perf_counter()
        for _ in range(reps):
            oracle.recurrence(host.A, host.b, host.lamK, nthreads)
        times.append(time.perf_counter() - t0)
    med = sorted(times)[len(times) // 2]
    return {
        "value": reps * n * (wl.K - 1) / med,
        "unit": "combines/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{n} of {wl.B} chains x {reps} pass(es) per run, all K={wl.K} slots, "
                  f"fp64 recurrence over the same {wl.dtype} inputs; median of {runs} runs "
                  f"({', '.join(f'{t:.2f}' for t in times)} s)",
        "cpu_model": cpu_model(),
        "threads": threads,
        "runs_s": times,
    }


# ----------------------------------------------------------------------------
# one adjoint-type measurement (the JSON line without the CPU baseline)
# ----------------------------------------------------------------------------

def time_launches(step, steps, warmup, torch, dev):
    """Warm-up, then ``steps`` timed launches bracketed by HIP events on the
    launch stream.  Returns (per-launch ms, first-start to last-end ms, wall
    s, warm-up launches)."""
    class _W:
        pass
    wa = _W()
    wa.warmup = warmup
    nwarm = warm_up(step, wa, torch)
    stream = torch.cuda.current_stream(dev)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for i in range(steps):
        starts[i].record(stream)
        step(i)
        ends[i].record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    per_launch_ms = [st.elapsed_time(en) for st, en in zip(starts, ends)]
    return per_launch_ms, starts[0].elapsed_time(ends[-1]), t_wall, nwarm


def chain_mapping(wl, op, layout, math_name, algo_name, need) -> str:
    """The chain mapping the library uses (for adjoints, its AUTO rule unless
    the two-level scan is taken: bf16 with r <= 32 and B <= 8192 one
    wavefront per chain; fp32 split arithmetic at r = 64 with B <= 256
    sixteen waves per chain; else one workgroup per chain)."""
    auto_adj = algo_name == "auto" and op == "adjoints" and layout == "padded"
    chunk = 8 if wl.r == 64 else 16
    if algo_name == "tree" or (auto_adj and wl.r <= 32 and wl.B <= 256 and wl.K <= chunk
                               and math_name == "split"
                               and wl.K >= (5 if wl.dtype == "f32" else 9)):
        return "log-depth tree scan (a workgroup per chunk of slots, levels of aggregates)"
    if need:
        return "two-level scan (segments in parallel)"
    ring_widths = wl.widths is not None and wl.widths[-1] == 64 and all(
        w in (32, 64, 128) for w in wl.widths) and all(
        (wl.widths[j] // 16) * (wl.widths[j + 1] // 32) <= 16 for j in range(wl.K))
    if algo_name == "chain_ring" or (layout == "compact" and wl.dtype == "bf16" and ring_widths
                                     and math_name != "bf16single") or (
            algo_name == "auto" and op == "adjoints" and wl.dtype == "bf16" and wl.r == 128
            and ring_widths and math_name != "bf16single"):
        return "one workgroup per chain, A tiles loaded into an LDS ring"
    if algo_name == "chain_wave" or (auto_adj and wl.dtype == "bf16" and wl.r <= 32
                                     and wl.B <= 8192 and math_name != "bf16single"):
        return "one wavefront per chain"
    if algo_name == "chain_splitk" or (auto_adj and wl.dtype == "f32" and math_name == "split"
                                       and wl.r == 64 and wl.B <= 256):
        return "sixteen waves per chain (split contraction, staging waves)"
    return "one workgroup per chain"


def roofline(wl, math_name, b_alg, avg_launch_s, f_alg):
    """(roofline dict without traffic, executed matrix-core flops, peak, ideal
    matrix-core s, ideal HBM s) of one launch: the bound is whichever of HBM
    and the matrix cores gives the larger ideal time."""
    mode = mode_of(wl, math_name)
    f_exec = mfma_flops_executed(wl, math_name)
    mfma_peak = PEAK["mfma_f32_tflops"] if mode == "f32-mfma" else PEAK["mfma_bf16_tflops"]
    t_mfma = f_exec / (mfma_peak * 1e12)
    t_hbm = b_alg / (PEAK["hbm_gbs"] * 1e9)
    tflops = f_alg / avg_launch_s / 1e12
    gbs = b_alg / avg_launch_s / 1e9
    if t_mfma >= t_hbm:
        # matrix-core bound: algorithmic flops against the fp32 peak when the
        # products run on the fp32 matrix cores, else executed bf16 flops
        # against the bf16 peak
        ach = tflops if mode == "f32-mfma" else f_exec / avg_launch_s / 1e12
        roof = {"bound": "mfma", "achieved": ach, "peak": mfma_peak, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": gbs, "peak": PEAK["hbm_gbs"], "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    return roof, f_exec, mfma_peak, t_mfma, t_hbm


# ----------------------------------------------------------------------------
# main
# ----------------------------------------------------------------------------

def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed launches (default: >= 5 and >= %.2f s of launches)" % WARMUP_MIN_S)
    ap.add_argument("--workload", default="long_chain")
    ap.add_argument("--math", choices=["split", "mfma", "bf16single"], default="split",
                    help="float32 arithmetic: three-part bf16 splits on the bf16 matrix "
                         "cores (the library default) or the fp32 matrix cores; for bf16 "
                         "storage, bf16single feeds the running composite back rounded "
                         "once to bf16 (opt-in, lower accuracy)")
    ap.add_argument("--algo", choices=["auto", "chain", "two_level", "chain_wave", "chain_splitk",
                                       "tree", "chain_ring"],
                    default="auto",
                    help="scan algorithm (auto: the library's choice)")
    ap.add_argument("--op", choices=["adjoints", "suffix_products", "streaming", "norms",
                                     "phase1"],
                    default="adjoints",
                    help="what one step computes: every lambda_j (lbi_scan_backward_ex), "
                         "every composite (P_j, c_j) (lbi_scan_suffix_products), every "
                         "lambda_j with progress published (lbi_scan_backward_streaming), or "
                         "the spectral and Frobenius norm of every A_j (lbi_matrix_norms; "
                         "reported in matrices/s), or Phase 1, the interface Jacobians of "
                         "every region (lbi_region_jacobians; --workload region_paper or "
                         "region_small)")
    ap.add_argument("--phi", choices=["mlp", "ssm"], default="mlp",
                    help="phase1: the region block, token-wise MLP (lbi_region_jacobians) or "
                         "token-mixing recurrence with a gated MLP (lbi_region_jacobians_ssm)")
    ap.add_argument("--chunk", type=int, default=16, help="streaming: slots per publication")
    ap.add_argument("--layout", choices=["padded", "compact"], default="padded",
                    help="adjoints: R x R tiles with the widths hint (lbi_scan_backward_ex), or "
                         "tiles at their true shapes back to back (lbi_scan_backward_ragged)")
    ap.add_argument("--B", type=int, default=0, help="override the workload's chain count")
    ap.add_argument("--K", type=int, default=0, help="override the workload's slot count")
    ap.add_argument("--r", type=int, default=0, help="override the workload's interface width")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="time only the chosen workload (by default a headline run also "
                         "times every other workload of the table, under extra.configs)")
    ap.add_argument("--per-launch", action="store_true",
                    help="print every timed launch's duration (µs) to stderr")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="also run a plain device copy of this many MiB (for PMC scaling)")
    ap.add_argument("--record-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic_<workload>.json from two rocprofv3 "
                         "counter-collection CSVs (FETCH_SIZE, WRITE_SIZE) of a run with "
                         "--copy-calibration MIB, then exit")
    args = ap.parse_args(argv)

    if args.record_traffic:
        if args.copy_calibration <= 0:
            print("--record-traffic needs the --copy-calibration MIB of the PMC runs",
                  file=sys.stderr)
            return 2
        rec = record_traffic(args.workload, args.record_traffic[0], args.record_traffic[1],
                             args.copy_calibration)
        print(json.dumps(rec))
        return 0

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(chains are independent, so B shards across GPUs with no communication)",
              file=sys.stderr)
        return 2
    if args.math == "bf16single" and args.op != "phase1":
        from paper_2605_09204_amd import synth as _synth
        wl0 = _synth.WORKLOADS.get(args.workload)
        if wl0 is not None and wl0.dtype != "bf16":
            print(f"--math bf16single needs bf16 storage; workload {args.workload} is "
                  f"{wl0.dtype}", file=sys.stderr)
            return 2

    import torch
    from paper_2605_09204_amd import binding, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    binding.load()  # fail loudly before any work if the library is missing
    if args.op == "phase1":
        return bench_phase1(args)
    if args.workload not in synth.WORKLOADS:
        print(f"unknown workload {args.workload}; one of {list(synth.WORKLOADS)}",
              file=sys.stderr)
        return 2
    wl = synth.WORKLOADS[args.workload]
    if args.B or args.K or args.r:
        if wl.widths is not None and (args.K or args.r):
            print("--K/--r apply to uniform-width workloads only", file=sys.stderr)
            return 2
        wl = wl.with_(B=args.B or wl.B, K=args.K or wl.K, r=args.r or wl.r,
                      name=f"{wl.name}_B{args.B or wl.B}_K{args.K or wl.K}_r{args.r or wl.r}")
    if args.layout == "compact" and (args.op != "adjoints" or args.algo == "two_level" or any(
            wk % 16 for wk in wl.interface_widths())):
        print("--layout compact: adjoints, chain scan, widths multiples of 16", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    out, x = measure(wl, args.op, args.layout, args.math, args.algo, args.steps, args.warmup,
                     args.chunk, torch, binding, synth, dev,
                     copy_calibration=args.copy_calibration, per_launch=args.per_launch)
    args.warmup = out["warmup"]
    if not args.no_cpu_baseline and args.op != "norms":
        print("[bench] timing the CPU oracle baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(x)
        # the same oracle on one core (a smaller sample)
        one = cpu_baseline(x, run_s=1.5, nthreads=1)
        out["extra"]["cpu_oracle_one_core"] = {"value": one["value"], "unit": one["unit"],
                                               "sample": one["sample"]}
    # the other workloads of the table, timed in the same run (one line, the
    # headline's; each of the others as an entry of extra.configs)
    headline = (args.op == "adjoints" and args.layout == "padded" and args.math == "split"
                and args.algo == "auto" and not (args.B or args.K or args.r)
                and not args.no_other_configs)
    if headline:
        del x
        torch.cuda.empty_cache()
        others = {}
        for name in synth.WORKLOAD_ORDER:
            if name == wl.name:
                continue
            w2 = synth.WORKLOADS[name]
            steps2 = 200 if w2.B * w2.K <= 4096 else 30
            o2, x2 = measure(w2, "adjoints", "padded", "split", "auto", steps2, None,
                             args.chunk, torch, binding, synth, dev)
            rec = {"ms_per_step": o2["ms_per_step"],
                   "avg_launch_ms": o2["extra"]["avg_launch_ms"],
                   "value": o2["value"], "unit": o2["unit"], "steps": steps2,
                   "warmup": o2["warmup"], "dtype": o2["dtype"], "config": o2["config"],
                   "roofline": o2["roofline"], "alg_tflops": o2["extra"]["alg_tflops"],
                   "alg_hbm_gbs": o2["extra"]["alg_hbm_gbs"],
                   "work_inflation_vs_sequential":
                       o2["extra"]["work_inflation_vs_sequential"]}
            if "graph_replay" in o2["extra"]:
                rec["graph_replay"] = o2["extra"]["graph_replay"]
            if not args.no_cpu_baseline:
                print(f"[bench] timing the CPU oracle baseline on {name}", file=sys.stderr,
                      flush=True)
                rec["cpu_baseline"] = cpu_baseline(x2, run_s=1.5)
            others[name] = rec
            del x2
            torch.cuda.empty_cache()
            if name == "mixed_widths":
                # the same workload in compact storage (tiles at their true
                # shapes back to back): no over-read of the zero padding
                o3, x3 = measure(w2, "adjoints", "compact", "split", "auto", steps2, None,
                                 args.chunk, torch, binding, synth, dev)
                others["mixed_widths_compact"] = {
                    "ms_per_step": o3["ms_per_step"],
                    "avg_launch_ms": o3["extra"]["avg_launch_ms"],
                    "value": o3["value"], "unit": o3["unit"], "steps": steps2,
                    "warmup": o3["warmup"], "dtype": o3["dtype"], "config": o3["config"],
                    "roofline": o3["roofline"], "alg_tflops": o3["extra"]["alg_tflops"],
                    "alg_hbm_gbs": o3["extra"]["alg_hbm_gbs"]}
                del x3
                torch.cuda.empty_cache()
        out["extra"]["configs"] = others
    print(json.dumps(out), flush=True)
    return 0


def measure(wl, op, layout, math_name, algo_name, steps, warmup, chunk, torch, binding, synth,
            dev, copy_calibration=0, per_launch=False):
    """Times ``steps`` launches of one operation on workload ``wl``; returns
    (the JSON record without the CPU baseline, the inputs)."""
    print(f"[bench] generating {wl.name}: B={wl.B} K={wl.K} r={wl.r} {wl.dtype}",
          file=sys.stderr, flush=True)
    t0 = time.time()
    x = synth.generate(wl, device=dev)
    torch.cuda.synchronize()
    print(f"[bench] inputs ready in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)

    # rotate through enough input copies that no step reuses the last-level cache
    in_bytes = bytes_alg(wl, padded=True)
    ncopy = max(1, min(8, -(-(1 << 30) // in_bytes)))
    copies = [x] + [synth.Inputs(x.A.clone(), None if x.b is None else x.b.clone(),
                                 x.lamK.clone(), x.widths, wl) for _ in range(ncopy - 1)]
    lam = torch.empty((wl.B, wl.K, wl.r), dtype=torch.float32, device=dev)
    hint = wl.widths

    math = {"split": binding.LBI_MATH_F32_SPLIT, "mfma": binding.LBI_MATH_F32_MFMA,
            "bf16single": binding.LBI_MATH_BF16_SINGLE}[math_name]
    algo = {"auto": binding.LBI_ALGO_AUTO, "chain": binding.LBI_ALGO_CHAIN,
            "two_level": binding.LBI_ALGO_TWO_LEVEL,
            "chain_wave": binding.LBI_ALGO_CHAIN_WAVE,
            "chain_splitk": binding.LBI_ALGO_CHAIN_SPLITK,
            "tree": binding.LBI_ALGO_TREE,
            "chain_ring": binding.LBI_ALGO_CHAIN_RING}[algo_name]
    need = binding.lbi_scan_backward_workspace_bytes_ex(wl.B, wl.K, wl.r,
                                                         0 if wl.dtype == "f32" else 1, algo)
    ws = torch.empty((need,), dtype=torch.uint8, device=dev) if need else None

    if op == "streaming":
        progress = torch.zeros(wl.B, dtype=torch.int32, device=dev)

        def step(i):
            c = copies[i % ncopy]
            progress.zero_()
            binding.lbi_scan_backward_streaming(c.A, c.b, c.lamK, progress, chunk, hint,
                                                math, lam=lam)
    elif op == "norms":
        spec = torch.empty((wl.B, wl.K), dtype=torch.float32, device=dev)
        fro = torch.empty((wl.B, wl.K), dtype=torch.float32, device=dev)

        def step(i):
            c = copies[i % ncopy]
            binding.lbi_matrix_norms(c.A, spec=spec, fro=fro)
    elif op == "suffix_products":
        Pout = torch.empty((wl.B, wl.K, wl.r, wl.r), dtype=torch.float32, device=dev)
        cout = torch.empty((wl.B, wl.K, wl.r), dtype=torch.float32, device=dev)

        def step(i):
            c = copies[i % ncopy]
            binding.lbi_scan_suffix_products(c.A, c.b, hint, math, P=Pout, c=cout)
    elif layout == "compact":
        packed = [synth.pack_ragged(c) for c in copies]
        lam_c = torch.empty((wl.B, sum(wl.interface_widths()[:wl.K])), dtype=torch.float32,
                            device=dev)

        def step(i):
            c = packed[i % ncopy]
            binding.lbi_scan_backward_ragged(c.A, c.b, c.lamK, c.widths, math, lam=lam_c)
    else:
        def step(i):
            c = copies[i % ncopy]
            binding.lbi_scan_backward_ex(c.A, c.b, c.lamK, hint, math, algo, lam=lam,
                                         workspace=ws)

    if copy_calibration > 0:
        # A plain streaming kernel of known size (torch's elementwise negation:
        # reads and writes MiB << 20 bytes each) against which the PMC byte
        # counters of the scan kernel are scaled.
        n = (copy_calibration << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    per_launch_ms, total_ms, t_wall, nwarm = time_launches(step, steps, warmup, torch, dev)
    graph = None
    if op == "adjoints" and sum(per_launch_ms) / len(per_launch_ms) < 0.05:
        graph = graph_replay(step, 64, torch)
    if per_launch:
        print("[bench] per-launch µs: " + " ".join(f"{t * 1e3:.1f}" for t in per_launch_ms),
              file=sys.stderr, flush=True)
    avg_launch_s = sum(per_launch_ms) / len(per_launch_ms) / 1e3
    ms_per_step = total_ms / steps

    if op == "norms":
        class _A:
            pass
        na = _A()
        na.steps, na.warmup = steps, nwarm
        return norms_record(wl, na, total_ms, avg_launch_s, per_launch_ms, ncopy), x
    value = combines(wl) * steps / (total_ms / 1e3)
    f_alg = flops_combines(wl) if op == "suffix_products" else flops_alg(wl)
    mapping = chain_mapping(wl, op, layout, math_name, algo_name, need)
    b_alg = (bytes_export(wl) if op == "suffix_products"
             else bytes_alg(wl, compact_out=layout == "compact"))
    tflops = f_alg / avg_launch_s / 1e12
    gbs = b_alg / avg_launch_s / 1e9
    mode = mode_of(wl, math_name)
    roof, f_exec, mfma_peak, t_mfma, t_hbm = roofline(wl, math_name, b_alg, avg_launch_s, f_alg)
    roof["traffic"] = (load_traffic(wl.name) if op == "adjoints" and layout == "padded" and
                       (math_name == "split" or (wl.dtype == "bf16" and
                                                 math_name != "bf16single")) else None)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "combines/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": nwarm,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded Haar-orthogonal x diag x Haar-orthogonal interface "
                "Jacobians; no dataset or checkpoint)",
        "config": {"workload": wl.name, "B": wl.B, "K": wl.K, "r": wl.r,
                   "storage": wl.dtype, "affine": wl.affine, "arithmetic": mode,
                   "algorithm": algo_name, "workspace_bytes": need, "op": op,
                   "layout": layout,
                   "widths": "cyclic 32/64/128" if wl.widths else "uniform",
                   "parallelism": "1 GPU, " + mapping},
        "roofline": roof,
        "extra": {
            "alg_tflops": tflops,
            "pct_of_fp32_mfma_peak": 100.0 * tflops / PEAK["mfma_f32_tflops"],
            "executed_mfma_tflops": f_exec / avg_launch_s / 1e12,
            "executed_mfma_peak_tflops": mfma_peak,
            "ideal_ms_hbm": t_hbm * 1e3,
            "ideal_ms_mfma": t_mfma * 1e3,
            "alg_hbm_gbs": gbs,
            "pct_of_hbm_peak": 100.0 * gbs / PEAK["hbm_gbs"],
            "avg_launch_ms": avg_launch_s * 1e3,
            "min_launch_ms": min(per_launch_ms),
            "work_inflation_vs_sequential": f_alg / flops_seq(wl),
            "alg_flops_per_launch": f_alg,
            "alg_bytes_per_launch": b_alg,
            "input_copies_rotated": ncopy,
            "wall_s_timed_region": t_wall,
        },
    }
    if graph is not None:
        # launch-bound calls replayed from a HIP graph (the library enqueues
        # kernels only, so a captured sequence of calls replays the same work)
        out["extra"]["graph_replay"] = {"calls_per_graph": graph[0], "us_per_call": graph[1],
                                        "combines_per_s": combines(wl) / (graph[1] * 1e-6)}
    return out, x


def graph_replay(step, n, torch):
    """(n, µs per call): n calls of ``step`` captured in one HIP graph (through
    torch's graph API) and replayed ten times back to back, timed with events."""
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g):
            for i in range(n):
                step(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(10):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return n, a.elapsed_time(b) * 1e3 / (10 * n)

if __name__ == "__main__":
    sys.exit(main())
