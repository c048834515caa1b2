"""Benchmark of the ID Balancing router + controller step on one MI355X.

One step = the whole hot path over one batch: fused gate contraction +
sigmoid + biased Top-K + gate weights + load counts (idb_router_forward),
the ID controller update (idb_controller_update) and MaxVio/MinVio
(idb_load_stats).  Inputs are synthetic, seeded, resident in HBM before the
timed region; the hidden-state batch rotates over several distinct buffers so
it is not served from the 256 MB Infinity Cache.  Each step is one HIP graph
replay (the graph holds exactly the ABI calls of one step).

Prints one JSON line: routed tokens/s for the step, with the dominant
kernel's roofline and the CPU oracle timed on a bounded sample of the same
workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
PROFILES = os.path.join(ROOT, "profiles")
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3  # MI355X fp32 (vector and 32x32x2 matrix path alike, dense)
PEAK_HBM_GBS = 8000.0


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def router_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("router.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2609_39137_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(workload: str, variant_id: int):
    """HBM bytes per launch of the dominant kernel from a committed PMC summary, or None if stale/absent."""
    path = os.path.join(PROFILES, f"router_score_select_{workload}_pmc.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_sha256") != router_source_hash() or d.get("variant") != variant_id:
        return None
    return d.get("hbm_bytes_per_launch")


def cpu_baseline(wl, W, target_s: float):
    """Time the CPU oracle (router + controller + stats) on a bounded sample of the workload."""
    import oracle
    from paper_2609_39137_amd import synth

    threads = oracle.num_threads()
    n = 64
    x = synth.hidden_states(wl, step=0, rows=np.arange(n))
    st = oracle.ControllerState(wl.E)
    t = oracle.step_seconds(x, W, wl.K, 6e-3, 6e-3, st)
    n = int(min(wl.T, max(n, n * target_s / max(t, 1e-6))))
    n = max(64, (n // 64) * 64)
    x = synth.hidden_states(wl, step=0, rows=np.arange(n))
    st = oracle.ControllerState(wl.E)
    t = oracle.step_seconds(x, W, wl.K, 6e-3, 6e-3, st)
    return {
        "value": n / t,
        "unit": "routed tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"first {n} of the {wl.T} tokens of step 0 ({wl.name}), one router step + ID update + "
                  f"MaxVio/MinVio, {t:.2f} s wall on {threads} OpenMP threads",
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None, help="synthetic workload name (default: the Top-10-of-768 shape)")
    ap.add_argument("--variant", type=int, default=0, help="router tiling (0 = automatic)")
    ap.add_argument("--buffers", type=int, default=0, help="distinct hidden-state buffers to rotate (0 = auto)")
    ap.add_argument("--eager", action="store_true", help="launch the ABI calls directly instead of graph replays")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=3.0, help="wall-clock target of the CPU oracle sample")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (the count all-reduce across "
              f"data-parallel ranks is design-only in this build)", file=sys.stderr)
        return 2

    import torch

    from paper_2609_39137_amd import binding as B
    from paper_2609_39137_amd import synth
    from paper_2609_39137_amd.pipeline import RouterStep

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = "cuda"
    wl = synth.WORKLOADS[args.workload or synth.HEADLINE]
    tdtype = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    x_bytes = wl.T * wl.d * (2 if wl.dtype == "bf16" else 4)
    nbuf = args.buffers or max(1, min(8, math.ceil(512 * 2**20 / x_bytes)))
    if x_bytes > 256 * 2**20:
        nbuf = args.buffers or 1  # already larger than the Infinity Cache
    log(f"workload {wl.name}: T={wl.T} d={wl.d} E={wl.E} K={wl.K} {wl.dtype}; {nbuf} input buffers")

    W_np = synth.router_weight(wl)

    def to_dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(a).to(dev)

    W = to_dev(W_np)
    xs = [to_dev(synth.hidden_states(wl, step=i)) for i in range(nbuf)]
    log("inputs resident on the GPU")

    rs = RouterStep(wl.T, wl.d, wl.E, wl.K, tdtype, B.ControllerCfg(wl.E, 6e-3, 6e-3), variant=args.variant)
    log(f"router tiling {rs.info}")
    stream = torch.cuda.Stream()  # default priority
    torch.cuda.synchronize()

    # eager warm-up (also validates every call)
    with torch.cuda.stream(stream):
        for i in range(2):
            rs.step(xs[i % nbuf], W)
    torch.cuda.synchronize()

    step_graphs, k1_graphs = [], []
    if not args.eager:
        with torch.cuda.stream(stream):
            for i in range(nbuf):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=stream):
                    rs.step(xs[i], W)
                step_graphs.append(g)
            for i in range(nbuf):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=stream):
                    rs.score_select(xs[i], W)
                k1_graphs.append(g)
        torch.cuda.synchronize()

    def run_steps(n, start=0):
        for k in range(start, start + n):
            if args.eager:
                rs.step(xs[k % nbuf], W, stream=stream)
            else:
                step_graphs[k % nbuf].replay()

    with torch.cuda.stream(stream):
        run_steps(args.warmup)
    torch.cuda.synchronize()
    log(f"warm-up of {args.warmup} steps done")

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        torch.cuda.synchronize()
        ev0.record(stream)
        run_steps(args.steps, args.warmup)
        ev1.record(stream)
    torch.cuda.synchronize()
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / args.steps
    log(f"timed {args.steps} steps: {ms_step * 1000:.2f} us/step")

    # sanity of the last step's outputs
    counts = rs.counts.cpu()
    assert int(counts.sum()) == wl.T * wl.K, "counts do not sum to T*K"
    assert int(rs.state.status.item()) == 0
    stats = rs.stats.cpu().tolist()

    # live timing of the dominant kernel (score/select) on the same stream
    n_k1 = max(args.steps, 50)
    with torch.cuda.stream(stream):
        for k in range(5):
            (k1_graphs[k % nbuf].replay() if k1_graphs else rs.score_select(xs[k % nbuf], W, stream=stream))
        torch.cuda.synchronize()
        ev0.record(stream)
        for k in range(n_k1):
            (k1_graphs[k % nbuf].replay() if k1_graphs else rs.score_select(xs[k % nbuf], W, stream=stream))
        ev1.record(stream)
    torch.cuda.synchronize()
    k1_ms = ev0.elapsed_time(ev1) / n_k1
    log(f"score/select kernel: {k1_ms * 1000:.2f} us/launch")

    flops = wl.flops
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = flops / (k1_ms * 1e-3) / 1e12
    roofline = {
        "bound": "mfma",
        "achieved": round(achieved, 2),
        "peak": peak,
        "unit": "TFLOP/s",
        "frac": round(achieved / peak, 4),
        "traffic": load_traffic(wl.name, rs.info["variant"]),
        "kernel": "router_score_select_kernel",
        "kernel_us": round(k1_ms * 1000, 2),
    }
    value = wl.T / (ms_step * 1e-3)
    out = {
        "metric": "routed tokens/sec for router+ID-update step, Top-10-of-768; % MFMA/HBM roofline",
        "value": round(value, 1),
        "unit": "routed tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "T": wl.T, "d": wl.d, "E": wl.E, "K": wl.K, "global_batch": wl.T,
                   "parallelism": "single GPU", "variant": rs.info["variant"],
                   "launch": "eager" if args.eager else "hip-graph per step", "input_buffers": nbuf},
        "roofline": roofline,
        "last_step": {"maxvio": stats[0], "minvio": stats[1]},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(wl, W_np, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
