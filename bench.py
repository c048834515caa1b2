"""Benchmark of the ID Balancing router + controller step on one MI355X.

One step = the whole hot path over one batch: repacking the router matrix
into the MFMA operand layout (a training step changes it after every
optimizer update), then idb_router_step: the fused gate contraction +
sigmoid + biased Top-K (per expert slice), the slice merge with gate weights
and load counts, and in the merge's last workgroup MaxVio/MinVio and the ID
controller update.  Inputs are
synthetic, seeded, resident in HBM before the timed region; the hidden-state
batch rotates over several distinct buffers so it is not served from the
256 MB Infinity Cache.  Steps are issued as HIP graph replays, each graph
holding the ABI calls of several consecutive steps (one per input buffer), so
exactly ``--steps`` steps run in the timed region.

``--pmc-pass`` instead runs a short eager sequence for hardware-counter
collection: one device-to-device copy of known size (the calibration for the
HBM byte counters) followed by a few launches of the fused router kernel.

Prints one JSON line: routed tokens/s for the step, with the dominant
kernel's roofline, the unfused selection's HBM roofline (idb_select_from_scores
over the router's own fp32 scores, materialised for this measurement only) and
the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
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
# length of the spin kernel ahead of each timed block (torch.cuda._sleep
# cycles, about 0.4 ms): longer than the host needs to submit the first graph
PRE_SPIN_CYCLES = 960_000


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def load_traffic(workload: str, variant_id: int, family: str = "router"):
    """HBM bytes per launch of a counted kernel (router, merge, select) from the committed counter summary, or
    None if it is stale (kernel sources changed since) or absent."""
    from paper_2609_39137_amd.profsum import router_source_hash

    path = os.path.join(PROFILES, f"router_step_{workload}_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_sha256") != router_source_hash() or d.get("variant") != variant_id:
        return None
    return d.get("kernels", {}).get(family, {}).get("hbm_bytes_per_launch")


def load_kernel_trace_us(workload: str, family: str = "router"):
    """Average kernel duration (us) of a kernel family in the committed rocprofv3 kernel trace of this benchmark,
    or None if the trace is stale (kernel sources changed since) or absent."""
    from paper_2609_39137_amd.profsum import router_source_hash

    path = os.path.join(PROFILES, f"router_step_{workload}_kernel_stats.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_sha256") != router_source_hash():
        return None
    k = d.get("kernels", {}).get(family)
    return None if k is None else round(k["avg_us"], 2)


def cpu_baseline(wl, W, target_s: float):
    """Time the CPU oracle (router + controller + stats) on a bounded sample of the workload.

    The sample is a prefix of batch 0's tokens, grown until one oracle step
    takes about a second, then that step is repeated (the controller state
    carries over, as in training) until about ``target_s`` seconds of CPU
    work have been timed."""
    import oracle
    from paper_2609_39137_amd import synth

    threads = oracle.num_threads()
    n = 256
    while True:
        x = synth.hidden_states(wl, step=0, rows=np.arange(n))
        t = oracle.step_seconds(x, W, wl.K, 6e-3, 6e-3, oracle.ControllerState(wl.E))
        if t >= 0.5 or n >= wl.T:
            break
        n = min(wl.T, n * 4)
    reps = max(1, int(round(target_s / max(t, 1e-6))))
    st = oracle.ControllerState(wl.E)
    total = 0.0
    for _ in range(reps):
        total += oracle.step_seconds(x, W, wl.K, 6e-3, 6e-3, st)
    # one thread on 1024 tokens
    x1 = synth.hidden_states(wl, step=0, rows=np.arange(min(1024, wl.T)))
    oracle.set_num_threads(1)
    try:
        t1 = oracle.step_seconds(x1, W, wl.K, 6e-3, 6e-3, oracle.ControllerState(wl.E))
    finally:
        oracle.set_num_threads(threads)
    return {
        "value": n * reps / total,
        "unit": "routed tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{reps} oracle steps (router + ID update + MaxVio/MinVio, controller state carried over) on the "
                  f"first {n} of the {wl.T} tokens of batch 0 of {wl.name}: {total:.2f} s wall on {threads} "
                  f"OpenMP threads",
        "cpu_model": cpu_model(),
        "single_thread_value": round(len(x1) / t1, 1),
        "single_thread_sample": f"one oracle step on the first {len(x1)} tokens, one thread",
    }


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default=None, help="synthetic workload name (default: the Top-10-of-768 shape)")
    ap.add_argument("--variant", type=int, default=0, help="router tiling (0 = automatic)")
    ap.add_argument("--buffers", type=int, default=0, help="distinct hidden-state buffers to rotate (0 = auto)")
    ap.add_argument("--eager", action="store_true", help="launch the ABI calls directly instead of graph replays")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="eager copy calibration + a few router launches, for rocprofv3 counter passes")
    ap.add_argument("--copy-mib", type=int, default=512, help="size of the calibration copy of --pmc-pass")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--controller", choices=("id", "qb", "aux"), default="id",
                    help="id: ID Balancing (the headline step); qb: Quantile Balancing, the paper's baseline; "
                         "aux: auxiliary-loss balancing's forward statistics (softmax router, no bias)")
    ap.add_argument("--aux-alpha", type=float, default=0.05, help="auxiliary-loss coefficient")
    ap.add_argument("--aux-variant", type=int, default=0, help="one-slice router tiling of --controller aux")
    ap.add_argument("--rho", type=float, default=0.0, help="Quantile Balancing EMA weight (0: the plain target)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="wall-clock target of the CPU oracle sample")
    ap.add_argument("--loop", action="store_true",
                    help="run the workload's closed loop instead (its number of controller steps, fresh batch each "
                         "step) with the ID controller, integral-only and DeepSeek's rule side by side, and report "
                         "the load-balance trajectory")
    ap.add_argument("--loop-steps", type=int, default=0, help="steps of --loop (0: the workload's own)")
    ap.add_argument("--loop-md", default=None, help="also write a markdown summary of --loop to this path")
    ap.add_argument("--gen-workers", type=int, default=8, help="processes generating the --loop input batches")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported (the count all-reduce across "
              f"data-parallel ranks is not implemented: one GPU runs the whole path)", file=sys.stderr)
        return 2

    pool = None
    if args.loop:
        # the input-generating workers start before anything initialises the
        # GPU in this process
        import multiprocessing as mp

        pool = mp.get_context("spawn").Pool(max(1, args.gen_workers))

    import torch

    from paper_2609_39137_amd import binding as B
    from paper_2609_39137_amd import synth
    from paper_2609_39137_amd.pipeline import RouterStep

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = "cuda"
    wl = synth.WORKLOADS[args.workload or synth.HEADLINE]
    if args.loop:
        try:
            return loop_report(args, wl, pool)
        finally:
            pool.terminate()
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

    qb = args.controller == "qb"
    aux = args.controller == "aux"
    if aux:
        rs.aux_buffers(args.aux_variant)

    def one_step(i):
        rs.pack(W, stream=stream)
        if qb:
            rs.qb_step(xs[i % nbuf], None, rho=args.rho, stream=stream)
        elif aux:
            rs.aux_step(xs[i % nbuf], None, alpha=args.aux_alpha, stream=stream)
        else:
            rs.step(xs[i % nbuf], None, stream=stream)

    # eager warm-up (also validates every call)
    with torch.cuda.stream(stream):
        for i in range(2):
            one_step(i)
    torch.cuda.synchronize()

    if args.pmc_pass:
        # counter passes: the router's own scores of one batch for the unfused
        # select (dumped before the calibration copy, so its extra writes stay
        # out of the counted launches), then the copy of known size, then three
        # steps (router kernel + slice merge with the update) and three
        # selections from the dumped scores
        n_copy = args.copy_mib * 2**20
        scores = torch.empty((wl.T, wl.E), dtype=torch.float32, device=dev)
        sidx = torch.empty((wl.T, wl.K), dtype=torch.int32, device=dev)
        sw = torch.empty((wl.T, wl.K), dtype=torch.float32, device=dev)
        sc = torch.zeros(wl.E, dtype=torch.int32, device=dev)
        with torch.cuda.stream(stream):
            rs.route(xs[0], None, scores_dump=scores, stream=stream)
        src = torch.empty(n_copy, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            dst.copy_(src)
            for i in range(3):
                rs.score_select(xs[i % nbuf], None, stream=stream)
                rs.merge_step(stream=stream)
            for i in range(3):
                B.idb_select_from_scores(scores, rs.state.bias, wl.K, sidx, sw, sc, accumulate=True, stream=stream)
        torch.cuda.synchronize()
        print(json.dumps({"pmc_pass": True, "copy_bytes": n_copy, "workload": wl.name,
                          "variant": rs.info["variant"], "router_launches": 3, "merge_launches": 3,
                          "select_launches": 3}), flush=True)
        return 0

    def capture(fn, n):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(stream):
            with torch.cuda.graph(g, stream=stream):
                for i in range(n):
                    fn(i)
        return g

    graphs = {}

    def run_steps(n):
        """Issue exactly n steps: one replay of the n-step graph."""
        if n == 0:
            return
        if args.eager:
            with torch.cuda.stream(stream):
                for i in range(n):
                    one_step(i)
            return
        with torch.cuda.stream(stream):
            graphs[n].replay()

    # Each block of steps (the warm-up, the timed region, a spread block) is
    # one graph, captured and instantiated up front, so no host-side capture
    # runs while the GPU is being timed and no graph launch boundary falls
    # between the steps of a block; every graph is uploaded to the device
    # (hipGraphUpload) before the warm-up, so no first launch is timed and the
    # warm-up steps are the only untimed steps.
    if not args.eager:
        import ctypes

        hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch has loaded
        hip.hipGraphUpload.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        for n in sorted({args.warmup, args.steps, 100} - {0}):
            graphs[n] = capture(one_step, n)
            rc = hip.hipGraphUpload(ctypes.c_void_p(graphs[n].raw_cuda_graph_exec()),
                                    ctypes.c_void_p(stream.cuda_stream))
            if rc != 0:
                raise RuntimeError(f"hipGraphUpload of the {n}-step graph failed ({rc})")
        torch.cuda.synchronize()
    run_steps(args.warmup)
    torch.cuda.synchronize()
    log(f"warm-up of {args.warmup} steps done")

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)

    def timed_block(n):
        """Host-side wall time (s) to enqueue n steps; the GPU time lies between ev0 and ev1.
        A short spin kernel ahead of ev0 holds the stream while the host submits
        the first graph, so that submission's latency is not inside the timed
        region (later graphs are submitted while the earlier ones run)."""
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            torch.cuda._sleep(PRE_SPIN_CYCLES)
        ev0.record(stream)
        t0 = time.perf_counter()
        run_steps(n)
        t1 = time.perf_counter()
        ev1.record(stream)
        torch.cuda.synchronize()
        return t1 - t0

    host_s = timed_block(args.steps)
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / args.steps
    log(f"timed {args.steps} steps: {ms_step * 1000:.2f} us/step (host enqueue {host_s * 1e6:.0f} us)")
    # spread: 5 more timed blocks of 100 steps each (outside the timed region above)
    reps_us = []
    for _ in range(5):
        timed_block(100)
        reps_us.append(ev0.elapsed_time(ev1) * 1000 / 100)
    spread = {"blocks": 5, "steps_per_block": 100, "p10": round(float(np.percentile(reps_us, 10)), 2),
              "median": round(float(np.median(reps_us)), 2), "p90": round(float(np.percentile(reps_us, 90)), 2),
              "unit": "us/step"}

    # sanity of the last step's outputs
    counts = rs.counts.cpu()
    assert int(counts.sum()) == wl.T * wl.K, "counts do not sum to T*K"
    assert int(rs.state.status.item()) == 0
    stats = rs.stats.cpu().tolist()
    if qb:
        return qb_report(args, wl, rs, xs, nbuf, stream, capture, ms_step, stats, spread)
    if aux:
        return aux_report(args, wl, rs, xs, nbuf, stream, capture, ms_step, stats, spread)

    # live timing of the dominant kernel inside steps like the timed ones: the
    # same calls split at the kernel boundary (pack, the fused router kernel,
    # the slice merge with the update; idb_router_score_select_timed +
    # idb_router_merge_step enqueue exactly the kernels of idb_router_step),
    # each router launch writing its own start and end into a pair of HIP
    # events on the benchmark's stream
    k1_ms, k1_how = kernel_time_in_steps(args, rs, W, xs, nbuf, stream)
    log(f"fused router kernel: {k1_ms * 1000:.2f} us/launch ({k1_how})")

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
        "kernel": f"fused router kernel, variant {rs.info['variant']} ({rs.info['tokens_per_wg']} tokens x "
                  f"{rs.info['waves'] * rs.info['experts_per_wave']} experts per workgroup)",
        "kernel_us": round(k1_ms * 1000, 2),
        "kernel_timing": k1_how,
        "flops_per_launch": flops,
    }
    # the committed kernel trace of this command (the kernel's average over
    # every launch of that run), reported beside; frac above is from the live
    # events
    trace_us = load_kernel_trace_us(wl.name)
    roofline["kernel_trace_us"] = trace_us
    roofline["frac_kernel_trace"] = None if trace_us is None else round(flops / (trace_us * 1e-6) / 1e12 / peak, 4)
    # the unfused selection (scores given) over materialised fp32 scores, an
    # HBM-bound pass: the router's own scores of each input batch, dumped
    # once; timed in accumulate mode, so each call is exactly one launch of
    # the select kernel
    sel_bufs = max(2, min(8, math.ceil(512 * 2**20 / (wl.T * wl.E * 4))))
    scores = []
    for i in range(sel_bufs):
        buf = torch.empty((wl.T, wl.E), dtype=torch.float32, device=dev)
        with torch.cuda.stream(stream):
            rs.route(xs[i % nbuf], None, scores_dump=buf, stream=stream)
        scores.append(buf)
    sidx = torch.empty((wl.T, wl.K), dtype=torch.int32, device=dev)
    sw = torch.empty((wl.T, wl.K), dtype=torch.float32, device=dev)
    sc = torch.zeros(wl.E, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    sel_per = sel_bufs * max(1, 16 // sel_bufs)
    n_rep = max(1, -(-max(args.steps, 64) // sel_per))
    sel_graph = capture(lambda i: B.idb_select_from_scores(scores[i % sel_bufs], rs.state.bias, wl.K, sidx, sw, sc,
                                                           accumulate=True, stream=stream), sel_per)
    with torch.cuda.stream(stream):
        sel_graph.replay()
    torch.cuda.synchronize()
    ev0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(n_rep):
            sel_graph.replay()
    ev1.record(stream)
    torch.cuda.synchronize()
    sel_ms = ev0.elapsed_time(ev1) / (n_rep * sel_per)
    sel_bytes = wl.T * wl.E * 4 + wl.T * wl.K * 8 + 2 * wl.E * 4
    sel_gbs = sel_bytes / (sel_ms * 1e-3) / 1e9
    log(f"select from scores: {sel_ms * 1000:.2f} us/launch, {sel_gbs:.0f} GB/s")
    select_roofline = {
        "bound": "hbm",
        "achieved": round(sel_gbs, 1),
        "peak": PEAK_HBM_GBS,
        "unit": "GB/s",
        "frac": round(sel_gbs / PEAK_HBM_GBS, 4),
        "kernel": ("select_reg_kernel" if wl.K <= 10 and wl.E % 4 == 0 else "select_kernel")
                  + " (idb_select_from_scores, fp32 scores [T][E] read from HBM)",
        "kernel_us": round(sel_ms * 1000, 2),
        "bytes_per_launch": sel_bytes,
        "traffic": load_traffic(wl.name, rs.info["variant"], "select"),
    }
    # the paper's diagnostics on the same step: the full-pool and top-K
    # routing entropies over this batch (scores [T][E] read from HBM), and
    # the batched controller of a 21-layer model (one launch, one
    # workgroup per layer, with MaxVio/MinVio and the update's diagnostics)
    ent_ws = torch.empty(int(B.lib().idb_routing_entropy_workspace_bytes()), dtype=torch.uint8, device=dev)
    ent_out = torch.empty(2, dtype=torch.float64, device=dev)
    ent_ms = graph_time_per_call(lambda i: B.idb_routing_entropy(sw, ent_out, scores[i % sel_bufs], rs.state.bias,
                                                                 ent_ws, stream=stream), sel_per, n_rep, stream,
                                 capture)
    ent_bytes = wl.T * wl.E * 4 + wl.T * wl.K * 4 + wl.E * 4
    ent_gbs = ent_bytes / (ent_ms * 1e-3) / 1e9
    del scores
    n_layers = 21
    lay_counts = rs.counts.repeat(n_layers, 1).contiguous()
    lay_state = B.ControllerState(wl.E, dev, layers=n_layers)
    lay_stats = torch.empty((n_layers, 2), dtype=torch.float64, device=dev)
    lay_diag = torch.empty((n_layers, 4), dtype=torch.float64, device=dev)
    lay_ms = graph_time_per_call(lambda i: B.idb_controller_update_layers(lay_counts, rs.cfg, lay_state, lay_stats,
                                                                          lay_diag, stream=stream), 16, n_rep, stream,
                                 capture)
    log(f"routing entropies: {ent_ms * 1000:.2f} us ({ent_gbs:.0f} GB/s); {n_layers}-layer controller with "
        f"diagnostics: {lay_ms * 1000:.2f} us")
    diagnostics = {
        "routing_entropy": {"bound": "hbm", "achieved": round(ent_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                            "frac": round(ent_gbs / PEAK_HBM_GBS, 4), "kernel_us": round(ent_ms * 1000, 2),
                            "bytes_per_call": ent_bytes, "launches": 2},
        "layers_controller": {"layers": n_layers, "kernel_us": round(lay_ms * 1000, 2), "bound": "latency",
                              "outputs": "bias, e_prev, MaxVio/MinVio and four diagnostics per layer"},
    }

    value = wl.T / (ms_step * 1e-3)
    out = {
        "metric": f"routed tokens/sec for router+ID-update step, Top-{wl.K}-of-{wl.E}; % MFMA/HBM roofline",
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
                   "launch": "eager" if args.eager else "one hip-graph per block of steps", "input_buffers": nbuf,
                   "weight": "bf16 row-major, repacked every step" if wl.dtype == "bf16" else
                             "fp32 row-major, repacked every step"},
        "roofline": roofline,
        "select_roofline": select_roofline,
        "diagnostics": diagnostics,
        "step_spread": spread,
        "assignments_per_s": round(wl.T * wl.K / (ms_step * 1e-3), 1),
        "last_step": {"maxvio": stats[0], "minvio": stats[1]},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(wl, W_np, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


def kernel_time_in_steps(args, rs, W, xs, nbuf, stream):
    """Average duration of the fused router kernel over ``args.steps`` steps like the timed ones.

    Each step is pack + idb_router_score_select_timed + idb_router_merge_step
    (the kernels of idb_router_step): the router kernel is started by an
    extended launch that writes its own start and end timestamps into a pair
    of HIP events on the benchmark's stream, so each interval is that
    kernel's execution (no dispatch, no separately recorded events).  The
    steps are launched eagerly: on ROCm, events recorded inside a captured
    graph carry no timestamps (only external events would, and they are not
    available there).  All steps are enqueued while a spin kernel holds the
    stream, so they run back to back like the timed ones; nbuf untimed steps
    run first."""
    import torch

    n = max(args.steps, nbuf)
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for a, b in pairs:  # torch creates an event on its first record
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()

    def split_step(i, timed):
        rs.pack(W, stream=stream)
        rs.score_select(xs[i % nbuf], None, stream=stream, events=pairs[i] if timed else None)
        rs.merge_step(stream=stream)

    with torch.cuda.stream(stream):
        # a spin kernel holds the stream while the host enqueues every step, so
        # the steps then run back to back from the queue (the host launches
        # more slowly than the GPU runs them; without it the launch gaps would
        # fall inside the event pairs)
        torch.cuda._sleep(12_000_000)
        for i in range(nbuf):
            split_step(i, False)
        for i in range(n):
            split_step(i, True)
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in pairs) / n
    return ms, (f"HIP events taking each router kernel's own start and end (extended launch) in {n} steps "
                f"(pack, router, merge + update) enqueued behind a spin kernel and run back to back")


def _gen_batch(name: str, step: int) -> np.ndarray:
    """Hidden states of one loop step (run in a worker process)."""
    from paper_2609_39137_amd import synth

    return synth.hidden_states(synth.WORKLOADS[name], step=step)


def loop_report(args, wl, pool) -> int:
    """Closed loop of Alg. 1 on the GPU: ``steps`` iterations of idb_router_step, each on a fresh batch.

    Three controllers route the same batches side by side: ID Balancing
    (K_i = K_d = 6e-3, centred), its integral-only ablation (K_d = 0) and
    DeepSeek's rule (SIGN mode, 1e-3, no centring).  Each step records
    MaxVio/MinVio (from the step itself) and the update's diagnostics
    (active-gate fraction, busiest-10% share, inactive-expert ratio, mean
    |bias change|) from idb_controller_update_layers applied to a copy of the
    pre-step state with the step's counts; that copy's new bias must equal the
    step's bit for bit.  Batches are generated by worker processes in step
    order while the GPU runs."""
    import torch

    from paper_2609_39137_amd import binding as B
    from paper_2609_39137_amd import metrics
    from paper_2609_39137_amd import synth
    from paper_2609_39137_amd.pipeline import RouterStep

    dev = "cuda"
    steps = args.loop_steps or wl.steps
    tdtype = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    W_np = synth.router_weight(wl)
    W = torch.from_numpy(W_np.view(np.int16) if W_np.dtype == np.uint16 else W_np).to(dev)
    if W_np.dtype == np.uint16:
        W = W.view(torch.bfloat16)
    ctrls = {
        "id": B.ControllerCfg(wl.E, 6e-3, 6e-3, B.IDB_INTEGRAL_ERROR, True),
        "integral-only": B.ControllerCfg(wl.E, 6e-3, 0.0, B.IDB_INTEGRAL_ERROR, True),
        "deepseek-sign": B.ControllerCfg(wl.E, 1e-3, 0.0, B.IDB_INTEGRAL_SIGN, False),
    }
    runs = {}
    for name, cfg in ctrls.items():
        rs = RouterStep(wl.T, wl.d, wl.E, wl.K, tdtype, cfg, variant=args.variant)
        rs.pack(W)
        shadow = B.ControllerState(wl.E, dev, layers=1)
        runs[name] = {"rs": rs, "shadow": shadow, "stats": torch.empty((1, 2), dtype=torch.float64, device=dev),
                      "diag": torch.empty((1, 4), dtype=torch.float64, device=dev), "rec": metrics.LoadRecord(),
                      "diag_rows": [], "us": []}
    log(f"closed loop {wl.name}: {steps} steps, T={wl.T} d={wl.d} E={wl.E} K={wl.K}; controllers {list(ctrls)}")
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    workers = max(1, args.gen_workers)
    t_start = time.time()
    window = 2 * workers  # batches in flight (bounded host memory)
    futs = {t: pool.apply_async(_gen_batch, (wl.name, t)) for t in range(min(window, steps))}
    for t in range(steps):
        x_np = futs.pop(t).get()
        if t + window < steps:
            futs[t + window] = pool.apply_async(_gen_batch, (wl.name, t + window))
        x = torch.from_numpy(x_np.view(np.int16) if x_np.dtype == np.uint16 else x_np).to(dev)
        if x_np.dtype == np.uint16:
            x = x.view(torch.bfloat16)
        for name, r in runs.items():
            rs, sh = r["rs"], r["shadow"]
            sh.bias.copy_(rs.state.bias.view(1, -1))
            sh.e_prev.copy_(rs.state.e_prev.view(1, -1))
            sh.step.copy_(rs.state.step)
            sh.status.copy_(rs.state.status)
            ev0.record()
            rs.step(x, None)
            ev1.record()
            B.idb_controller_update_layers(rs.counts.view(1, -1), rs.cfg, sh, r["stats"], r["diag"])
            torch.cuda.synchronize()
            r["us"].append(ev0.elapsed_time(ev1) * 1000.0)
            if not torch.equal(sh.bias.view(-1).view(torch.int32), rs.state.bias.view(torch.int32)):
                raise RuntimeError(f"{name} step {t}: the one-call step and the layers kernel disagree")
            st = rs.stats.cpu().numpy()
            if not np.array_equal(st.view(np.int64), r["stats"].cpu().numpy().reshape(-1).view(np.int64)):
                raise RuntimeError(f"{name} step {t}: MaxVio/MinVio differ between the two kernels")
            r["rec"].add(st)
            r["diag_rows"].append(r["diag"].cpu().numpy().reshape(-1).copy())
            if wl.E <= 64:  # small pools: the per-expert trajectory too
                r.setdefault("counts", []).append(rs.counts.cpu().numpy().tolist())
                r.setdefault("bias", []).append([float(v) for v in rs.state.bias.cpu().numpy()])
        if t % 10 == 0 or t == steps - 1:
            mv = {n: round(float(r["rec"].maxvio[-1, 0]), 4) for n, r in runs.items()}
            log(f"step {t}: MaxVio {mv} ({time.time() - t_start:.1f} s)")
    out = {"metric": f"closed-loop load balance, Top-{wl.K}-of-{wl.E} ({wl.name}), {steps} controller steps",
           "workload": wl.name, "T": wl.T, "d": wl.d, "E": wl.E, "K": wl.K, "steps": steps, "data": "synthetic",
           "controllers": {}}
    for name, r in runs.items():
        diag = np.stack(r["diag_rows"])
        last = max(1, steps // 10)
        summ = r["rec"].summary(last=last)
        summ.update({
            "cumulative_excess_above_1": r["rec"].cumulative_excess(1.0),
            "gate_fraction_first10_mean": float(np.nanmean(diag[1:11, 0])) if steps > 1 else None,
            "gate_fraction_last10pct_mean": float(np.nanmean(diag[-last:, 0])),
            "busiest10_share_last10pct_mean": float(np.mean(diag[-last:, 1])),
            "inactive_ratio_last10pct_mean": float(np.mean(diag[-last:, 2])),
            "step_us_median": float(np.median(r["us"])),
            "last_window_steps": last,
            "cfg": {"Ki": r["rs"].cfg.Ki, "Kd": r["rs"].cfg.Kd, "mode": r["rs"].cfg.integral_mode,
                    "center": bool(r["rs"].cfg.center)},
            "maxvio": [round(float(v), 6) for v in r["rec"].maxvio[:, 0]],
            "minvio": [round(float(v), 6) for v in r["rec"].minvio[:, 0]],
            "gate_fraction": [round(float(v), 6) for v in diag[:, 0]],
            "busiest10_share": [round(float(v), 6) for v in diag[:, 1]],
        })
        if "counts" in r:
            summ["counts"] = r["counts"]
            summ["bias_after_step"] = r["bias"]
        out["controllers"][name] = summ
    if args.loop_md:
        with open(args.loop_md, "w") as f:
            f.write(loop_markdown(out, sys.argv))
    print(json.dumps(out), flush=True)
    return 0


def loop_markdown(out: dict, argv) -> str:
    """Markdown summary of a --loop run: per-controller aggregates, then the per-step trajectory."""
    c = out["controllers"]
    names = list(c)
    last = c[names[0]]["last_window_steps"]
    lines = [f"# Closed loop, {out['workload']} (T={out['T']}, d={out['d']}, E={out['E']}, K={out['K']}), "
             f"{out['steps']} steps", "", "Command:", "", "```", "python " + " ".join(argv), "```", "",
             "Each step: a fresh synthetic batch routed by idb_router_step with the controller's current bias "
             "(the fused router kernel, then the slice merge with the update and MaxVio/MinVio in its last "
             "workgroup, or the controller step when one slice covers all experts). "
             "Diagnostics from idb_controller_update_layers on a copy of the pre-step state (its bias equals the "
             "step's bit for bit, checked every step).", "",
             f"| controller | K_i | K_d | mode | centre | MaxVio last {last} | MaxVio avg | MaxVio worst | "
             f"MinVio last {last} | MinVio avg | excess above 1 | gate frac. steps 1-10 | gate frac. last {last} | "
             f"busiest-10% share last {last} | step us (median) |",
             "|---|---:|---:|---|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for n in names:
        s = c[n]
        mode = "sign" if s["cfg"]["mode"] == 1 else "error"
        lines.append(f"| {n} | {s['cfg']['Ki']:g} | {s['cfg']['Kd']:g} | {mode} | {s['cfg']['center']} | "
                     f"{s['maxvio_last']:.4f} | {s['maxvio_avg']:.4f} | {s['maxvio_worst']:.4f} | "
                     f"{s['minvio_last']:.4f} | {s['minvio_avg']:.4f} | {s['cumulative_excess_above_1']:.2f} | "
                     f"{s['gate_fraction_first10_mean']:.4f} | {s['gate_fraction_last10pct_mean']:.4f} | "
                     f"{s['busiest10_share_last10pct_mean']:.4f} | {s['step_us_median']:.1f} |")
    lines += ["", "Per step (MaxVio, MinVio, active-gate fraction, busiest-10% share):", "",
              "| step | " + " | ".join(f"{n} MaxVio | {n} MinVio" for n in names) + " | id gate frac. | "
              "id busiest-10% |", "|---:|" + "---:|" * (2 * len(names) + 2)]
    for t in range(out["steps"]):
        cells = []
        for n in names:
            cells += [f"{c[n]['maxvio'][t]:.4f}", f"{c[n]['minvio'][t]:.4f}"]
        lines.append(f"| {t} | " + " | ".join(cells) + f" | {c['id']['gate_fraction'][t]:.4f} | "
                     f"{c['id']['busiest10_share'][t]:.4f} |")
    if "counts" in c["id"]:
        E = out["E"]
        lines += ["", "ID Balancing, per step: the counts n_i (experts 0..E-1), then the bias b_i after the step's "
                  "update (fp32, 9 significant digits):", ""]
        for t in range(out["steps"]):
            lines.append(f"- step {t} counts: " + " ".join(str(v) for v in c["id"]["counts"][t]))
            lines.append(f"- step {t} bias: " + " ".join(f"{v:.9g}" for v in c["id"]["bias_after_step"][t]))
    return "\n".join(lines) + "\n"


def graph_time_per_call(fn, per, reps, stream, capture):
    """Average duration of fn on the stream: graph replays of per calls, reps times, between HIP events."""
    import torch

    g = capture(fn, per)
    with torch.cuda.stream(stream):
        g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    with torch.cuda.stream(stream):
        for _ in range(reps):
            g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / (reps * per)


def aux_report(args, wl, rs, xs, nbuf, stream, capture, ms_step, stats, spread) -> int:
    """JSON line of the auxiliary-loss statistics step (softmax router + f, P, loss; MaxVio/MinVio)."""
    from paper_2609_39137_amd import binding as B

    per = nbuf * max(1, 16 // nbuf)
    reps = max(1, -(-max(args.steps, 64) // per))

    def aux_call(i):
        B.idb_aux_router_forward(xs[i % nbuf], rs.W_packed, wl.K, args.aux_alpha, rs.idx, rs.w, rs.counts, rs.aux_f,
                                 rs.aux_P, rs.aux_loss, rs.aux_workspace, None, rs.aux_variant, stream,
                                 B.IDB_WEIGHT_PACKED, stats=rs.stats)

    route_ms = graph_time_per_call(aux_call, per, reps, stream, capture)
    info = B.idb_router_variant_info(wl.T, wl.d, wl.E, wl.K, rs.dtype_code, rs.aux_variant) if rs.aux_variant \
        else None
    log(f"softmax router + auxiliary-loss statistics: {route_ms * 1000:.2f} us per call")
    achieved = wl.flops / (route_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    loss = float(rs.aux_loss.item())
    out = {
        "metric": "routed tokens/sec for the auxiliary-loss router step (softmax Top-K, f_i, P_i, loss; the paper's "
                  "baseline, forward statistics)",
        "value": round(wl.T / (ms_step * 1e-3), 1),
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
                   "parallelism": "single GPU", "variant": info["variant"] if info else "auto (one slice)",
                   "controller": "auxiliary-loss statistics", "alpha": args.aux_alpha,
                   "launch": "one hip-graph per block of steps", "input_buffers": nbuf},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None,
                     "kernel": "fused router kernel in softmax mode (one slice of all experts, per-tile softmax "
                               "column sums) + the statistics kernel",
                     "kernel_us": round(route_ms * 1000, 2), "flops_per_launch": wl.flops},
        "last_step": {"maxvio": stats[0], "minvio": stats[1], "aux_loss": loss},
        "step_spread": spread,
    }
    print(json.dumps(out), flush=True)
    return 0


def qb_report(args, wl, rs, xs, nbuf, stream, capture, ms_step, stats, spread) -> int:
    """JSON line of the Quantile Balancing step (router in its QB mode, MaxVio/MinVio, the update)."""
    import torch

    from paper_2609_39137_amd import binding as B

    def time_per_call(fn, per, reps):
        g = capture(fn, per)
        with torch.cuda.stream(stream):
            g.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        with torch.cuda.stream(stream):
            for _ in range(reps):
                g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (reps * per)

    per = nbuf * max(1, 16 // nbuf)
    reps = max(1, -(-max(args.steps, 64) // per))
    route_ms = time_per_call(lambda i: rs.qb_route(xs[i % nbuf], None, stream=stream), per, reps)
    upd_ms = time_per_call(lambda i: B.idb_qb_update(rs.scores_t, rs.alpha, wl.K, args.rho, rs.state.bias, stream,
                                                     counts=rs.counts, stats=rs.stats), per, reps)
    log(f"router in QB mode (fused kernel + slice merge): {route_ms * 1000:.2f} us; update {upd_ms * 1000:.2f} us")
    achieved = wl.flops / (route_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    upd_bytes = wl.E * wl.T * 4 + wl.T * 4 + 3 * wl.E * 4 + 16
    upd_gbs = upd_bytes / (upd_ms * 1e-3) / 1e9
    out = {
        "metric": "routed tokens/sec for router + Quantile Balancing step (the paper's baseline controller)",
        "value": round(wl.T / (ms_step * 1e-3), 1),
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
                   "parallelism": "single GPU", "variant": rs.info["variant"], "controller": "quantile-balancing",
                   "rho": args.rho, "launch": "one hip-graph per block of steps", "input_buffers": nbuf},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None,
                     "kernel": "router in Quantile Balancing mode: fused kernel (K+1 candidates, expert-major "
                               "scores written) + slice merge",
                     "kernel_us": round(route_ms * 1000, 2), "flops_per_launch": wl.flops},
        "qb_update_roofline": {"bound": "hbm", "achieved": round(upd_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                               "frac": round(upd_gbs / PEAK_HBM_GBS, 4),
                               "kernel": "qb_update_reg_kernel (MaxVio/MinVio in its first workgroup)",
                               "kernel_us": round(upd_ms * 1000, 2), "bytes_per_launch": upd_bytes},
        "last_step": {"maxvio": stats[0], "minvio": stats[1]},
        "step_spread": spread,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
