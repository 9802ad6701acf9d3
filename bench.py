#!/usr/bin/env python3
"""SBVR GEMV benchmark on one MI355X.

A step is one decoder layer's seven SBVR GEMVs (q, k, v, o, gate, up, down)
at batch 1 with 4-bit SBVR weights (k = 4 planes, 128-weight groups, fp16
coefficients), fp16 activations and outputs, in the Llama-3-8B projection
shapes (Llama-3-70B with --model llama3-70b).  Steps cycle through L
independent layers of weights so the rotated working set (~1.9 GiB) exceeds
every cache and the bytes really come from HBM.  Each layer's seven calls
are captured in one HIP graph, as decode steps are served.

Weights are drawn directly in SBVR form (uniform bit planes, Gaussian fp16
coefficients, seeded): GEMV time does not depend on the values.  The parity
tests run these same shapes and launch configurations against the CPU oracle.

One JSON line is printed:
  value         aggregate algorithmic HBM throughput (GB/s) of the timed steps
  per_call_us   mean duration of each projection's launch, from HIP events
                around a graph of L back-to-back launches of that shape (one
                per layer) on the launch stream
  roofline      the dominant kernel instance (largest time per step):
                algorithmic bytes per launch / its mean launch duration, vs the
                8 TB/s HBM peak
  cpu_baseline  the CPU oracle (binary64 decompress + GEMV) on layer 0's seven
                GEMVs, bounded to ~10 s of work, in the same unit
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_GBPS = 8000.0
PROJ_ORDER = ("q", "k", "v", "o", "gate", "up", "down")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--model", choices=("llama3-8b", "llama3-70b"), default="llama3-8b")
    ap.add_argument("--layers", type=int, default=0, help="distinct weight sets (0: ~1.9 GiB)")
    ap.add_argument("--k", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    return ap.parse_args()


def b1_kernel_instance(O: int, k: int) -> str:
    """Name of the batch-1 kernel instance a launch with O rows runs: the
    library takes T tiles (4T rows) per workgroup, the most of 8/4/2/1 that
    still leaves >= 256 workgroups."""
    n_tiles = (O + 3) // 4
    T = next((t for t in (8, 4, 2) if n_tiles // t >= 256), 1)
    return f"gemv_b1_kernel<{k}, {T}>"


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the SBVR GEMV path "
              "has no multi-GPU mode.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2509_18172_amd as sb
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    shapes = synth.LLAMA8B if args.model == "llama3-8b" else synth.LLAMA70B
    k = args.k
    nbytes = {n: sb.algorithmic_bytes(*shapes[n], k) for n in PROJ_ORDER}
    layer_bytes = sum(nbytes.values())
    L = args.layers or max(2, int(np.ceil(1.9 * 2 ** 30 / layer_bytes)))
    cfg_index = 1 if args.model == "llama3-8b" else 3

    # ---- weights: L layers x 7 projections, packed into the device format ----
    host_layer0 = {}
    layers = []
    for li in range(L):
        lay = {}
        for pi, name in enumerate(PROJ_ORDER):
            O, I = shapes[name]
            seed = synth.seed_for(cfg_index, li, pi)
            planes, coeffs = synth.random_sbvr(O, I, k, seed=seed)
            if li == 0:
                host_layer0[name] = (planes, coeffs)
            W = sb.pack(torch.from_numpy(planes.view(np.int32)).to(dev),
                        torch.from_numpy(coeffs.view(np.int16)).to(dev))
            x = torch.from_numpy(synth.activations(I, seed=seed + synth.X_SEED_OFFSET)).to(dev)
            y = torch.empty(O, dtype=torch.float16, device=dev)
            lay[name] = (W, x, y)
        layers.append(lay)
        torch.cuda.synchronize()

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for name in PROJ_ORDER:  # eager warm-up of every shape before capture
            W, x, y = layers[0][name]
            sb.gemv(W, x, out=y, stream=stream)
    torch.cuda.synchronize()

    def capture(calls):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for W, x, y in calls:
                sb.gemv(W, x, out=y, stream=stream)
        return g

    def timed_replays(graphs, n):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            e0.record(stream)
            for i in range(n):
                graphs[i % len(graphs)].replay()
            e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)  # ms

    # ---- timed region: K steps, one layer graph per step ----
    step_graphs = [capture([layers[li][n] for n in PROJ_ORDER]) for li in range(L)]
    torch.cuda.synchronize()
    if args.warmup:
        timed_replays(step_graphs, args.warmup)
    total_ms = timed_replays(step_graphs, args.steps)
    ms_per_step = total_ms / args.steps
    value = layer_bytes * args.steps / (total_ms * 1e-3) / 1e9

    # ---- per-shape launch durations: L back-to-back launches per graph ----
    per_call_us = {}
    for name in PROJ_ORDER:
        g = capture([layers[li][name] for li in range(L)])
        timed_replays([g], 1)
        reps = [timed_replays([g], 1) * 1e3 / L for _ in range(3)]
        per_call_us[name] = float(np.median(reps))
        del g
    per_call_gbps = {n: nbytes[n] / (per_call_us[n] * 1e3) for n in PROJ_ORDER}

    # dominant kernel instance: largest launch time per step
    by_kernel = {}
    for n in PROJ_ORDER:
        kname = b1_kernel_instance(shapes[n][0], k)
        t, b, c = by_kernel.get(kname, (0.0, 0, 0))
        by_kernel[kname] = (t + per_call_us[n], b + nbytes[n], c + 1)
    dom = max(by_kernel, key=lambda kk: by_kernel[kk][0])
    dt, db, dc = by_kernel[dom]
    achieved = db / (dt * 1e3)  # (bytes per launch) / (mean launch duration), GB/s
    roofline = {
        "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_GBPS, "unit": "GB/s",
        "frac": round(achieved / PEAK_GBPS, 4), "traffic": None,
        "kernel": dom,
        "launches_per_step": dc,
        "projections": [n for n in PROJ_ORDER if b1_kernel_instance(shapes[n][0], k) == dom],
        "bytes_per_launch": round(db / dc),
        "mean_launch_us": round(dt / dc, 3),
    }

    # ---- CPU baseline: the oracle on layer 0, bounded ----
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        done_bytes, elapsed, passes, threads = 0, 0.0, 0, 0
        while elapsed < args.cpu_seconds or passes == 0:
            for name in PROJ_ORDER:
                planes, coeffs = host_layer0[name]
                x = layers[0][name][1].cpu().numpy()
                ts = time.perf_counter()
                _, threads = oracle.sbvr_gemv(planes, coeffs, x, return_threads=True)
                elapsed += time.perf_counter() - ts
                done_bytes += nbytes[name]
            passes += 1
        cpu = {"value": round(done_bytes / elapsed / 1e9, 4), "unit": "GB/s", "cores": threads,
               "kind": "oracle",
               "sample": f"{passes} pass(es) over layer 0's seven GEMVs ({args.model}, k={k}, batch 1): "
                         f"{elapsed:.1f} s of binary64 decompress + GEMV on {threads} threads "
                         f"({os.cpu_count()} host CPUs, {platform.machine()})"}

    out = {
        "metric": "SBVR GEMV us/call and achieved HBM GB/s (% of MI355X peak), 4-bit, batch 1",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 in/out, f32 accumulate",
        "data": "synthetic: seeded SBVR planes and fp16 coefficients, N(0,1) fp16 activations",
        "config": {
            "workload": f"{args.model} decode-layer projections q,k,v,o,gate,up,down; SBVR k={k}, "
                        f"group 128, batch 1; {L} rotating layers; one hipGraph per layer",
            "bytes_per_step": layer_bytes,
            "layers_rotated": L,
            "shapes": {n: list(shapes[n]) for n in PROJ_ORDER},
        },
        "pct_of_peak": round(100 * value / PEAK_GBPS, 2),
        "per_call_us": {n: round(v, 3) for n, v in per_call_us.items()},
        "per_call_gbps": {n: round(v, 1) for n, v in per_call_gbps.items()},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
