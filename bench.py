#!/usr/bin/env python3
"""SBVR GEMV benchmark on one MI355X.

A step is one decoder layer's seven SBVR GEMVs (q, k, v, o, gate, up, down)
at batch 1 with 4-bit SBVR weights (k = 4 planes, 128-weight groups, fp16
coefficients), fp16 activations and outputs, in the Llama-3-8B projection
shapes (Llama-3-70B with --model llama3-70b).  The weights of L = 32 decoder
layers (3.93 GB at 4 bits, more than every cache) are resident in HBM; the
timed region is one replay of a HIP graph of exactly K layer-steps on one
stream, step i running layer i mod L's seven GEMVs, after one replay of a
W-step warm-up graph and three untimed replays of the timed graph -- so
ms_per_step does not depend on how K relates to L.

Weights are drawn directly in SBVR form (uniform bit planes, Gaussian fp16
coefficients, seeded): GEMV time does not depend on the values.  The parity
tests run these same shapes and launch configurations against the CPU oracle
(and the configurations' own encoded weights).

One JSON line is printed:
  value         aggregate algorithmic HBM throughput (GB/s) of the timed steps
  decode_step   the L-layer graph alone: microseconds per token (median and
                mean of 50 replays), GB/s
  per_call_events  per projection: median and mean of 200 single launches,
                each between its own pair of events (after 20 warm-up calls)
  decode_step_w4a8  the same graph with SBVR-8 activations (sbvr_gemv_a8)
  decode_step_fused the same weights with q|k|v and gate|up packed as one
                matrix each (rows concatenated), 4 GEMVs per layer
  decode_step_grouped the 224 GEMVs on the separate weights, q, k, v and
                gate, up each enqueued as one grouped launch
                (sbvr_gemv_grouped): 4 launches per layer; w4a8_*: the same
                with SBVR-8 activations (sbvr_gemv_grouped_a8)
  per_call_us   mean duration of each projection's launch, from HIP events
                around a graph of 64 back-to-back launches of that shape
                cycling through >= 1 GB of distinct weight copies (median
                of 11 replays after 2 warm-up replays)
  roofline      the dominant kernel instance (largest time per step):
                algorithmic bytes per launch / its mean launch duration, vs the
                8 TB/s HBM peak.  The launch duration is what the launch adds
                to the timed graph: the K-step graph minus the same graph
                without that projection's launches, per launch
                (step_launch_us: the same for every projection);
                traffic = calibrated FETCH_SIZE + WRITE_SIZE
                bytes per launch from the recorded counter runs, when they were
                taken on the current kernel sources (else null);
                mean_launch_interval_us = the per_call_us of its projections;
                practical_peak = a plain streaming read of the same bytes per
                launch, timed like per_call_us (frac = its time / the interval)
  headline_spread  five more replays of the timed graph (ms per step)
  small_batch   per projection at B = 2, 4, 8 activation vectors
                (sbvr_gemm_small_batch), same timing
  w4a8          per projection, batch 1 with the activations converted online
                to 8-bit SBVR codes (sbvr_gemv_a8), same timing
  indexed       per projection in the coefficient-cache format (one 16-bit
                coefficient-set index per group, a table of one set per ten
                groups): us and GB/s of its own algorithmic bytes, with fp16
                (sbvr_gemv_indexed) and SBVR-8 activations (sbvr_gemv_indexed_a8)
  low_bit       per projection at k = 2 and 3 planes, same timing
  prefill       per projection: sbvr_decompress to binary16 (us, GB/s of the
                SBVR bytes read plus the 2 bytes per weight written), a 64- and
                a 512-token library GEMM (torch linear) on the result, and the
                fused prefill GEMM on the SBVR weights (sbvr_gemm_prefill) at
                1, 16, 64, 128 and 512 tokens
  llama3_70b    per projection of the Llama-3-70B shapes, same timing
  encoder       sbvr_encode (Algorithm 1 on the GPU, the 1024-entry grid) on an
                fp32 q/o-shaped matrix: seconds and groups per second, and the
                CPU oracle's encoder on a sample of its rows; `cached`: the
                same with the encoder cache of Sec. 4.2 (sbvr_encode_cached, 64
                sets per row): time, hit rate, mean error over the exhaustive
                search's, distinct coefficient sets with and without it
  cpu_baseline  the CPU oracle (binary64 decompress + GEMV) on layer 0's seven
                GEMVs, bounded to ~10 s of work, in the same unit, on all host
                threads; one_core: the same oracle on one thread over the q
                projection (~2.5 s); cpu_model from /proc/cpuinfo

--headline-only stops after the timed steps, the event-timed replica and the
decode step (the command whose rocprofv3 kernel statistics are compared with
roofline.mean_launch_us); --kernel-summary TRACE_CSV prints per-kernel
duration statistics of a rocprofv3 kernel trace.

--traffic-probe runs, eagerly, four launches of every projection shape (fp16
and W4A8 activations, the grouped q|k|v and gate|up launches, small batch
B = 8, the coefficient-cache format, and the prefill decompression to
binary16) and an elementwise
negation over 256 MiB of float32 (reads and writes 256 MiB: the counter
calibration), for
  rocprofv3 --pmc FETCH_SIZE -- python3 bench.py --traffic-probe   (and WRITE_SIZE);
--traffic-summary FETCH_CSV WRITE_CSV turns the two counter files into the
record kept under profiles/; --counter-summary A_CSV B_CSV does the same for
two instruction/cycle counter passes over the probe (the pass lists are in
counter_summary's docstring).

--prefill-probe runs, eagerly, sbvr_decompress, the library GEMM on its
result and the fused sbvr_gemm_prefill on every distinct Llama-3-8B shape at
each prompt length, separated by marker fills, for
  rocprofv3 --kernel-trace -- python3 bench.py --prefill-probe;
--prefill-summary TRACE_CSV turns the trace into the record kept under
profiles/.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import platform
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_GBPS = 8000.0
PROJ_ORDER = ("q", "k", "v", "o", "gate", "up", "down")
PREFILL_TOKENS = (1, 16, 64, 128, 256, 512)  # prompt lengths of the fused prefill GEMM timings
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "hbm_traffic_llama3-8b_k4.md")
ROCPROF_RECORD = "sbvr_gemv_llama3-8b_headline_kernel_stats.md"
CALIB_BYTES = 256 << 20
DECODE_REPLAYS = 50   # replays of the L-layer decode graph
EVENT_WARMUP, EVENT_CALLS = 20, 200  # per-call event timing
PROBE_LAUNCHES = 4
PREFILL_PROBE_CALLS = 16  # launches per phase of --prefill-probe


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--model", choices=("llama3-8b", "llama3-70b"), default="llama3-8b")
    ap.add_argument("--layers", type=int, default=0, help="decoder layers in the decode-step graph (0: 32)")
    ap.add_argument("--quick", action="store_true", help="skip the small-batch, k = 2/3 and other-model tables")
    ap.add_argument("--headline-only", action="store_true",
                    help="only the timed steps, the dominant kernel's event-timed launches and the decode step "
                         "(the run whose kernel statistics are compared with the headline)")
    ap.add_argument("--kernel-summary", nargs="+", metavar="PATH",
                    help="KERNEL_TRACE_CSV [BENCH_JSON]: print per-dispatch duration statistics from a rocprofv3 "
                         "kernel trace (with the traced run's own JSON line: its per-launch times) and exit")
    ap.add_argument("--k", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--traffic-probe", action="store_true",
                    help="eager launches of every shape plus a calibration copy, for counter runs")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="summarise two rocprofv3 --pmc counter files (no GPU needed)")
    ap.add_argument("--counter-summary", nargs=2, metavar=("PASS_A_CSV", "PASS_B_CSV"),
                    help="instruction and cycle counters per SBVR kernel from two rocprofv3 --pmc passes over "
                         "--traffic-probe (no GPU needed)")
    ap.add_argument("--prefill-probe", action="store_true",
                    help="eager prefill launches (decompress, library GEMM, fused GEMM) per shape and prompt "
                         "length, separated by marker fills, for a rocprofv3 kernel trace")
    ap.add_argument("--prefill-summary", metavar="KERNEL_TRACE_CSV",
                    help="per-kernel durations of a --prefill-probe kernel trace (no GPU needed)")
    return ap.parse_args()


# The sources the batch-1 kernels (code and launch shapes) are compiled from.
B1_KERNEL_SOURCES = ("device_ops.h", "gemv_b1.hip", "gemv_b1s.hip", "layout.h")


def kernel_source_digest() -> str:
    """sha256 over the sources of the batch-1 kernels: identifies the kernels a
    counter record was taken on."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2509_18172_amd", "csrc")
    for name in B1_KERNEL_SOURCES:
        h.update(name.encode())
        with open(os.path.join(csrc, name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def short_kernel_name(full: str) -> str:
    m = re.search(r"sbvr::(\w+_kernel<[^>]*>)", full) or re.search(r"sbvr::(\w+)\(", full)
    return m.group(1) if m else full


def read_counter_csv(path: str, counter: str):
    """{kernel name: [per-dispatch value of `counter`]} from a rocprofv3
    counter-collection CSV."""
    out = {}
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] == counter:
                out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return out


def read_counter_by_grid(path: str, counter: str):
    """{(kernel instance, grid threads): [per-dispatch value of `counter`]}
    for the SBVR kernels, plus the calibration copy under ("neg", 0)."""
    out = {}
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            key = ("neg", 0) if "neg_kernel" in name else (short_kernel_name(name), int(r["Grid_Size"]))
            if key[0] == "neg" or "sbvr::" in name:
                out.setdefault(key, []).append(float(r["Counter_Value"]))
    return out


def traffic_summary(fetch_csv: str, write_csv: str) -> str:
    """The profiles/ record: per-launch FETCH_SIZE and WRITE_SIZE of every GEMV
    kernel (per kernel instance and grid), scaled by what the same counters
    read for a copy of known size.  An instance launched with one grid only is
    keyed by its name, else by "name grid G"."""
    import numpy as np
    fetch, write = read_counter_by_grid(fetch_csv, "FETCH_SIZE"), read_counter_by_grid(write_csv, "WRITE_SIZE")
    copy = ("neg", 0)
    # KiB per dispatch; the copy reads and writes CALIB_BYTES
    f_scale = CALIB_BYTES / (np.median(fetch[copy]) * 1024)
    w_scale = CALIB_BYTES / (np.median(write[copy]) * 1024)
    rec = {"source_sha256": kernel_source_digest(), "calibration": {
        "copy_bytes": CALIB_BYTES, "fetch_kib": float(np.median(fetch[copy])),
        "write_kib": float(np.median(write[copy])), "fetch_scale": f_scale, "write_scale": w_scale},
        "kernels": {}}
    grids = {}
    for name, grid in fetch:
        grids.setdefault(name, set()).add(grid)
    lines = ["| kernel | grid | dispatches | FETCH_SIZE KiB (median) | WRITE_SIZE KiB | calibrated bytes / launch |",
             "|---|---:|---:|---:|---:|---:|"]
    for (name, grid) in sorted(k for k in fetch if k != copy):
        if "gemv_b1" not in name and "gemm_sbs" not in name:
            continue
        # one launch configuration can serve two shapes (same grid): split
        # its dispatches where the sorted FETCH_SIZE values jump by > 25 %
        vals = sorted(fetch[(name, grid)])
        clusters = [[vals[0]]]
        for v in vals[1:]:
            (clusters[-1] if v <= clusters[-1][-1] * 1.25 else clusters.append([]) or clusters[-1]).append(v)
        wk = float(np.median(write.get((name, grid), [0.0])))
        for ci, cl in enumerate(clusters):
            fk = float(np.median(cl))
            nbytes = round(fk * 1024 * f_scale + wk * 1024 * w_scale)
            key = name if len(grids[name]) == 1 else f"{name} grid {grid}"
            if len(clusters) > 1:
                key += f" size {ci + 1} of {len(clusters)}"
            rec["kernels"][key] = {"dispatches": len(cl), "fetch_kib": fk, "write_kib": wk,
                                   "grid": grid, "bytes_per_launch": nbytes}
            lines.append(f"| `{name}` | {grid} | {len(cl)} | {fk:.1f} | {wk:.1f} | {nbytes:,} |")
    lines += ["", "traffic-record: " + json.dumps(rec, sort_keys=True)]
    return "\n".join(lines)


def read_counters(path: str):
    """{(kernel instance, grid): {"dispatches": [{counter: value}, ...] in
    dispatch order, "vgpr", "agpr"}} for the SBVR kernels of a rocprofv3
    counter CSV."""
    out = {}
    with open(path) as fh:
        rows = sorted(csv.DictReader(fh), key=lambda r: int(r["Dispatch_Id"]))
    for r in rows:
        if "sbvr::" not in r["Kernel_Name"]:
            continue
        key = (short_kernel_name(r["Kernel_Name"]), int(r["Grid_Size"]))
        e = out.setdefault(key, {"ids": {}, "vgpr": int(r["VGPR_Count"]), "agpr": int(r["Accum_VGPR_Count"])})
        e["ids"].setdefault(int(r["Dispatch_Id"]), {})[r["Counter_Name"]] = float(r["Counter_Value"])
    for e in out.values():
        e["dispatches"] = [e["ids"][i] for i in sorted(e["ids"])]
        del e["ids"]
    return out


def counter_summary(a_csv: str, b_csv: str) -> str:
    """Markdown table of two rocprofv3 --pmc passes over --traffic-probe:
    pass A with SQ_WAVES SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_LDS
    SQ_INSTS_VMEM_RD SQ_INSTS_SALU SQ_BUSY_CYCLES SQ_WAVE_CYCLES, pass B with
    SQ_ACTIVE_INST_VALU SQ_VALU_MFMA_BUSY_CYCLES SQ_WAIT_INST_ANY
    SQ_ACTIVE_INST_ANY SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE.  Medians over the
    dispatches of each (kernel instance, grid); a launch configuration that
    serves two shapes is split where its per-dispatch VALU count jumps by
    more than 25 % (the two passes run the same probe, so the k-th dispatch
    of an instance is the same launch in both).  Instruction counts per
    wavefront; cycle counters per wavefront as the counters report them."""
    import numpy as np
    A, Bp = read_counters(a_csv), read_counters(b_csv)
    lines = ["| kernel | grid | VGPR (rocprof) | waves | VALU / wave | MFMA / wave | LDS / wave | "
             "VMEM rd / wave | SALU / wave | MFMA busy / MFMA | active VALU / wave | active any / wave | "
             "wait any / wave | wave cycles / wave | LDS conflicts / CU |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    rec = {"source_sha256": kernel_source_digest(), "kernels": {}}
    for (kname, grid), e in sorted(A.items()):
        da = e["dispatches"]
        db = Bp.get((kname, grid), {"dispatches": []})["dispatches"]
        order = sorted(range(len(da)), key=lambda i: da[i].get("SQ_INSTS_VALU", 0.0))
        clusters = [[order[0]]]
        for i in order[1:]:
            prev = da[clusters[-1][-1]].get("SQ_INSTS_VALU", 0.0)
            if da[i].get("SQ_INSTS_VALU", 0.0) > prev * 1.25:
                clusters.append([])
            clusters[-1].append(i)
        for ci, idx in enumerate(clusters):
            def med(rows, n):
                v = [rows[i][n] for i in idx if i < len(rows) and n in rows[i]]
                return float(np.median(v)) if v else float("nan")
            w = med(da, "SQ_WAVES")
            if not w > 0:
                continue
            nm = med(da, "SQ_INSTS_MFMA")
            row = {"vgpr": e["vgpr"], "agpr": e["agpr"], "waves": w, "dispatches": len(idx),
                   "valu": med(da, "SQ_INSTS_VALU") / w, "mfma": nm / w, "lds_insts": med(da, "SQ_INSTS_LDS") / w,
                   "vmem": med(da, "SQ_INSTS_VMEM_RD") / w, "salu": med(da, "SQ_INSTS_SALU") / w,
                   "mfma_busy_per_inst": med(db, "SQ_VALU_MFMA_BUSY_CYCLES") / nm if nm else 0.0,
                   "active_valu": med(db, "SQ_ACTIVE_INST_VALU") / w, "active_any": med(db, "SQ_ACTIVE_INST_ANY") / w,
                   "wait_any": med(db, "SQ_WAIT_INST_ANY") / w, "wave_cycles": med(da, "SQ_WAVE_CYCLES") / w,
                   "lds_conflicts_per_cu": med(db, "SQ_LDS_BANK_CONFLICT") / 256}
            key = f"{kname} grid {grid}" + (f" size {ci + 1} of {len(clusters)}" if len(clusters) > 1 else "")
            rec["kernels"][key] = {k: round(v, 2) if isinstance(v, float) else v for k, v in row.items()}
            lines.append(f"| `{kname}` | {grid} | {e['vgpr']}+{e['agpr']} | {w:.0f} | {row['valu']:.0f} | "
                         f"{row['mfma']:.1f} | {row['lds_insts']:.1f} | {row['vmem']:.1f} | {row['salu']:.0f} | "
                         f"{row['mfma_busy_per_inst']:.0f} | {row['active_valu']:.0f} | {row['active_any']:.0f} | "
                         f"{row['wait_any']:.0f} | {row['wave_cycles']:.0f} | {row['lds_conflicts_per_cu']:.0f} |")
    lines += ["", "counter-record: " + json.dumps(rec, sort_keys=True)]
    return "\n".join(lines)


def kernel_summary(trace_csv: str, bench_json: str = None) -> str:
    """Markdown table of a rocprofv3 kernel trace: dispatches of the SBVR
    kernels grouped by kernel instance, workgroup size and grid size (threads),
    with count and mean / median / min / max duration (end - start timestamp),
    and the same over the back-to-back dispatches -- those that started when
    the dispatch before them (any kernel) ended, as every launch of a timed
    graph does when nothing holds the queue; the tracer itself delays some
    dispatches, and those start on an idle GPU.  With the traced run's own
    JSON line (bench_json), the record also carries that run's per-launch
    times of the batch-1 instances (step_launch_us), the live measurement
    taken under the same tracer."""
    import numpy as np
    disp = []
    with open(trace_csv, newline="") as f:
        for row in csv.DictReader(f):
            disp.append((int(row["Start_Timestamp"]), int(row["End_Timestamp"]), row["Kernel_Name"],
                         int(row["Workgroup_Size_X"]), int(row["Grid_Size_X"])))
    disp.sort()
    groups, b2b = {}, {}
    prev_end = None
    for start, end, name, wg, grid in disp:
        back_to_back = prev_end is not None and start <= prev_end
        prev_end = end if prev_end is None else max(prev_end, end)
        if "sbvr" not in name:
            continue
        key = (short_kernel_name(name), wg, grid)
        groups.setdefault(key, []).append(end - start)
        if back_to_back:
            b2b.setdefault(key, []).append(end - start)
    traced_live = {}
    if bench_json:
        with open(bench_json) as fh:
            line = json.loads([ln for ln in fh.read().splitlines() if ln.startswith("{")][-1])
        shapes = line["config"]["shapes"]
        k = int(re.search(r"SBVR k=(\d+)", line["config"]["workload"]).group(1))
        for proj, us in line.get("step_launch_us", {}).items():
            traced_live.setdefault(b1_kernel_instance(*shapes[proj], k), []).append(us)
    lines = ["| kernel | workgroup | grid | calls | mean ns | median ns | min ns | max ns | back-to-back calls | "
             "back-to-back mean ns | back-to-back median ns |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    rec = {"source_sha256": kernel_source_digest(), "kernels": {}}
    for key, d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        kname, wg, grid = key
        a = np.array(d, dtype=np.float64)
        bb = np.array(b2b.get(key, []), dtype=np.float64)
        bb_cols = f"{bb.size} | {bb.mean():.0f} | {np.median(bb):.0f}" if bb.size else "0 | - | -"
        lines.append(f"| `{kname}` | {wg} | {grid} | {a.size} | {a.mean():.0f} | {np.median(a):.0f} | "
                     f"{a.min():.0f} | {a.max():.0f} | {bb_cols} |")
        if kname.startswith("gemv_b1") and kname not in rec["kernels"]:  # the most-timed grid of each instance
            r = {"workgroup": wg, "grid": grid, "calls": int(a.size),
                 "mean_ns": round(float(a.mean()), 1), "median_ns": round(float(np.median(a)), 1)}
            if bb.size:
                r.update({"b2b_calls": int(bb.size), "b2b_mean_ns": round(float(bb.mean()), 1),
                          "b2b_median_ns": round(float(np.median(bb)), 1)})
            if kname in traced_live:
                r["traced_live_us"] = round(float(np.mean(traced_live[kname])), 3)
            rec["kernels"][kname] = r
    lines += ["", "rocprof-record: " + json.dumps(rec, sort_keys=True)]
    return "\n".join(lines)


def prefill_probe_cases():
    """(label, O, I, T) in the order --prefill-probe runs them: the distinct
    Llama-3-8B projection shapes times PREFILL_TOKENS."""
    import synth
    seen, cases = set(), []
    for name in PROJ_ORDER:
        O, I = synth.LLAMA8B[name]
        if (O, I) in seen:
            continue
        seen.add((O, I))
        cases += [(f"{name} {O}x{I}", O, I, T) for T in PREFILL_TOKENS]
    return cases


def prefill_summary(trace_csv: str) -> str:
    """Markdown table of a --prefill-probe kernel trace: per case, the mean
    duration of sbvr_decompress, of the library GEMM's kernels (per call) and
    of the fused sbvr_gemm_prefill, from the second of the two passes."""
    import numpy as np
    rows = []
    with open(trace_csv, newline="") as f:
        for r in csv.DictReader(f):
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]))
    rows.sort()
    segs = []
    for t0, t1, name in rows:
        if "FillFunctor" in name:  # the marker between phases
            segs.append([])
        elif segs:
            segs[-1].append((t1 - t0, name))
    segs = segs[1:]  # the marker tensor's own initial fill
    lines = ["| case | tokens | decompress us | library GEMM us | decompress + library us | fused us |",
             "|---|---:|---:|---:|---:|---:|"]
    rec = {}
    for i, (label, O, I, T) in enumerate(prefill_probe_cases()):
        dec, lib, fus = segs[6 * i + 3: 6 * i + 6]
        d = np.mean([x for x, n in dec if "decompress_kernel" in n]) / 1e3
        lb = sum(x for x, n in lib if "sbvr::" not in n) / PREFILL_PROBE_CALLS / 1e3
        fu = np.mean([x for x, n in fus if "prefill_kernel" in n or "prefill_long_kernel" in n]) / 1e3
        lines.append(f"| {label} | {T} | {d:.1f} | {lb:.1f} | {d + lb:.1f} | {fu:.1f} |")
        rec[f"{label} T={T}"] = {"decompress_us": round(d, 2), "library_us": round(lb, 2), "fused_us": round(fu, 2)}
    lines += ["", "prefill-record: " + json.dumps(rec, sort_keys=True)]
    return "\n".join(lines)


def load_rocprof(kernel: str):
    """The dominant kernel's mean dispatch duration from the committed
    rocprofv3 record of the headline command, when it was taken on the
    current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", ROCPROF_RECORD)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        recs = [json.loads(line.split(":", 1)[1]) for line in f if line.startswith("rocprof-record:")]
    if not recs or recs[-1].get("source_sha256") != kernel_source_digest():
        return None
    return recs[-1]["kernels"].get(kernel)


def load_traffic(kernel: str):
    """Calibrated HBM bytes per launch of `kernel` from the committed counter
    record, or None when there is none or it predates the current sources."""
    try:
        with open(TRAFFIC_RECORD) as fh:
            m = re.search(r"^traffic-record: (\{.*\})$", fh.read(), re.M)
        rec = json.loads(m.group(1))
    except (OSError, AttributeError, ValueError):
        return None
    if rec.get("source_sha256") != kernel_source_digest():
        return None
    k = rec["kernels"].get(kernel)
    return None if k is None else k["bytes_per_launch"]


def b1_kernel_instance(O: int, I: int, k: int, a8: bool = False, ix: bool = False) -> str:
    """Name of the batch-1 kernel instance the library launches for an O x I
    matrix: the streaming kernel (ring depth D, several gblocks per wavefront
    or one) when a row has more than 16 gblocks of 512 elements or the matrix
    has at least 24576 (tile, gblock) blocks (tiles of 16/k rows, 4 at k = 3),
    ring depth 2, or 3 with several gblocks per wavefront and >= 8 tiles per
    workgroup (256 workgroups), or 4 at k = 4 with one gblock per wavefront,
    at most 8 of them and per-group coefficients (256 workgroups); otherwise the one-shot
    kernel with T tiles per workgroup, the most of 8/4/2/1 that still leaves
    >= 256 workgroups and >= 2048 wavefronts (one per gblock).  The last two template arguments select the W4A8 build
    (activations converted online to SBVR-8) and the coefficient-cache format."""
    a8 = "true" if a8 else "false"
    ix = "true" if ix else "false"
    tr = {1: 16, 2: 8}.get(k, 4)  # rows per tile: 16 matrix-core rows of (row, plane)
    n_tiles, n_gblocks = (O + tr - 1) // tr, (I + 511) // 512
    if n_gblocks > 16 or n_tiles * n_gblocks >= 24576:
        multi = n_gblocks > 16
        tpw = (n_tiles + 255) // 256
        wide = k == 4 and not multi and n_gblocks <= 8 and ix == "false"
        depth = (3 if tpw >= 8 else 2) if multi else (4 if wide else 2)
        return f"gemv_b1s_kernel<{k}, {depth}, {'true' if multi else 'false'}, {a8}, {ix}>"
    T = next((t for t in (8, 4, 2) if n_tiles // t >= 256 and (n_tiles // t) * n_gblocks >= 2048), 1)
    return f"gemv_b1_kernel<{k}, {T}, {a8}, {ix}>"


ROTATE_BYTES = 1e9  # 4x the 256 MB MALL: a cyclic sweep gets no cache reuse


def cpu_model_name():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def prefill_probe(k, dev):
    """Eager launches for a kernel trace: per case (prefill_probe_cases), two
    passes of [marker] 16 x sbvr_decompress [marker] 16 x library GEMM on the
    decompressed matrix [marker] 16 x sbvr_gemm_prefill, over 16 packed copies
    of one random SBVR matrix."""
    import numpy as np
    import torch

    import paper_2509_18172_amd as sb
    import synth
    marker = torch.zeros(1, device=dev)
    cur = None
    for label, O, I, T in prefill_probe_cases():
        if cur != (O, I):
            Ws = None
            torch.cuda.empty_cache()
            planes, coeffs = synth.random_sbvr(O, I, k, seed=O + I)
            p = torch.from_numpy(planes.view(np.int32)).to(dev)
            c = torch.from_numpy(coeffs.view(np.int16)).to(dev)
            Ws = [sb.pack(p, c) for _ in range(PREFILL_PROBE_CALLS)]
            M = torch.empty((O, I), dtype=torch.float16, device=dev)
            cur = (O, I)
        X = torch.from_numpy(synth.activations(I, seed=T, batch=T)).to(dev)
        Y = torch.empty((T, O), dtype=torch.float16, device=dev)
        for _ in range(2):  # the first pass settles the library's kernel choice
            marker.fill_(1.0)
            for W in Ws:
                sb.decompress(W, out=M)
            marker.fill_(2.0)
            for _ in range(PREFILL_PROBE_CALLS):
                torch.nn.functional.linear(X, M)
            marker.fill_(3.0)
            for W in Ws:
                sb.gemm_prefill(W, X, out=Y)
            torch.cuda.synchronize()
        print(f"prefill-probe: {label} T={T} done", flush=True)


def main():
    args = parse()
    if args.traffic_summary:
        print(traffic_summary(*args.traffic_summary))
        return
    if args.kernel_summary:
        print(kernel_summary(*args.kernel_summary[:2]))
        return
    if args.prefill_summary:
        print(prefill_summary(args.prefill_summary))
        return
    if args.counter_summary:
        print(counter_summary(*args.counter_summary))
        return
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
    if args.prefill_probe:
        prefill_probe(args.k, dev)
        return
    shapes = synth.LLAMA8B if args.model == "llama3-8b" else synth.LLAMA70B
    k = args.k
    nbytes = {n: sb.algorithmic_bytes(*shapes[n], k) for n in PROJ_ORDER}
    layer_bytes = sum(nbytes.values())
    L = args.layers or 32
    if args.traffic_probe:
        L = PROBE_LAUNCHES
    cfg_index = 1 if args.model == "llama3-8b" else 3

    def to_dev(planes, coeffs):
        return (torch.from_numpy(planes.view(np.int32)).to(dev), torch.from_numpy(coeffs.view(np.int16)).to(dev))

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
            W = sb.pack(*to_dev(planes, coeffs))
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

    if args.traffic_probe:
        with torch.cuda.stream(stream):
            for name in PROJ_ORDER:
                for li in range(L):
                    W, x, y = layers[li][name]
                    sb.gemv(W, x, out=y, stream=stream)
            for name in PROJ_ORDER:  # the W4A8 build of the same kernels
                for li in range(L):
                    W, x, y = layers[li][name]
                    sb.gemv_a8(W, x, out=y, stream=stream)
            for li in range(L):  # grouped launches: q|k|v and gate|up of each layer
                for names in (("q", "k", "v"), ("gate", "up")):
                    lay = layers[li]
                    sb.gemv_grouped([lay[n][0] for n in names], [lay[names[0]][1]] * len(names),
                                    outs=[lay[n][2] for n in names], stream=stream)
            for name in PROJ_ORDER:  # small batch, B = 8 vectors
                O, I = shapes[name]
                X8 = torch.from_numpy(synth.activations(I, seed=77, batch=8)).to(dev)
                Y8 = torch.empty((8, O), dtype=torch.float16, device=dev)
                for li in range(L):
                    sb.gemm_small_batch(layers[li][name][0], X8, out=Y8, stream=stream)
            for name in PROJ_ORDER:  # coefficient-cache format, one set per ten groups
                O, I = shapes[name]
                n_sets = max(1, min(65536, (O * (I // 128) + 9) // 10))
                planes, index, table = synth.random_indexed_sbvr(O, I, k, n_sets, seed=synth.seed_for(6, 0, 0))
                Wi = sb.pack_indexed(*(torch.from_numpy(a).to(dev) for a in (planes.view(np.int32), index.view(np.int16),
                                                                              table.view(np.int16))))
                x, y = layers[0][name][1], layers[0][name][2]
                for _ in range(L):
                    sb.gemv_indexed(Wi, x, out=y, stream=stream)
            for name in PROJ_ORDER:  # prefill decompression of the same weights
                O, I = shapes[name]
                M = torch.empty((O, I), dtype=torch.float16, device=dev)
                for li in range(L):
                    sb.decompress(layers[li][name][0], out=M, stream=stream)
            # calibration: an elementwise kernel that reads and writes CALIB_BYTES
            src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"traffic_probe": True, "launches_per_shape": L, "copy_bytes": CALIB_BYTES}))
        return

    def capture(calls):
        """One graph of (fn, args) launches on the bench stream."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for fn, a in calls:
                fn(*a, stream=stream)
        return g

    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)

    def timed(fn):
        with torch.cuda.stream(stream):
            e0.record(stream)
            fn()
            e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)  # ms

    def gemv_call(W, x, y):
        return (lambda W, x, y, stream: sb.gemv(W, x, out=y, stream=stream)), (W, x, y)

    # ---- timed region: one graph of exactly K layer-steps, step i running
    # layer i % L's seven GEMVs (so the weights cycle through all L layers and
    # no step hits a cache), after one replay of a W-step warm-up graph ----
    def step_calls(n, first=0):
        return [gemv_call(*layers[(first + i) % L][nm]) for i in range(n) for nm in PROJ_ORDER]

    steps_graph = capture(step_calls(args.steps))
    if args.warmup:
        warm_graph = capture(step_calls(args.warmup, first=args.steps))
        timed(warm_graph.replay)
        del warm_graph
    # the first replays of a new graph are untimed as well (with a single one,
    # the timed replay after it was at times up to 9 % slower than the rest)
    for _ in range(3):
        timed(steps_graph.replay)
    torch.cuda.synchronize()
    total_ms = timed(steps_graph.replay)
    ms_per_step = total_ms / args.steps
    value = layer_bytes * args.steps / (total_ms * 1e-3) / 1e9
    # the same K-step graph replayed again: spread of the headline measurement
    rep_ms = [timed(steps_graph.replay) / args.steps for _ in range(5)]
    headline_spread = {"replays": len(rep_ms), "ms_per_step_median": round(float(np.median(rep_ms)), 5),
                       "ms_per_step_min": round(min(rep_ms), 5), "ms_per_step_max": round(max(rep_ms), 5)}
    del steps_graph

    # The launch durations inside the timed region, per projection: the timed
    # K-step graph against the same graph without that projection's launches,
    # replayed alternately (nine pairs, each replay timed with events on the
    # bench stream); the median difference over the launches removed is the
    # time one launch adds to a step (its kernel plus the gap to the next).
    def step_graph_without(skip):
        return capture([gemv_call(*layers[i % L][nm]) for i in range(args.steps) for nm in PROJ_ORDER
                        if nm not in skip])

    def launch_times_in_steps(pairs=9):
        full = step_graph_without(())
        timed(full.replay)
        t, full_ms = {}, []
        for nm in PROJ_ORDER:
            if nm in t:
                continue
            group = [m for m in PROJ_ORDER if shapes[m] == shapes[nm]]  # same shape, same kernel
            part = step_graph_without(group)
            timed(part.replay)
            diffs = []
            for _ in range(pairs):
                a_ms = timed(full.replay)
                diffs.append(a_ms - timed(part.replay))
                full_ms.append(a_ms)
            del part
            per = float(np.median(diffs)) * 1e3 / (args.steps * len(group))
            for m in group:
                t[m] = [per]
        del full
        return t, float(np.median(full_ms))

    launch_times, full_ms = launch_times_in_steps()
    # dominant kernel instance: largest launch time per step
    by_kernel = {}
    for n in PROJ_ORDER:
        kname = b1_kernel_instance(*shapes[n], k)
        t, b, c = by_kernel.get(kname, (0.0, 0, 0))
        by_kernel[kname] = (t + float(np.mean(launch_times[n])), b + nbytes[n], c + 1)
    dom = max(by_kernel, key=lambda kk: by_kernel[kk][0])
    dt, db, dc = by_kernel[dom]
    dom_projs = [n for n in PROJ_ORDER if b1_kernel_instance(*shapes[n], k) == dom]
    launch_durations = [t for n in dom_projs for t in launch_times[n]]
    dom_us = float(np.mean(launch_durations))
    bytes_per_launch = db / dc
    achieved = bytes_per_launch / (dom_us * 1e3)  # GB/s
    roofline = {
        "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_GBPS, "unit": "GB/s",
        "frac": round(achieved / PEAK_GBPS, 4),
        "traffic": load_traffic(dom) if k == 4 and args.model == "llama3-8b" else None,
        "kernel": dom,
        "launches_per_step": dc,
        "projections": dom_projs,
        "bytes_per_launch": round(bytes_per_launch),
        "mean_launch_us": round(dom_us, 3),
        "launch_timing": f"the timed {args.steps}-step graph ({full_ms:.3f} ms) minus the same graph without "
                         f"its {dc * args.steps} launches, per launch: median of 9 alternating replay pairs, "
                         f"HIP events on the bench stream",
    }
    prof = load_rocprof(dom) if k == 4 and args.model == "llama3-8b" else None
    if prof is not None:
        prof_us = prof["mean_ns"] / 1e3
        med_us = prof["median_ns"] / 1e3
        roofline["rocprof"] = {"mean_launch_us": round(prof_us, 3), "median_launch_us": round(med_us, 3),
                               "frac_mean": round(bytes_per_launch / (prof_us * 1e3) / PEAK_GBPS, 4),
                               "frac_median": round(bytes_per_launch / (med_us * 1e3) / PEAK_GBPS, 4),
                               "mean_over_live": round(prof_us / dom_us, 4),
                               "median_over_live": round(med_us / dom_us, 4),
                               "record": f"profiles/{ROCPROF_RECORD} ({prof['calls']} dispatches, grid {prof['grid']})"}
        if "b2b_mean_ns" in prof:  # dispatches that started when the one before them ended
            bm, bmed = prof["b2b_mean_ns"] / 1e3, prof["b2b_median_ns"] / 1e3
            roofline["rocprof"]["back_to_back"] = {
                "calls": prof["b2b_calls"], "mean_launch_us": round(bm, 3), "median_launch_us": round(bmed, 3),
                "frac_mean": round(bytes_per_launch / (bm * 1e3) / PEAK_GBPS, 4),
                "frac_median": round(bytes_per_launch / (bmed * 1e3) / PEAK_GBPS, 4),
                "mean_over_live": round(bm / dom_us, 4), "median_over_live": round(bmed / dom_us, 4)}
        if "traced_live_us" in prof:  # the traced run's own per-launch time, under the same tracer
            roofline["rocprof"]["traced_live_us"] = prof["traced_live_us"]
            roofline["rocprof"]["mean_over_traced_live"] = round(prof_us / prof["traced_live_us"], 4)
    step_launch_us = {n: round(float(np.mean(launch_times[n])), 3) for n in PROJ_ORDER}

    decode_graph = capture([gemv_call(*layers[li][n]) for li in range(L) for n in PROJ_ORDER])
    torch.cuda.synchronize()

    # the decode step alone (configs: one token through all L layers)
    step_reps = [timed(decode_graph.replay) * 1e3 for _ in range(DECODE_REPLAYS)]
    decode_us = float(np.median(step_reps))
    decode_step = {"layers": L, "gemvs": 7 * L, "bytes": layer_bytes * L, "us_per_token": round(decode_us, 2),
                   "gbps": round(layer_bytes * L / (decode_us * 1e3), 1),
                   "mean_us_per_token": round(float(np.mean(step_reps)), 2),
                   "replays": len(step_reps)}
    del decode_graph

    def result_line(extra):
        return {
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
                            f"group 128, batch 1; {args.steps} layer-steps in one hipGraph on one stream, "
                            f"step i on layer i mod {L} ({L} layers' weights, {L * layer_bytes / 1e9:.2f} GB)",
                "bytes_per_step": layer_bytes,
                "layers_rotated": L,
                "shapes": {n: list(shapes[n]) for n in PROJ_ORDER},
            },
            "pct_of_peak": round(100 * value / PEAK_GBPS, 2),
            "headline_spread": headline_spread,
            "roofline": roofline,
            "step_launch_us": step_launch_us,
            "decode_step": decode_step,
            **extra,
        }

    if args.headline_only:
        print(json.dumps(result_line({})), flush=True)
        return

    # the same decode step with SBVR-8 activations (the paper's W4A8 decode)
    decode_step_a8 = None
    if not args.quick:
        a8_graph = capture([((lambda W, x, y, stream: sb.gemv_a8(W, x, out=y, stream=stream)), layers[li][n])
                            for li in range(L) for n in PROJ_ORDER])
        timed(a8_graph.replay)
        reps = [timed(a8_graph.replay) * 1e3 for _ in range(5)]
        us = float(np.median(reps))
        decode_step_a8 = {"us_per_token": round(us, 2), "gbps": round(layer_bytes * L / (us * 1e3), 1)}
        del a8_graph

    # the same weights with the projections that share an input packed as one
    # matrix each (rows concatenated: q|k|v and gate|up), as a serving stack
    # lays them out: 4 GEMVs per layer instead of 7, same weight bytes
    decode_step_fused = None
    if not args.quick:
        def fuse_rows(ws):
            parts = [sb.unpack(w) for w in ws]
            return sb.pack(torch.cat([p for p, _ in parts]), torch.cat([c for _, c in parts]))

        fused_calls = []
        fused_layers = []
        for li in range(L):
            lay = layers[li]
            qkv = fuse_rows([lay[n][0] for n in ("q", "k", "v")])
            gu = fuse_rows([lay[n][0] for n in ("gate", "up")])
            y_qkv = torch.empty(qkv.O, dtype=torch.float16, device=dev)
            y_gu = torch.empty(gu.O, dtype=torch.float16, device=dev)
            fused_layers.append((qkv, gu, y_qkv, y_gu))
            fused_calls += [gemv_call(qkv, lay["q"][1], y_qkv), gemv_call(*lay["o"]),
                            gemv_call(gu, lay["gate"][1], y_gu), gemv_call(*lay["down"])]
        torch.cuda.synchronize()
        fused_graph = capture(fused_calls)
        timed(fused_graph.replay)
        reps = [timed(fused_graph.replay) * 1e3 for _ in range(5)]
        us = float(np.median(reps))
        decode_step_fused = {"gemvs": len(fused_calls), "us_per_token": round(us, 2),
                             "gbps": round(layer_bytes * L / (us * 1e3), 1)}
        del fused_graph, fused_layers
        torch.cuda.empty_cache()

    # the same 224 GEMVs on the separate weights, the projections that share
    # an input (q, k, v; gate, up) each enqueued as one grouped launch
    # (sbvr_gemv_grouped): 4 launches per layer, no repacking
    decode_step_grouped = None
    if not args.quick:
        def grouped_call(names, lay):
            Ws, ys = [lay[n][0] for n in names], [lay[n][2] for n in names]
            x = lay[names[0]][1]
            return (lambda Ws, x, ys, stream: sb.gemv_grouped(Ws, [x] * len(Ws), outs=ys, stream=stream)), (Ws, x, ys)

        grouped_calls = []
        for li in range(L):
            lay = layers[li]
            grouped_calls += [grouped_call(("q", "k", "v"), lay), gemv_call(*lay["o"]),
                              grouped_call(("gate", "up"), lay), gemv_call(*lay["down"])]
        grouped_graph = capture(grouped_calls)
        timed(grouped_graph.replay)
        reps = [timed(grouped_graph.replay) * 1e3 for _ in range(DECODE_REPLAYS)]
        us = float(np.median(reps))
        decode_step_grouped = {"launches": len(grouped_calls), "gemvs": 7 * L, "us_per_token": round(us, 2),
                               "mean_us_per_token": round(float(np.mean(reps)), 2),
                               "gbps": round(layer_bytes * L / (us * 1e3), 1), "replays": len(reps)}
        del grouped_graph
        # the same with SBVR-8 activations (the paper's W4A8 decode configuration)
        a8_calls = []
        for li in range(L):
            lay = layers[li]
            for names in (("q", "k", "v"), ("o",), ("gate", "up"), ("down",)):
                Ws, ys = [lay[n][0] for n in names], [lay[n][2] for n in names]
                a8_calls.append(((lambda Ws, x, ys, stream: sb.gemv_grouped(Ws, [x] * len(Ws), outs=ys, stream=stream,
                                                                            a8=True)), (Ws, lay[names[0]][1], ys)))
        a8_graph = capture(a8_calls)
        timed(a8_graph.replay)
        reps = [timed(a8_graph.replay) * 1e3 for _ in range(DECODE_REPLAYS)]
        us = float(np.median(reps))
        decode_step_grouped["w4a8_us_per_token"] = round(us, 2)
        decode_step_grouped["w4a8_gbps"] = round(layer_bytes * L / (us * 1e3), 1)
        del a8_graph

    # ---- per-launch durations: >= 64 back-to-back launches per graph, cycling
    # through distinct weight copies totalling >= ROTATE_BYTES ----
    def launch_us(calls, n_launch=64, replays=11):
        g = capture([calls[i % len(calls)] for i in range(max(n_launch, len(calls)))])
        n = max(n_launch, len(calls))
        for _ in range(2):
            timed(g.replay)
        reps = [timed(g.replay) * 1e3 / n for _ in range(replays)]
        del g
        return float(np.median(reps))

    def copies(O, I, kk, planes, coeffs, have):
        """Extra packed copies (same content, distinct memory) so that `have`
        copies plus these rotate through >= ROTATE_BYTES."""
        per = sb.algorithmic_bytes(O, I, kk)
        need = max(0, int(np.ceil(ROTATE_BYTES / per)) - have)
        if need == 0:
            return []
        p, c = to_dev(planes, coeffs)
        return [sb.pack(p, c) for _ in range(need)]

    weights = {}  # projection -> list of packed copies (the L layers first)
    for name in PROJ_ORDER:
        O, I = shapes[name]
        extra = copies(O, I, k, *host_layer0[name], have=L)
        weights[name] = [layers[li][name][0] for li in range(L)] + extra
    torch.cuda.synchronize()

    per_call_us = {}
    for name in PROJ_ORDER:
        O, I = shapes[name]
        ws = weights[name]
        xs = [torch.from_numpy(synth.activations(I, seed=900 + i)).to(dev) for i in range(min(len(ws), 64))]
        ys = [torch.empty(O, dtype=torch.float16, device=dev) for _ in range(len(xs))]
        per_call_us[name] = launch_us([gemv_call(w, xs[i % len(xs)], ys[i % len(ys)]) for i, w in enumerate(ws)])
    per_call_gbps = {n: nbytes[n] / (per_call_us[n] * 1e3) for n in PROJ_ORDER}

    # the same calls timed one by one: an event pair around each of
    # EVENT_CALLS eager launches (after EVENT_WARMUP), cycling through the
    # same copies; median and mean per call (these include each launch's
    # share of the host-side enqueue gaps that a graph removes)
    per_call_events = {}
    for name in PROJ_ORDER:
        O, I = shapes[name]
        ws = weights[name]
        x = layers[0][name][1]
        y = torch.empty(O, dtype=torch.float16, device=dev)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(EVENT_CALLS)]
        with torch.cuda.stream(stream):
            for i in range(EVENT_WARMUP):
                sb.gemv(ws[i % len(ws)], x, out=y, stream=stream)
            for i, (a, b) in enumerate(evs):
                a.record(stream)
                sb.gemv(ws[(EVENT_WARMUP + i) % len(ws)], x, out=y, stream=stream)
                b.record(stream)
        torch.cuda.synchronize()
        t = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])
        per_call_events[name] = {"median_us": round(float(np.median(t)), 3), "mean_us": round(float(t.mean()), 3)}


    # ---- practical ceiling: a plain streaming read of the same bytes (the
    # helper in read_probe.hip), grid-interleaved and chunked per workgroup ----
    def stream_read_us(nbytes):
        import ctypes as C
        from paper_2509_18172_amd.build import probe_path
        probe = C.CDLL(probe_path())
        probe.sbvr_probe_stream_read.argtypes = [C.c_void_p, C.c_size_t, C.c_int, C.c_void_p, C.c_void_p]
        n16 = (nbytes + 15) // 16 * 16
        copies_r = max(2, int(np.ceil(ROTATE_BYTES / n16)))
        buf = torch.ones(copies_r * n16, dtype=torch.uint8, device=dev)
        sink = torch.zeros(4, dtype=torch.int32, device=dev)
        res = {}
        def read(off, chunked, stream):
            st = probe.sbvr_probe_stream_read(buf.data_ptr() + off, n16, chunked, sink.data_ptr(),
                                              stream.cuda_stream)
            if st != 0:
                raise RuntimeError(f"stream-read probe launch failed ({st})")

        for tag, chunked in (("interleaved", 0), ("chunked", 1)):
            res[tag] = launch_us([(read, (i * n16, chunked)) for i in range(copies_r)])
        del buf
        return res

    ceiling = stream_read_us(roofline["bytes_per_launch"])
    best = min(ceiling.values())
    roofline["practical_peak"] = {
        "what": "plain streaming read of the same bytes per launch (16-byte loads, same 64-launch graphs, "
                ">= 1 GB rotation)",
        "read_us": {kk: round(v, 3) for kk, v in ceiling.items()},
        "gbps": round(roofline["bytes_per_launch"] / (best * 1e3), 1),
        "frac": round(best / float(np.mean([per_call_us[n] for n in dom_projs])), 4)}

    def gemm_call(W, X, Y):
        return (lambda W, X, Y, stream: sb.gemm_small_batch(W, X, out=Y, stream=stream)), (W, X, Y)

    # ---- small batch (B = 2, 4, 8) on the same weight copies ----
    small_batch = {}
    if not args.quick:
        for B in (2, 4, 8):
            res = {}
            for name in PROJ_ORDER:
                O, I = shapes[name]
                ws = weights[name]
                Xs = [torch.from_numpy(synth.activations(I, seed=700 + i, batch=B)).to(dev) for i in range(8)]
                Ys = [torch.empty((B, O), dtype=torch.float16, device=dev) for _ in range(8)]
                us = launch_us([gemm_call(w, Xs[i % 8], Ys[i % 8]) for i, w in enumerate(ws)])
                bb = sb.algorithmic_bytes(O, I, k, B)
                res[name] = {"us": round(us, 3), "gbps": round(bb / (us * 1e3), 1)}
            small_batch[str(B)] = res

    # ---- W4A8 decode (sbvr_gemv_a8: activations converted online to SBVR-8)
    # on the same weight copies ----
    w4a8 = {}
    if not args.quick:
        def a8_call(W, x, y):
            return (lambda W, x, y, stream: sb.gemv_a8(W, x, out=y, stream=stream)), (W, x, y)
        for name in PROJ_ORDER:
            O, I = shapes[name]
            ws = weights[name]
            xs = [torch.from_numpy(synth.activations(I, seed=800 + i)).to(dev) for i in range(8)]
            ys = [torch.empty(O, dtype=torch.float16, device=dev) for _ in range(8)]
            us = launch_us([a8_call(w, xs[i % 8], ys[i % 8]) for i, w in enumerate(ws)])
            w4a8[name] = {"us": round(us, 3), "gbps": round(nbytes[name] / (us * 1e3), 1)}

    # ---- prefill path: decompression to binary16 (HBM-bound: reads the SBVR
    # bytes, writes 2 bytes per weight), then a library GEMM over T tokens ----
    prefill = {}
    if not args.quick:
        T = 512
        for name in PROJ_ORDER:
            O, I = shapes[name]
            if any(shapes[m] == (O, I) for m in prefill):
                prefill[name] = prefill[next(m for m in prefill if shapes[m] == (O, I))]
                continue
            ws = weights[name][:32]
            n_out = max(2, int(np.ceil(ROTATE_BYTES / (2 * O * I))))
            outs = [torch.empty((O, I), dtype=torch.float16, device=dev) for _ in range(n_out)]
            dec = (lambda W, M, stream: sb.decompress(W, out=M, stream=stream))
            us = launch_us([(dec, (w, outs[i % n_out])) for i, w in enumerate(ws)], n_launch=32)
            bb = sb.algorithmic_bytes(O, I, k, 0) + 2 * O * I
            # the paper's prefill: decompression, then Y[T][O] = X[T][I] W^T in
            # the library GEMM (the layout of a linear layer, faster in the
            # library than W X^T for these shapes) on the matrix just written;
            # timed as pairs in one graph over the rotating SBVR copies, as
            # the fused GEMM below is
            Xs = torch.from_numpy(synth.activations(I, seed=31, batch=T)).to(dev)

            def dec_gemm(W, M, X, Y, stream):
                sb.decompress(W, out=M, stream=stream)
                with torch.cuda.stream(stream):
                    torch.mm(X, M.t(), out=Y)

            paper_path = {}
            for TT in PREFILL_TOKENS:
                XT = Xs[:TT].contiguous()
                Y = torch.empty((TT, O), dtype=torch.float16, device=dev)
                for _ in range(3):   # library handles and heuristics set up outside the capture
                    dec_gemm(ws[0], outs[0], XT, Y, stream=stream)
                torch.cuda.synchronize()
                paper_path[str(TT)] = round(launch_us([(dec_gemm, (w, outs[i % n_out], XT, Y))
                                                       for i, w in enumerate(ws[:16])],
                                                      n_launch=16, replays=5), 2)
            # the fused GEMM (sbvr_gemm_prefill: the binary16 weights never
            # reach memory) over the same SBVR copies, per prompt length
            fused = {}
            pf = (lambda W, X, Y, stream: sb.gemm_prefill(W, X, out=Y, stream=stream))
            for TT in PREFILL_TOKENS:
                XT = Xs[:TT].contiguous()
                Ys = [torch.empty((TT, O), dtype=torch.float16, device=dev) for _ in range(2)]
                fused[str(TT)] = round(launch_us([(pf, (w, XT, Ys[i % 2])) for i, w in enumerate(ws[:16])],
                                                 n_launch=16, replays=5), 2)
            prefill[name] = {"decompress_us": round(us, 3), "decompress_gbps": round(bb / (us * 1e3), 1),
                             "decompress_bytes": bb, "decompress_gemm_us": paper_path,
                             "fused_gemm_us": fused}
            del outs
            torch.cuda.empty_cache()

    # ---- fewer planes (k = 2, 3) and the other model's shapes ----
    def shape_table(shp, kk, seed_cfg):
        res = {}
        for pi, name in enumerate(PROJ_ORDER):
            O, I = shp[name]
            if name in res or any(shp[m] == (O, I) and m in res for m in res):
                same = next(m for m in res if shp[m] == (O, I))
                res[name] = res[same]
                continue
            planes, coeffs = synth.random_sbvr(O, I, kk, seed=synth.seed_for(seed_cfg, 0, pi))
            ws = copies(O, I, kk, planes, coeffs, have=0)
            x = torch.from_numpy(synth.activations(I, seed=seed_cfg + pi + synth.X_SEED_OFFSET)).to(dev)
            y = torch.empty(O, dtype=torch.float16, device=dev)
            us = launch_us([gemv_call(w, x, y) for w in ws])
            bb = sb.algorithmic_bytes(O, I, kk)
            res[name] = {"us": round(us, 3), "gbps": round(bb / (us * 1e3), 1), "copies": len(ws)}
            del ws
            torch.cuda.empty_cache()
        return res

    # ---- coefficient-cache format (index + table of coefficient sets), with
    # fp16 and SBVR-8 activations; one set per ten groups (a 90 % encoder cache
    # hit rate), at most 65536 ----
    def indexed_table(shp, kk, seed_cfg):
        res = {}
        for pi, name in enumerate(PROJ_ORDER):
            O, I = shp[name]
            same = next((m for m in res if shp[m] == (O, I)), None)
            if same is not None:
                res[name] = res[same]
                continue
            n_sets = max(1, min(65536, (O * (I // 128) + 9) // 10))
            planes, index, table = synth.random_indexed_sbvr(O, I, kk, n_sets, seed=synth.seed_for(seed_cfg, 0, pi))
            p, ix, tb = (torch.from_numpy(a).to(dev) for a in (planes.view(np.int32), index.view(np.int16),
                                                                  table.view(np.int16)))
            per = sb.algorithmic_bytes_indexed(O, I, kk, n_sets)
            ws = [sb.pack_indexed(p, ix, tb) for _ in range(int(np.ceil(ROTATE_BYTES / per)))]
            x = torch.from_numpy(synth.activations(I, seed=seed_cfg + pi + synth.X_SEED_OFFSET)).to(dev)
            y = torch.empty(O, dtype=torch.float16, device=dev)
            entry = {"n_sets": n_sets, "bytes": per, "copies": len(ws)}
            for tag, a8 in (("fp16", False), ("a8", True)):
                fn = (lambda W, x, y, stream, a8=a8: sb.gemv_indexed(W, x, out=y, a8=a8, stream=stream))
                us = launch_us([(fn, (w, x, y)) for w in ws])
                entry[f"us_{tag}"] = round(us, 3)
                entry[f"gbps_{tag}"] = round(per / (us * 1e3), 1)
            res[name] = entry
            del ws
            torch.cuda.empty_cache()
        return res

    indexed = None
    if not args.quick and k == 4:
        indexed = indexed_table(shapes, k, 6)

    low_bit, other_model = {}, None
    if not args.quick:
        if args.model == "llama3-8b" and k == 4:
            for kk in (2, 3):
                low_bit[str(kk)] = shape_table(shapes, kk, 2)
            other_model = shape_table(synth.LLAMA70B, 4, 3)
        elif args.model == "llama3-70b":
            other_model = shape_table(synth.LLAMA8B, k, 1)

    # ---- encoder (Algorithm 1 on the GPU, bit-identical to the oracle's) on a
    # q/o-shaped fp32 matrix, and the oracle's encoder on a sample of its rows ----
    encoder = None
    if not args.quick:
        O, I = shapes["q"]
        Wf = synth.weights(O, I, 0.02 if args.model == "llama3-8b" else 0.015, seed=synth.seed_for(cfg_index, 0, 0))
        Wd = torch.from_numpy(Wf).to(dev)
        with torch.cuda.stream(stream):
            sb.encode(Wd, k, stream=stream)
        torch.cuda.synchronize()
        reps = [timed(lambda: sb.encode(Wd, k, stream=stream)) * 1e-3 for _ in range(3)]
        sec = float(np.median(reps))
        groups = O * (I // 128)
        encoder = {"shape": [O, I], "k": k, "groups": groups, "entries_per_group": 1024,
                   "gpu_s": round(sec, 4), "gpu_groups_per_s": round(groups / sec)}
        # the encoder cache of Sec. 4.2 (64 sets per row): time, hit rate, the
        # error against the exhaustive search, and the distinct coefficient
        # sets (the indexed format's table) with and without it
        with torch.cuda.stream(stream):
            _, c0, m0 = sb.encode(Wd, k, want_mse=True, stream=stream)
            _, cc, mc, hc = sb.encode_cached(Wd, k, 64, stream=stream)
        torch.cuda.synchronize()
        reps = [timed(lambda: sb.encode_cached(Wd, k, 64, stream=stream)) * 1e-3 for _ in range(3)]
        sec_c = float(np.median(reps))
        n_sets = lambda c: int(torch.unique(c.reshape(-1, k), dim=0).shape[0])
        encoder["cached"] = {"cache_slots": 64, "gpu_s": round(sec_c, 4), "gpu_groups_per_s": round(groups / sec_c),
                             "hit_rate": round(float(hc.float().mean()), 4),
                             "mse_over_exhaustive": round(float(mc.mean() / m0.mean()), 4),
                             "distinct_sets": n_sets(cc), "distinct_sets_exhaustive": n_sets(c0)}
        del c0, m0, cc, mc, hc
        if not args.no_cpu_baseline:
            import oracle
            rows = 128
            ts = time.perf_counter()
            oracle.encode_matrix(Wf[:rows], k)
            el = time.perf_counter() - ts
            encoder["oracle_groups_per_s"] = round(rows * (I // 128) / el, 1)
            encoder["oracle_sample"] = f"{rows} rows ({rows * (I // 128)} groups), {el:.1f} s on {os.cpu_count()} threads"
        del Wd

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
        # the same oracle on one thread, over layer 0's q projection
        one_bytes, one_el, one_passes = 0, 0.0, 0
        planes, coeffs = host_layer0["q"]
        xq = layers[0]["q"][1].cpu().numpy()
        while one_el < args.cpu_seconds / 4 or one_passes == 0:
            ts = time.perf_counter()
            oracle.sbvr_gemv(planes, coeffs, xq, nthreads=1)
            one_el += time.perf_counter() - ts
            one_bytes += nbytes["q"]
            one_passes += 1
        cpu = {"value": round(done_bytes / elapsed / 1e9, 4), "unit": "GB/s", "cores": threads,
               "kind": "oracle",
               "sample": f"{passes} pass(es) over layer 0's seven GEMVs ({args.model}, k={k}, batch 1): "
                         f"{elapsed:.1f} s of binary64 decompress + GEMV on {threads} threads "
                         f"({os.cpu_count()} host CPUs, {platform.machine()})",
               "cpu_model": cpu_model_name(),
               "one_core": {"value": round(one_bytes / one_el / 1e9, 4), "unit": "GB/s",
                            "us_per_gemv": round(one_el / one_passes * 1e6, 1),
                            "sample": f"{one_passes} q GEMV(s) ({shapes['q'][0]}x{shapes['q'][1]}), "
                                      f"{one_el:.1f} s on 1 thread"}}

    roofline["mean_launch_interval_us"] = round(float(np.mean([per_call_us[n] for n in dom_projs])), 3)
    roofline["interval_timing"] = ("events around a graph of 64 back-to-back launches over >= 1 GB of weight copies "
                                   "(includes the gap between kernels)")
    out = result_line({
        "per_call_us": {n: round(v, 3) for n, v in per_call_us.items()},
        "per_call_gbps": {n: round(v, 1) for n, v in per_call_gbps.items()},
        "per_call_events": per_call_events,
        "decode_step_w4a8": decode_step_a8,
        "decode_step_fused": decode_step_fused,
        "decode_step_grouped": decode_step_grouped,
        "small_batch": small_batch or None,
        "w4a8": w4a8 or None,
        "indexed": indexed,
        "encoder": encoder,
        "low_bit": low_bit or None,
        "prefill": prefill or None,
        ("llama3_70b" if args.model == "llama3-8b" else "llama3_8b"): other_model,
        "cpu_baseline": cpu,
    })
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
