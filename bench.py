#!/usr/bin/env python3
"""Benchmark of the Carryover drafter round on one MI355X.

One step = one full drafter round (route -> E_carry + F -> all-layer K/V with
RoPE, commit/replace -> block attention over committed + carry KV) of the
ragged batch-32 serving workload: 32 sequences, block 16, Dcat 768 -> d 256,
4 query / 2 KV heads, head_dim 64, bf16, committed contexts drawn uniformly in
512..8192 tokens in a seeded random 16-token page order, accepted lengths
geometric (p = 0.25) truncated at 16.  Rounds are chained: each round commits
its accepted rows and replaces the carry segment.  All inputs are synthetic,
seeded and resident in HBM before timing starts.

Timing: ``value`` is chained rounds per second, each round one
``carryover_round`` call, over the timed steps.  The attention entry point is
then timed on its own with HIP events around each ``drafter_block_attention``
call, on the state the chain reached, for the roofline fraction (the round
call launches its kernels back to back, so they cannot be bracketed inside
it).

Prints one JSON line (see the repository's benchmark contract) with the
attention kernel's roofline fraction and an fp64 CPU oracle baseline.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense bf16 MFMA; fp32 vector (cfg1 path)
PROFILES = os.path.join(ROOT, "profiles")
# sources of the attention kernels: traffic counters taken on another version
# of these are not reported
ATTN_SOURCES = [os.path.join(ROOT, "paper_2609_14717_amd", "csrc", f)
                for f in ("attention.hip", "co_device.h", "co_kernels.h")]
PROJ_SOURCES = [os.path.join(ROOT, "paper_2609_14717_amd", "csrc", f)
                for f in ("project.hip", "co_device.h", "co_kernels.h", "co_store.h")]
PROJ_KERNELS = ("gemm_bf16_kernel", "gemm_wide_kernel", "proj_fused_kernel", "epi_z_kernel",
                "epi_kv_kernel", "z_norm_kernel", "gemm_f32_kernel")
# the attention backward's kernels and sources (its MFMA counters, --only backward)
BWD_SOURCES = [os.path.join(ROOT, "paper_2609_14717_amd", "csrc", f)
               for f in ("backward.hip", "co_device.h", "co_kernels.h")]
BWD_KERNELS = ("bwd_prep_kernel", "bwd_copy_kernel", "bwd_attn_kernel", "bwd_dkv_carry_kernel")
ATTN_KERNELS = ("attn_bf16_kernel", "attn_wave_kernel", "attn_bf16_combine_kernel",
                "attn_group_kernel", "attn_share_merge_kernel")
ATTN_KERNELS_F32 = ("attn_f32_kernel", "attn_chunk_merge_kernel")
ATTN_WARM = 5       # untimed attention calls before the timed ones
COLD_CALLS = 50     # cold calls timed (each after a cache scrub)
TRAIN_ATTN_WARM = 3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="ragged_batch32")
    ap.add_argument("--cpu-baseline-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy-mb", type=int, default=0,
                    help="after the timed region, run one plain copy of this many MiB "
                         "(the reference kernel for byte-counter calibration)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the attention traffic summary from two rocprofv3 --pmc runs "
                         "(FETCH_SIZE, then WRITE_SIZE) and exit")
    ap.add_argument("--summarize-stats", metavar="STATS_CSV",
                    help="write the kernel-time summary of a rocprofv3 --stats run and exit")
    ap.add_argument("--summarize-mfma", metavar="RUN_DIR",
                    help="write the MFMA counter summary of a rocprofv3 --pmc run of "
                         "'--only projection' or '--only prefill' and exit")
    ap.add_argument("--bench-json", metavar="FILE",
                    help="the JSON line the profiled bench command printed (for the summaries)")
    ap.add_argument("--only", choices=("projection", "prefill", "backward"),
                    help="time only carryover_project_kv: the projection of a round's rows "
                         "('projection'), or the whole context as one call ('prefill'); or, "
                         "for the training-shaped workload, only the attention backward "
                         "('backward'); prints one JSON line (the run the MFMA counters are "
                         "taken on)")
    ap.add_argument("--command", default="", help="command recorded in a summary")
    return ap.parse_args()


def source_digest(files):
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def attention_digest():
    return source_digest(ATTN_SOURCES)


def read_summary(path):
    """key: value lines of a committed profile summary."""
    vals = {}
    if os.path.exists(path):
        with open(path) as fh:
            for line in fh:
                if ":" in line and not line.startswith("#"):
                    k, v = line.split(":", 1)
                    vals[k.strip()] = v.strip()
    return vals


def traffic_file(workload):
    return os.path.join(PROFILES, f"attention_traffic_{workload}.txt")


def recorded_traffic(workload, steps, warmup, per_launch):
    """(traffic, profiled): HBM bytes per attention launch from the committed
    counter summary when it was taken on the same kernels at the same chain
    state as this run (same workload, steps and warm-up, same algorithmic
    bytes), else None; ``profiled`` describes the profiled state and its
    measured / algorithmic ratio whenever the kernels match."""
    vals = read_summary(traffic_file(workload))
    if not vals or vals.get("attention_source_digest") != attention_digest():
        return None, None
    try:
        t = float(vals["traffic_bytes_per_launch"])
        a = float(vals["algorithmic_bytes_per_launch"])
        st, wu = int(vals["profiled_steps"]), int(vals["profiled_warmup"])
    except (KeyError, ValueError):
        return None, None
    prof = {"file": os.path.relpath(traffic_file(workload), ROOT), "steps": st, "warmup": wu,
            "traffic_bytes_per_launch": t, "algorithmic_bytes_per_launch": a,
            "ratio": t / a if a else None}
    same = st == steps and wu == warmup and per_launch is not None and abs(a - per_launch) < 0.5
    return (t if same else None), prof


def mfma_file(workload, only):
    return os.path.join(PROFILES, f"mfma_{workload}_{only}.txt")


def mfma_scope(only):
    """(call, kernels, sources digest key, sources) of an MFMA summary."""
    if only == "backward":
        return ("drafter_block_attention_backward", BWD_KERNELS, "backward_source_digest",
                BWD_SOURCES)
    return "carryover_project_kv", PROJ_KERNELS, "projection_source_digest", PROJ_SOURCES


def recorded_mfma(workload, only):
    """Counter figures of the call from the committed MFMA summary, when it was
    taken on the same kernels; else None."""
    path = mfma_file(workload, only)
    vals = read_summary(path)
    _, _, key, sources = mfma_scope(only)
    if not vals or vals.get(key) != source_digest(sources):
        return None
    try:
        return {"file": os.path.relpath(path, ROOT),
                "mfma_busy_frac": float(vals["mfma_busy_frac"]),
                "counted_bf16_flops_per_call": float(vals["counted_bf16_flops_per_call"]),
                "counted_mfma_frac": float(vals["counted_mfma_frac"])}
    except (KeyError, ValueError):
        return None


def attention_window(args):
    """(first, count): the timed stand-alone attention calls among each attention
    kernel's dispatches, in the order bench.py launches them (one dispatch of
    each of the call's kernels per call)."""
    from synth import workloads as wl
    if wl.WORKLOADS[args.workload].anchors:
        return args.warmup + args.steps + TRAIN_ATTN_WARM, min(args.steps, 100)
    return args.warmup + args.steps + ATTN_WARM, args.steps


def _counter_values(run_dir):
    """Counter value of every dispatch, in dispatch order, per (kernel name,
    counter), from a --pmc run."""
    import glob
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    acc = {}
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                per = acc.setdefault((r["Kernel_Name"], r["Counter_Name"]), {})
                did = r["Dispatch_Id"]
                per[did] = per.get(did, 0.0) + float(r["Counter_Value"])
    return {k: [v[d] for d in sorted(v, key=int)] for k, v in acc.items()}


def summarize_pmc(args):
    win = attention_window(args)
    fetch = _counter_values(args.summarize_pmc[0])
    write = _counter_values(args.summarize_pmc[1])
    copy_bytes = args.calibrate_copy_mb * (1 << 20)
    if copy_bytes <= 0:
        raise SystemExit("--calibrate-copy-mb must give the copy size of the profiled runs")

    def one(table, counter, name, window=None):
        """Sum over the kernels matching ``name`` of the mean per dispatch (over
        the window of dispatches if given), and the dispatches averaged."""
        # the plain instantiations only: the EXT ones (last template argument
        # true) serve drafter_block_attention_ext, timed separately
        rows = [v for k, v in table.items()
                if k[1] == counter and name in k[0] and "true>" not in k[0]]
        if not rows:
            raise SystemExit(f"no {counter} rows for {name}")
        tot, cnt = 0.0, 0
        for vals in rows:
            if window is not None:
                vals = vals[window[0]:window[0] + window[1]]
                if len(vals) != window[1]:
                    raise SystemExit(f"{name}: fewer dispatches than the attention window")
            tot += sum(vals) / len(vals)
            cnt += len(vals)
        return tot, cnt

    if not args.bench_json:
        raise SystemExit("--bench-json must give the JSON line of the profiled run")
    bj = load_bench_json(args.bench_json)
    if bj["config"]["workload"] != args.workload or (bj["steps"], bj["warmup"]) != (
            args.steps, args.warmup):
        raise SystemExit("--bench-json is not the line of this workload, steps and warm-up")
    alg = bj["roofline"]["algorithmic_bytes_per_launch"]
    cf, _ = one(fetch, "FETCH_SIZE", "copy16_kernel")
    cw, _ = one(write, "WRITE_SIZE", "copy16_kernel")   # the calibration copy: one dispatch
    f_fac = copy_bytes / (cf * 1024.0)
    w_fac = copy_bytes / (cw * 1024.0)
    lines = [f"# HBM traffic of drafter_block_attention, workload {args.workload}",
             f"command (FETCH_SIZE pass): {args.command.replace('{COUNTER}', 'FETCH_SIZE')}",
             f"command (WRITE_SIZE pass): {args.command.replace('{COUNTER}', 'WRITE_SIZE')}",
             f"attention_source_digest: {attention_digest()}",
             f"profiled_steps: {args.steps}",
             f"profiled_warmup: {args.warmup}",
             f"algorithmic_bytes_per_launch: {alg:.0f}",
             f"dispatches used: {win[1]} of each attention kernel from index {win[0]} (the "
             f"timed stand-alone attention calls on the final state)",
             f"copy_kernel_bytes: {copy_bytes}",
             f"copy FETCH_SIZE KiB: {cf:.1f}  (factor {f_fac:.4f})",
             f"copy WRITE_SIZE KiB: {cw:.1f}  (factor {w_fac:.4f})"]
    tot = 0.0
    for kn in ATTN_KERNELS:
        if not any(k[1] == "FETCH_SIZE" and kn in k[0] for k in fetch):
            continue                            # a kernel this workload does not launch
        kf, nf = one(fetch, "FETCH_SIZE", kn, win)
        kw, nw = one(write, "WRITE_SIZE", kn, win)
        b = kf * 1024.0 * f_fac + kw * 1024.0 * w_fac
        tot += b
        lines.append(f"{kn}: FETCH_SIZE {kf:.1f} KiB/dispatch ({nf} dispatches), "
                     f"WRITE_SIZE {kw:.1f} KiB/dispatch ({nw} dispatches), "
                     f"calibrated {b / 1e6:.3f} MB")
    lines.append(f"traffic_bytes_per_launch: {tot:.0f}")
    lines.append(f"measured / algorithmic: {tot / alg:.3f}")
    os.makedirs(PROFILES, exist_ok=True)
    with open(traffic_file(args.workload), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def load_bench_json(path):
    """The last JSON line of a bench run's output."""
    with open(path) as fh:
        lines = [ln for ln in fh if ln.lstrip().startswith("{")]
    if not lines:
        raise SystemExit(f"no JSON line in {path}")
    return json.loads(lines[-1])


MFMA_GAP_NS = 50_000_000   # the pause bench.py --only leaves before the calls it times


def summarize_mfma(args):
    """MFMA counters of the projection call (or of the attention backward)
    from a rocprofv3 --pmc run (with --kernel-trace) of ``bench.py --only
    ...``: the call's kernel dispatches after the last pause of more than
    50 ms are the warm-up and timed calls (``bench.py --only`` pauses before
    them), all of the same shape.  Per call: the MFMA busy share of the SIMD cycles (rocprofv3's
    MfmaUtil, time-weighted over the dispatches), counted bf16 MFMA flops
    (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512) against the algorithmic flops, and
    the counted rate over the call's event time."""
    import glob
    if not args.bench_json:
        raise SystemExit("--bench-json must give the JSON line of the profiled run")
    bj = load_bench_json(args.bench_json)
    only, ncalls = bj["only"], bj["calls"] + bj["warm"]
    call_name, kernels, digest_key, sources = mfma_scope(only)
    files = glob.glob(os.path.join(args.summarize_mfma, "**", "*counter_collection.csv"),
                      recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {args.summarize_mfma}")
    disp = {}
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if not any(is_kernel(r["Kernel_Name"], k) for k in kernels):
                    continue
                d = disp.setdefault(int(r["Dispatch_Id"]), {
                    "name": r["Kernel_Name"], "grid": int(r["Grid_Size"]),
                    "t0": int(r["Start_Timestamp"]), "t1": int(r["End_Timestamp"])})
                d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    order = sorted(disp.values(), key=lambda d: d["t0"])
    cut = 0
    for i in range(1, len(order)):
        if order[i]["t0"] - order[i - 1]["t1"] > MFMA_GAP_NS:
            cut = i
    window = order[cut:]
    kinds = {}
    for d in window:
        k = kinds.setdefault((d["name"], d["grid"]), {"n": 0, "dur": 0.0, "util_t": 0.0,
                                                     "mops": 0.0})
        dur = (d["t1"] - d["t0"]) / 1e3
        k["n"] += 1
        k["dur"] += dur
        k["util_t"] += d.get("MfmaUtil", 0.0) / 100.0 * dur
        k["mops"] += d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
    if not kinds or any(k["n"] % ncalls for k in kinds.values()):
        raise SystemExit("the dispatches after the pause are not whole calls")
    dur = sum(k["dur"] for k in kinds.values()) / ncalls
    busy = sum(k["util_t"] for k in kinds.values()) / max(sum(k["dur"] for k in kinds.values()),
                                                          1e-12)
    counted = sum(k["mops"] for k in kinds.values()) * 512.0 / ncalls
    ev_s = bj["avg_call_us"] / 1e6
    peak = MFMA_PEAK_TFLOPS["bf16"]
    lines = [f"# MFMA counters of {call_name}, workload {args.workload} ({only})",
             f"command (counter pass): {args.command}",
             f"{digest_key}: {source_digest(sources)}",
             f"call: {bj['call']}",
             f"rows per call: {bj['rows']}",
             f"calls in the window: {ncalls} ({bj['warm']} warm-up + {bj['calls']} timed), "
             f"{len(window)} dispatches",
             f"event time per call (bench line, no profiler): {bj['avg_call_us']:.2f} us",
             f"algorithmic flops per call: {bj['flops_per_call']:.6g}",
             f"algorithmic rate: {bj['tflops']:.1f} TFLOP/s = {bj['mfma_frac']:.3f} of "
             f"{peak:.0f} TFLOP/s",
             "",
             f"{'kernel':80s} {'grid':>9s} {'per call':>8s} {'us(pmc)':>8s} {'MfmaUtil':>8s} "
             f"{'bf16 GFLOP':>10s}"]
    for (kn, grid), k in sorted(kinds.items(), key=lambda x: -x[1]["dur"]):
        short = kn if len(kn) <= 80 else kn[:77] + "..."
        lines.append(f"{short:80s} {grid:9d} {k['n'] // ncalls:8d} {k['dur'] / k['n']:8.2f} "
                     f"{k['util_t'] / max(k['dur'], 1e-12):8.3f} "
                     f"{k['mops'] * 512 / k['n'] / 1e9:10.3f}")
    lines += ["",
              f"kernel time per call under the counters: {dur:.2f} us",
              f"mfma_busy_frac: {busy:.4f}",
              f"counted_bf16_flops_per_call: {counted:.6g}",
              f"counted / algorithmic flops: {counted / bj['flops_per_call']:.3f}",
              f"counted_mfma_frac: {counted / ev_s / 1e12 / peak:.4f}",
              "(mfma_busy_frac: rocprofv3's MfmaUtil -- MFMA busy cycles over the SIMD cycles "
              "of each dispatch -- weighted by dispatch time; counted_mfma_frac: counted bf16 "
              "MFMA flops per call over the call's event time, against the dense bf16 peak)"]
    os.makedirs(PROFILES, exist_ok=True)
    with open(mfma_file(args.workload, only), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def is_kernel(name, kernel):
    return "::" + kernel + "<" in name or "::" + kernel + "(" in name


def summarize_stats(args):
    rows = []
    with open(args.summarize_stats) as fh:
        for r in csv.DictReader(fh):
            rows.append((r["Name"], int(r["Calls"]), float(r["AverageNs"]) / 1e3,
                         float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
                         float(r["Percentage"])))
    rows.sort(key=lambda x: -x[1] * x[2])
    lines = [f"# rocprofv3 kernel statistics, workload {args.workload}",
             f"command: {args.command}",
             "",
             f"{'kernel':90s} {'calls':>6s} {'avg_us':>8s} {'min_us':>8s} {'max_us':>8s} {'pct':>6s}"]
    for n, c, a, lo, hi, pct in rows:
        short = n if len(n) <= 90 else n[:87] + "..."
        lines.append(f"{short:90s} {c:6d} {a:8.2f} {lo:8.2f} {hi:8.2f} {pct:6.2f}")
    # the plain instantiations (the EXT ones, last template argument true, serve
    # drafter_block_attention_ext)
    att = [(k, r) for k in ATTN_KERNELS for r in rows if is_kernel(r[0], k) and "true>" not in r[0]]
    if att:
        lines += ["", "drafter_block_attention, all dispatches = " + " + ".join(
            f"{k} {r[2]:.2f} us" for k, r in att) +
            f" = {sum(r[2] for _, r in att):.2f} us per launch (kernel time, no launch gaps)"]
    trace = os.path.join(os.path.dirname(args.summarize_stats),
                         os.path.basename(args.summarize_stats).replace("kernel_stats",
                                                                        "kernel_trace"))
    if att and os.path.exists(trace):
        first, count = attention_window(args)
        per = {}
        with open(trace) as fh:
            for r in csv.DictReader(fh):
                for k, _ in att:
                    if is_kernel(r["Kernel_Name"], k) and "true>" not in r["Kernel_Name"]:
                        per.setdefault(k, []).append(
                            (int(r["Dispatch_Id"]),
                             (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3))
        parts = []
        for k, _ in att:
            d = [t for _, t in sorted(per.get(k, []))][first:first + count]
            if len(d) == count:
                parts.append((k, float(np.mean(d))))
        if len(parts) == len(att):
            lines.append("drafter_block_attention, the timed stand-alone calls (dispatches "
                         f"{first}..{first + count - 1} of each kernel, from the kernel trace) = " +
                         " + ".join(f"{k} {t:.2f} us" for k, t in parts) +
                         f" = {sum(t for _, t in parts):.2f} us per launch")
    os.makedirs(PROFILES, exist_ok=True)
    out = os.path.join(PROFILES, f"kernel_stats_{args.workload}.txt")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def attention_bytes(w, ctx, carry):
    """Algorithmic HBM bytes of one attention launch: every committed and carry
    key/value row read once per (layer, sequence), queries read once, outputs
    (and fp32 LSE) written once."""
    es = 2 if w.dtype == "bf16" else 4
    kv = int(np.sum(ctx + carry)) * w.L * w.Hkv * w.hd * 2 * es
    q = w.L * w.S * w.B * w.Hq * w.hd * es
    return kv + 2 * q + w.L * w.S * w.B * w.Hq * 4


def train_attention_bytes(w, carried):
    """Algorithmic HBM bytes of the training-shaped attention: every recorded
    position's K/V read once (the blocks of a response share its pages), every
    carry row read once, queries read once, outputs and fp32 LSE written once."""
    es = 2 if w.dtype == "bf16" else 4
    V = w.S * w.anchors
    kv = (w.S * w.seq_len + carried) * w.L * w.Hkv * w.hd * 2 * es
    q = w.L * V * w.B * w.Hq * w.hd * es
    return float(kv + 2 * q + w.L * V * w.B * w.Hq * 4)


def projection_work(w, M):
    """Algorithmic flops and HBM bytes of one carryover_project_kv call over M
    window rows: both products (F over Dcat, then K/V of every layer over d),
    weights and rows read once, K/V rows written once."""
    es = 2 if w.dtype == "bf16" else 4
    flops = 2.0 * M * (w.Dcat * w.d + w.d * w.n_kv)
    nbytes = (w.d * w.Dcat + w.n_kv * w.d + M * w.Dcat + M * w.n_kv) * es
    return flops, float(nbytes)


def attention_flops(w, keys_total):
    """q.k and p.v products of every query row against every key of its KV head."""
    return 2.0 * 2.0 * keys_total * w.L * w.B * w.Hq * w.hd


TIMED_WARM = 3      # untimed calls before the timed ones in timed_calls


def timed_calls(torch, stream, n, call, warm=TIMED_WARM, between=None):
    """Duration (s) of ``call``: n calls, each bracketed by HIP events recorded
    on ``stream`` (``between``, untimed, runs before each), split into 5
    consecutive repeats; the median of the repeats' means (the plain mean
    below 5 calls)."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n)]
    for _ in range(warm):
        call()
    for a, b in ev:
        if between is not None:
            between()
        a.record(stream)
        call()
        b.record(stream)
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in ev]) / 1e3
    if len(t) < 5:
        return float(np.mean(t))
    return float(np.median([np.mean(r) for r in np.array_split(t, 5)]))


def projection_result(w, flops, nbytes, sec, rows=None):
    peak = MFMA_PEAK_TFLOPS[w.dtype]
    tflops = flops / sec / 1e12
    gbs = nbytes / sec / 1e9
    return {"call": "carryover_project_kv", "rows": w.S * w.B if rows is None else rows,
            "flops_per_call": flops,
            "bytes_per_call": nbytes, "avg_call_us": sec * 1e6, "tflops": tflops,
            "mfma_peak_tflops": peak, "mfma_frac": tflops / peak, "gbs": gbs,
            "hbm_frac": gbs / HBM_PEAK_GBS}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, budget_s):
    """The fp64 oracle on this host, on a bounded sample of the same workload:
    for half the budget with numpy's BLAS on all its threads, then for the
    other half on one thread, each from the same initial state.  Serving
    workloads run consecutive full rounds of all sequences, or of two of them
    where the contexts are long (the rate is then scaled to the whole batch:
    sequences are independent); the training-shaped forward runs the anchored
    blocks of one response (scaled to all responses)."""
    import oracle  # noqa: F401  (test infrastructure: CPU baseline leg only)
    from threadpoolctl import threadpool_info, threadpool_limits
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from helpers import OracleRun, OracleTrain

    if w.anchors:
        unit, scale = "forwards/s", 1.0 / w.S
        sample = (f"the second drafter pass of the {w.anchors} anchored blocks of one response "
                  f"(projection of its {w.seq_len} recorded rows, carry rows, block attention; "
                  f"float64), rate scaled to all {w.S} responses")

        def leg(seconds):
            t0 = time.perf_counter()
            n = 0
            while True:
                OracleTrain(w, range(w.anchors))
                n += 1
                if time.perf_counter() - t0 >= seconds:
                    break
            return n, time.perf_counter() - t0
    else:
        long_ctx = w.L * w.ctx_hi * w.Hkv * w.hd > (1 << 24)
        seqs = [0, 1] if long_ctx else list(range(w.S))
        unit, scale = "rounds/s", len(seqs) / w.S
        sample = (f"consecutive full rounds of {w.name} ({len(seqs)} of {w.S} sequences, "
                  f"route+project+attention in float64) from the same initial state"
                  + (", rate scaled to the whole batch" if len(seqs) < w.S else ""))

        def leg(seconds):
            orc = OracleRun(w, seqs=seqs, store=np.float32 if long_ctx else np.float64)
            t0 = time.perf_counter()
            n = 0
            while True:
                orc.round(n)
                n += 1
                if time.perf_counter() - t0 >= seconds:
                    break
            return n, time.perf_counter() - t0

    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    n_all, dt_all = leg(budget_s / 2)
    with threadpool_limits(limits=1):
        n_one, dt_one = leg(budget_s / 2)
    return {"value": n_all / dt_all * scale, "unit": unit, "cores": int(threads),
            "kind": "oracle", "sample": f"{n_all} x " + sample,
            "single_thread": {"value": n_one / dt_one * scale, "steps": n_one},
            "host": {"cpu_model": cpu_model(), "nproc": os.cpu_count(),
                     "affinity": len(os.sched_getaffinity(0)), "blas_threads": int(threads)}}


def main():
    args = parse()
    if args.summarize_pmc:
        return summarize_pmc(args)
    if args.summarize_stats:
        return summarize_stats(args)
    if args.summarize_mfma:
        return summarize_mfma(args)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the drafter step "
              "shards by sequence with no exchange, so multi-GPU runs are not part of this "
              "build", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2609_14717_amd as co
    from synth import workloads as wl
    from synth.scenario import Scenario

    w = wl.WORKLOADS[args.workload]
    if w.anchors:
        return run_train(args, w)
    total = args.warmup + args.steps
    w = w.replace(rounds=max(w.rounds, total))
    torch.cuda.set_device(0)
    sc = Scenario(w)
    stream = torch.cuda.current_stream()
    if args.only:
        return only_projection(args, torch, co, sc, w, stream)

    # pre-stage every round's inputs in HBM
    inputs = [sc.round_inputs(r) for r in range(total)]
    outs = [sc.new_output() for _ in range(2)]
    # host replica of the length bookkeeping (checked against the device afterwards)
    ctx = sc.ctx0.astype(np.int64).copy()
    for r in range(total):
        ctx = ctx + inputs[r][4]

    lib = co.lib()
    import ctypes
    dims_p = ctypes.byref(sc.dims)
    W_p = ctypes.byref(sc.W)
    st_s, rt_s = co.state(sc.st), co.route(sc.rt)
    st_p, rt_p = ctypes.byref(st_s), ctypes.byref(rt_s)
    ws_ptr, ws_n = sc.ws.data_ptr(), sc.ws.numel()
    sptr = stream.cuda_stream
    flags = 0

    def step(r):
        """One chained drafter round: one carryover_round call."""
        hidden, q, draft, target, _ = inputs[r]
        out, lse = outs[r & 1]
        rc = lib.carryover_round(dims_p, W_p, hidden.data_ptr(), draft.data_ptr(),
                                 target.data_ptr(), q.data_ptr(), st_p, rt_p, out.data_ptr(),
                                 lse.data_ptr(), flags, ws_ptr, ws_n, sptr)
        if rc:
            raise RuntimeError(f"carryover_round failed ({rc})")

    def chain(mode_flags):
        """The timed rounds warmup..total-1, chained; wall time (s)."""
        nonlocal flags
        flags = mode_flags
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            step(args.warmup + i)
        torch.cuda.synchronize()
        flags = 0
        return time.perf_counter() - t0

    for r in range(args.warmup):
        step(r)
    torch.cuda.synchronize()
    # lengths after the warm-up rounds: restoring them rewinds the chain (rows
    # beyond ctx_len are never read and the carry segment is replaced before it
    # is read, so the timed rounds can be run again from here)
    snap = (sc.st["ctx_len"].clone(), sc.st["carry_len"].clone())

    def rewind():
        sc.st["ctx_len"].copy_(snap[0])
        sc.st["carry_len"].copy_(snap[1])

    dt = chain(0)
    status = co.carryover_read_status(sc.st)
    if status:
        raise RuntimeError(f"device status {co.status_string(status)}")

    # The attention entry point on its own, timed with HIP events on its stream:
    # the same call the rounds make, on the state the chain reached (the round
    # call launches its kernels back to back, so they cannot be bracketed there).
    wsa_ptr, wsa_n = ws_ptr + sc.ws_project, ws_n - sc.ws_project
    q_last = inputs[total - 1][1]
    out, lse = outs[0]

    def attend():
        rc = lib.drafter_block_attention(dims_p, 0, w.L, q_last.data_ptr(), st_p, out.data_ptr(),
                                         lse.data_ptr(), 0, wsa_ptr, wsa_n, sptr)
        if rc:
            raise RuntimeError(f"drafter_block_attention failed ({rc})")

    att_s = timed_calls(torch, stream, args.steps, attend, warm=ATTN_WARM)
    if co.carryover_read_status(sc.st):
        raise RuntimeError("device status after attention")
    ctx_f = sc.st["ctx_len"].cpu().numpy().astype(np.int64)
    car_f = sc.st["carry_len"].cpu().numpy().astype(np.int64)
    assert np.array_equal(ctx_f, ctx), "host replica of the lengths diverged"
    per_launch = float(attention_bytes(w, ctx_f, car_f))
    achieved = per_launch / att_s / 1e9
    traffic, traffic_profiled = recorded_traffic(w.name, args.steps, args.warmup, per_launch)

    # The projection entry point, timed the same way: the last round's rows
    # projected again into the slots they already occupy (same values).
    h_last = inputs[total - 1][0]

    def project():
        rc = lib.carryover_project_kv(dims_p, W_p, h_last.data_ptr(), rt_p, st_p, ws_ptr,
                                      sc.ws_project, sptr)
        if rc:
            raise RuntimeError(f"carryover_project_kv failed ({rc})")

    proj_s = timed_calls(torch, stream, min(args.steps, 100), project)
    pflops, pbytes = projection_work(w, w.S * w.B)

    # Cold: the same calls with a 512 MiB copy (twice the 256 MB Infinity
    # Cache) between them, outside the events, so that no K/V, weight or state
    # byte is served from a cache filled by the previous call.  Attention on
    # the final state first, then the timed rounds again from the snapshot.
    n_cold = min(args.steps, COLD_CALLS)
    scrub = Scrub(torch)
    cold_att_s = timed_calls(torch, stream, n_cold, attend, warm=0, between=scrub)
    rewind()
    cold_r = iter(range(n_cold))
    cold_round_s = timed_calls(torch, stream, n_cold, lambda: step(args.warmup + next(cold_r)),
                               warm=0, between=scrub)
    del scrub

    # t_reuse (the cost of carrying over): the same timed rounds from the same
    # state in Algorithm 1's baseline mode (commit the accepted rows only, no
    # carry segment, no E)
    rewind()
    dt_base = chain(co.CO_BASELINE_MODE)
    if co.carryover_read_status(sc.st):
        raise RuntimeError("device status after baseline rounds")
    assert np.array_equal(sc.st["ctx_len"].cpu().numpy().astype(np.int64), ctx)

    variants = variant_costs(torch, co, sc, w, lib, step, rewind, chain, args, stream, attend,
                             q_last, lse=outs[0][1], dt=dt)
    prefill = prefill_point(torch, co, sc, w) if w.ctx_mode == "projected" else None
    calibrate_copy(torch, args)

    metric = ("drafter rounds/s (block-16) at batch 32" if w.name == "ragged_batch32"
              else f"drafter rounds/s ({w.name})")
    keys = float(np.sum(ctx_f + car_f))
    result = {
        "metric": metric,
        "value": args.steps / dt,
        "unit": "rounds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dt * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "sequences": w.S, "block": w.B, "feat_dim": w.Dcat,
                   "model_dim": w.d, "layers": w.L, "q_heads": w.Hq, "kv_heads": w.Hkv,
                   "head_dim": w.hd, "ctx0": [w.ctx_lo, w.ctx_hi], "accept": list(w.accept),
                   "chained_rounds": total, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm",
                     "kernel": "drafter_block_attention (" + " + ".join(
                         ATTN_KERNELS if w.dtype == "bf16" else ATTN_KERNELS_F32) + ")",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic,
                     "traffic_profiled": traffic_profiled,
                     "algorithmic_bytes_per_launch": per_launch,
                     "avg_launch_us": att_s * 1e6,
                     "tflops": attention_flops(w, keys) / att_s / 1e12,
                     "cold": {"avg_launch_us": cold_att_s * 1e6,
                              "achieved": per_launch / cold_att_s / 1e9,
                              "frac": per_launch / cold_att_s / 1e9 / HBM_PEAK_GBS}},
        "projection": dict(projection_result(w, pflops, pbytes, proj_s),
                           counters=recorded_mfma(w.name, "projection")),
        "cold_round_us": cold_round_s * 1e6,
        "baseline_mode": {"rounds_per_s": args.steps / dt_base,
                          "t_reuse_us": (dt - dt_base) / args.steps * 1e6},
    }
    result["variants"] = variants
    if prefill is not None:
        result["prefill_projection"] = prefill
    add_measured_peaks(result, "hbm")
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w.replace(rounds=w.rounds), args.cpu_baseline_seconds)
    print(json.dumps(result), flush=True)


def add_measured_peaks(result, bound):
    """The achievable HBM read and bf16 MFMA rates measured on this device
    (``synth.device.measured_peaks``), and the roofline and projection
    fractions against them beside those against the spec peaks."""
    from synth import device as sdev
    mp = sdev.measured_peaks()
    result["measured_peaks"] = mp
    r = result["roofline"]
    ref = mp["hbm_read_gbs"] if bound == "hbm" else mp["mfma_bf16_tflops"]
    r["frac_of_measured"] = r["achieved"] / ref
    if "cold" in r:
        r["cold"]["frac_of_measured"] = r["cold"]["achieved"] / ref
    p = result.get("projection")
    if p and "tflops" in p:
        p["mfma_frac_of_measured"] = p["tflops"] / mp["mfma_bf16_tflops"]
    b = result.get("backward")
    if b:
        b["attention_mfma_frac_of_measured"] = b["attention_tflops"] / mp["mfma_bf16_tflops"]


def variant_costs(torch, co, sc, w, lib, step, rewind, chain, args, stream, attend, q_last, lse,
                  dt):
    """Costs of the variants next to the path, on the same state:
    * the separate-projector update and the RMS-normalised updates (F's
      output; every key head): the timed rounds again from the snapshot,
      rounds/s;
    * the attention mass on the carried rows (drafter_carry_mass) and the
      block self-segment merge (drafter_self_merge) after the attention call on
      the final state, per call (the merge repeats on the same output buffer:
      only its time is used)."""
    from synth import device as sdev
    from synth import workloads as wl
    # the rounds read sc.W through a pointer: set its carry projector for them
    wfc = sdev.materialise(w, wl.spec_wfc(w), "cuda")
    sc.W.w_f_carry = wfc.data_ptr()
    rewind()
    dt_sep = chain(0)
    sc.W.w_f_carry = None
    if co.carryover_read_status(sc.st):
        raise RuntimeError("device status after the separate-projector rounds")
    del wfc
    # RMS-normalised F output: the timed rounds again from the snapshot
    off = sdev.materialise(w.replace(dtype="f32"), wl.spec_znorm(w), "cuda")
    gain = torch.tensor(np.float32(w.sigma_z), device="cuda") * (1.0 + off)
    sc.W.z_norm = gain.data_ptr()
    rewind()
    dt_norm = chain(0)
    sc.W.z_norm = None
    if co.carryover_read_status(sc.st):
        raise RuntimeError("device status after the normalised rounds")
    # per-head key normalisation in the K/V epilogue: the timed rounds again
    koff = sdev.materialise(w.replace(dtype="f32"), wl.spec_knorm(w), "cuda")
    kgain = torch.tensor(np.float32(w.sigma_kv), device="cuda") * (1.0 + koff)
    sc.W.k_norm = kgain.data_ptr()
    rewind()
    dt_knorm = chain(0)
    sc.W.k_norm = None
    if co.carryover_read_status(sc.st):
        raise RuntimeError("device status after the key-normalised rounds")
    # the chain ends with carry segments again: the mass of the last attention,
    # and the block's own rows merged in as a third segment
    n = min(args.steps, 100)
    mass = torch.empty_like(lse)
    attend()
    mass_s = timed_calls(torch, stream, n, lambda: co.drafter_carry_mass(
        sc.dims, 0, w.L, q_last, sc.st, lse, mass))
    ks, vs = sc.self_kv(0)
    out = torch.zeros((w.L, w.S, w.B, w.Hq, w.hd), dtype=sc.tdtype, device="cuda")
    self_s = timed_calls(torch, stream, n, lambda: co.drafter_self_merge(
        sc.dims, 0, w.L, q_last, ks, vs, sc.st, out, lse))
    # the same extras inside the one-pass merge: whole attention calls, next
    # to the plain call on the same state
    plain_s = timed_calls(torch, stream, n, lambda: co.drafter_block_attention(
        sc.dims, 0, w.L, q_last, sc.st, out, lse, 0, sc.ws))
    ext = {}
    for name, kv, ms in (("self", (ks, vs), None), ("mass", (None, None), mass),
                         ("self_and_mass", (ks, vs), mass)):
        ext[name + "_call_us"] = 1e6 * timed_calls(
            torch, stream, n, lambda kv=kv, ms=ms: co.drafter_block_attention_ext(
                sc.dims, 0, w.L, q_last, kv[0], kv[1], sc.st, out, lse, ms, 0, sc.ws))
    ext["plain_call_us"] = plain_s * 1e6
    return {"carry_mass_call_us": mass_s * 1e6,
            "self_merge_call_us": self_s * 1e6,
            "attention_ext": ext,
            "separate_projector": {"rounds_per_s": args.steps / dt_sep,
                                   "vs_embedding": dt / dt_sep},
            "z_norm": {"rounds_per_s": args.steps / dt_norm, "vs_plain": dt / dt_norm},
            "k_norm": {"rounds_per_s": args.steps / dt_knorm, "vs_plain": dt / dt_knorm}}


class Scrub:
    """A 512 MiB device copy (torch's copy kernel, so that it is never taken for
    the counter-calibration copy)."""

    def __init__(self, torch):
        n = (512 << 20) // 4
        self.a = torch.ones(n, dtype=torch.float32, device="cuda")
        self.b = torch.empty_like(self.a)

    def __call__(self):
        self.b.copy_(self.a)


def only_projection(args, torch, co, sc, w, stream):
    """``--only``: carryover_project_kv alone, ``args.steps`` calls timed with
    HIP events (after 3 untimed ones): the rows of round 0 projected again into
    the slots they occupy, or the whole initial context as one call."""
    if args.only == "prefill":
        if w.ctx_mode != "projected":
            raise SystemExit(f"{w.name} has no projected context to prefill")
        res = prefill_point(torch, co, sc, w, calls=args.steps, pause_first=True)
    else:
        hidden, q, draft, target, _ = sc.round_inputs(0)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        pause(torch)
        sec = timed_calls(torch, stream, args.steps, lambda: co.carryover_project_kv(
            sc.dims, sc.W, hidden, sc.rt, sc.st, sc.ws, ws_bytes=sc.ws_project))
        flops, nbytes = projection_work(w, w.S * w.B)
        res = projection_result(w, flops, nbytes, sec)
    if co.carryover_read_status(sc.st):
        raise RuntimeError("device status after the projection calls")
    res.update(only=args.only, calls=args.steps, warm=TIMED_WARM, config={"workload": w.name})
    print(json.dumps(res), flush=True)


def pause(torch):
    """A pause of 0.1 s on an idle GPU: marks the start of the calls a counter
    pass summarises."""
    torch.cuda.synchronize()
    time.sleep(0.1)


def prefill_point(torch, co, sc, w, calls=20, pause_first=False):
    """The context projection as one call (every row committed, no E) over the
    initial contexts of all sequences: the rows are projected again into the
    slots they already hold (same values), timed like the other calls."""
    from synth import device as sdev
    from synth import workloads as wl
    n = int(sc.ctx0[0])
    h = torch.empty((w.S, n, w.Dcat), dtype=sc.tdtype, device="cuda")
    for s in range(w.S):
        st_, shape, strides, base, sigma = wl.spec_hctx(w, s, 0, n)
        sdev.fill(h[s], w.key(st_), shape, strides, base, sigma)
    d = sc.dims
    pd = co.make_dims(w.S, n, d.feat_dim, d.model_dim, d.num_layers, d.num_q_heads,
                      d.num_kv_heads, d.head_dim, d.max_pages_per_seq, d.num_pages, d.dtype,
                      d.rope_theta)
    rt = co.alloc_route(w.S, n)
    ws = torch.empty(max(co.workspace_bytes(pd, co.CO_WS_PROJECT), 256), dtype=torch.uint8,
                     device="cuda")
    saved = (sc.st["ctx_len"].clone(), sc.st["carry_len"].clone())
    sc.st["ctx_len"].zero_()
    co.carryover_route(pd, None, None, co.CO_ROUTE_ACCEPT_ALL, sc.st, rt)
    if pause_first:
        pause(torch)
    sec = timed_calls(torch, torch.cuda.current_stream(), calls,
                      lambda: co.carryover_project_kv(pd, sc.W, h, rt, sc.st, ws))
    sc.st["ctx_len"].copy_(saved[0])
    sc.st["carry_len"].copy_(saved[1])
    if co.carryover_read_status(sc.st):
        raise RuntimeError("device status after the prefill projection")
    flops, nbytes = projection_work(w, w.S * n)
    return dict(projection_result(w, flops, nbytes, sec, rows=w.S * n),
                counters=recorded_mfma(w.name, "prefill"))


def calibrate_copy(torch, args):
    """One plain copy of --calibrate-copy-mb MiB: the reference dispatch that the
    HBM counters of a --pmc run are scaled by."""
    if args.calibrate_copy_mb <= 0:
        return
    from synth import device as sdev
    nb = args.calibrate_copy_mb << 20
    src = torch.ones(nb // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    sdev.copy_bytes(dst, src, nb)
    torch.cuda.synchronize()
    del src, dst


def run_train(args, w):
    """The training-shaped forward (second drafter pass of Algorithm 2): one
    step = one forward: K/V of every recorded position of every response
    (committed), every anchored block's rejected rows projected with E into its
    carry segment, then block attention of all blocks."""
    import torch
    import paper_2609_14717_amd as co
    from synth.scenario import TrainScenario
    torch.cuda.set_device(0)
    sc = TrainScenario(w)
    stream = torch.cuda.current_stream()
    V = w.S * w.anchors
    vw = w.replace(S=V)
    wsp = co.workspace_bytes(sc.vdims, co.CO_WS_PROJECT)

    def projection_calls(n):
        """The projection of one forward, each of its two calls timed alone: the
        committed rows of every response (one call, every row committed) and
        the rows of every anchored block (one call, the rejected rows go to the
        block's carry segment, the others are skipped)."""
        pc = timed_calls(torch, stream, n, lambda: co.carryover_project_kv(
            sc.dims, sc.W, sc.h_committed, sc.crt, sc.st, sc.cws))
        pv = timed_calls(torch, stream, n, lambda: co.carryover_project_kv(
            sc.vdims, sc.W, sc.hidden, sc.vrt, sc.vst, sc.ws, ws_bytes=wsp))
        carried = int(sc.vst["carry_len"].sum().item())
        prows = w.S * w.seq_len + carried
        pflops, pbytes = projection_work(vw, prows)
        return pc, pv, prows, dict(
            projection_result(vw, pflops, pbytes, pc + pv, rows=prows),
            call="carryover_project_kv x2 (committed rows; anchored blocks' rows)",
            committed_call_us=pc * 1e6, block_call_us=pv * 1e6,
            rows_computed=w.S * w.seq_len + V * w.B)

    if args.only == "backward":
        return only_backward(args, torch, co, sc, w, stream)
    if args.only:
        if args.only != "projection":
            raise SystemExit(f"{w.name}: only the projection or the backward can be timed alone")
        sc.forward()
        pause(torch)
        *_, res = projection_calls(args.steps)
        if co.carryover_read_status(sc.vst) or co.carryover_read_status(sc.st):
            raise RuntimeError("device status")
        res.update(only=args.only, calls=args.steps, warm=TIMED_WARM,
                   config={"workload": w.name})
        print(json.dumps(res), flush=True)
        return

    for _ in range(args.warmup):
        sc.forward()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        sc.forward()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    if co.carryover_read_status(sc.vst) or co.carryover_read_status(sc.st):
        raise RuntimeError("device status")
    n = min(args.steps, 100)
    att_s = timed_calls(torch, stream, n, lambda: co.drafter_block_attention(
        sc.vdims, 0, w.L, sc.q, sc.vst, sc.out, sc.lse, co.CO_ATTN_SHARED_PREFIX, sc.ws),
        warm=TRAIN_ATTN_WARM)
    pc_s, pv_s, prows, proj = projection_calls(n)
    proj["counters"] = recorded_mfma(w.name, "projection")
    keys = float(np.sum(sc.vst["ctx_len"].cpu().numpy().astype(np.int64) +
                        sc.vst["carry_len"].cpu().numpy().astype(np.int64)))
    carried = int(sc.vst["carry_len"].sum().item())
    aflops = attention_flops(vw, keys)
    abytes = train_attention_bytes(w, carried)
    traffic, traffic_profiled = recorded_traffic(w.name, args.steps, args.warmup, abytes)
    atfl = aflops / att_s / 1e12
    backward = train_backward(torch, co, sc, w, stream, n, args, aflops, prows)
    calibrate_copy(torch, args)
    result = {
        "metric": f"training-shaped forwards/s ({w.name})",
        "value": args.steps / dt,
        "unit": "forwards/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dt * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "responses": w.S, "positions": w.seq_len,
                   "anchored_blocks": V, "block": w.B, "feat_dim": w.Dcat, "model_dim": w.d,
                   "layers": w.L, "q_heads": w.Hq, "kv_heads": w.Hkv, "head_dim": w.hd,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "drafter_block_attention, shared prefixes "
                     "(attn_group_kernel)", "achieved": atfl,
                     "peak": MFMA_PEAK_TFLOPS[w.dtype], "unit": "TFLOP/s",
                     "frac": atfl / MFMA_PEAK_TFLOPS[w.dtype], "traffic": traffic,
                     "traffic_profiled": traffic_profiled,
                     "algorithmic_flops_per_launch": aflops,
                     "algorithmic_bytes_per_launch": abytes, "avg_launch_us": att_s * 1e6},
        "projection": proj,
        "backward": backward,
    }
    add_measured_peaks(result, "mfma")
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_baseline_seconds)
    print(json.dumps(result), flush=True)


def only_backward(args, torch, co, sc, w, stream):
    """``--only backward``: drafter_block_attention_backward alone, ``args.steps``
    calls timed with HIP events after a forward (and 3 untimed calls)."""
    sc.forward()
    attn_bwd, _ = backward_calls(torch, co, sc, w)
    attn_bwd()
    V = w.S * w.anchors
    keys = float(np.sum(sc.vst["ctx_len"].cpu().numpy().astype(np.int64) +
                        sc.vst["carry_len"].cpu().numpy().astype(np.int64)))
    aflops = attention_flops(w.replace(S=V), keys)
    pause(torch)
    sec = timed_calls(torch, stream, args.steps, attn_bwd)
    if co.carryover_read_status(sc.vst):
        raise RuntimeError("device status after the backward")
    peak = MFMA_PEAK_TFLOPS[w.dtype]
    flops = 2.5 * aflops   # S, dP, dV, dK, dQ: 10 hd flops per (query, key)
    res = {"only": "backward", "call": "drafter_block_attention_backward (one group per response)",
           "rows": V * w.B, "calls": args.steps, "warm": TIMED_WARM, "avg_call_us": sec * 1e6,
           "flops_per_call": flops, "tflops": flops / sec / 1e12,
           "mfma_frac": flops / sec / 1e12 / peak, "config": {"workload": w.name}}
    print(json.dumps(res), flush=True)


def backward_calls(torch, co, sc, w):
    """(attention backward, projection backward) of the training-shaped pass as
    closures over freshly zeroed gradient buffers and workspaces."""
    from synth import device as sdev
    from synth import workloads as wl
    V = w.S * w.anchors
    d_out = sdev.materialise(w, wl.spec_dout(w, S=V), "cuda")
    z = lambda t: torch.zeros(t.shape, dtype=torch.float32, device="cuda")
    dk, dv, dkc, dvc = (z(sc.vst["k_cache"]), z(sc.vst["v_cache"]), z(sc.vst["k_carry"]),
                        z(sc.vst["v_carry"]))
    dq = torch.zeros(tuple(sc.q.shape), dtype=torch.float32, device="cuda")
    n_kv = 2 * w.L * w.Hkv * w.hd
    dwf = torch.zeros((w.d, w.Dcat), dtype=torch.float32, device="cuda")
    dwkv = torch.zeros((n_kv, w.d), dtype=torch.float32, device="cuda")
    de = torch.zeros(w.Dcat, dtype=torch.float32, device="cuda")
    wsa = torch.zeros(co.workspace_bytes(sc.vdims, co.CO_WS_ATTENTION_BACKWARD),
                      dtype=torch.uint8, device="cuda")
    wsc = torch.zeros(co.workspace_bytes(sc.dims, co.CO_WS_PROJECT_BACKWARD),
                      dtype=torch.uint8, device="cuda")
    wsv = torch.zeros(co.workspace_bytes(sc.vdims, co.CO_WS_PROJECT_BACKWARD),
                      dtype=torch.uint8, device="cuda")

    def attn_bwd():
        co.drafter_block_attention_backward(sc.vdims, 0, w.L, sc.q, sc.vst, sc.out, sc.lse, d_out,
                                            w.anchors, dq, dk, dv, dkc, dvc, wsa)

    def proj_bwd():
        co.carryover_project_kv_backward(sc.dims, sc.W, sc.h_committed, sc.crt, dk, dv, dkc, dvc,
                                         dwf, dwkv, de, wsc)
        co.carryover_project_kv_backward(sc.vdims, sc.W, sc.hidden, sc.vrt, dk, dv, dkc, dvc,
                                         dwf, dwkv, de, wsv)

    return attn_bwd, proj_bwd


def train_backward(torch, co, sc, w, stream, n, args, aflops, prows):
    """The training side of the same pass (Algorithm 2): the attention backward
    from a seeded output gradient (the blocks of a response share its pages:
    one group per response), then the projection backward of both projection
    calls; each timed alone, and whole training steps (forward + backward)."""
    attn_bwd, proj_bwd = backward_calls(torch, co, sc, w)
    sc.forward()
    ab_s = timed_calls(torch, stream, n, attn_bwd, warm=TRAIN_ATTN_WARM)
    pb_s = timed_calls(torch, stream, n, proj_bwd)
    if co.carryover_read_status(sc.vst):
        raise RuntimeError("device status after the backward")
    steps = max(1, min(args.steps, 20))
    for _ in range(2):
        sc.forward()
        attn_bwd()
        proj_bwd()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        sc.forward()
        attn_bwd()
        proj_bwd()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    abfl = 2.5 * aflops                      # S, dP, dV, dK, dQ: 10 hd flops per (query, key)
    pf, _ = projection_work(w.replace(S=w.S * w.anchors), prows)
    pbfl = 2.0 * pf                          # Z again, dW_KV, dZ, dW_F
    peak = MFMA_PEAK_TFLOPS[w.dtype]
    return {"attention_call": "drafter_block_attention_backward (one group per response)",
            "attention_counters": recorded_mfma(w.name, "backward"),
            "attention_call_us": ab_s * 1e6,
            "attention_algorithmic_flops": abfl,
            "attention_tflops": abfl / ab_s / 1e12,
            "attention_mfma_frac": abfl / ab_s / 1e12 / peak,
            "projection_call": "carryover_project_kv_backward x2 (committed rows; blocks' rows)",
            "projection_us": pb_s * 1e6,
            "projection_algorithmic_flops": pbfl,
            "projection_tflops": pbfl / pb_s / 1e12,
            "projection_mfma_frac": pbfl / pb_s / 1e12 / peak,
            "train_steps_per_s": steps / dt,
            "train_step_ms": dt * 1e3 / steps}


if __name__ == "__main__":
    main()
