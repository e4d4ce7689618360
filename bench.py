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

Prints one JSON line (see the repository's benchmark contract) with the
attention kernel's roofline fraction and an fp64 CPU oracle baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="ragged_batch32")
    ap.add_argument("--cpu-baseline-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    return ap.parse_args()


def attention_bytes(w, ctx, carry):
    """Algorithmic HBM bytes of one attention launch: every committed and carry
    key/value row read once per (layer, sequence), queries read once, outputs
    (and fp32 LSE) written once."""
    es = 2 if w.dtype == "bf16" else 4
    kv = int(np.sum(ctx + carry)) * w.L * w.Hkv * w.hd * 2 * es
    q = w.L * w.S * w.B * w.Hq * w.hd * es
    return kv + 2 * q + w.L * w.S * w.B * w.Hq * 4


def cpu_baseline(w, budget_s):
    """The fp64 oracle on this host: full rounds of the same workload."""
    import oracle  # noqa: F401  (test infrastructure: CPU baseline leg only)
    from threadpoolctl import threadpool_info
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from helpers import OracleRun
    orc = OracleRun(w)
    t0 = time.perf_counter()
    n = 0
    while True:
        orc.round(n)
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": n / dt, "unit": "rounds/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n} consecutive full rounds of {w.name} (all {w.S} sequences, "
                      f"route+project+attention in float64) from the same initial state"}


def main():
    args = parse()
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
    total = args.warmup + args.steps
    w = w.replace(rounds=max(w.rounds, total))
    torch.cuda.set_device(0)
    sc = Scenario(w)
    stream = torch.cuda.current_stream()

    # pre-stage every round's inputs in HBM
    inputs = [sc.round_inputs(r) for r in range(total)]
    outs = [sc.new_output() for _ in range(2)]
    # host replica of the length bookkeeping, for the algorithmic byte count
    ctx = sc.ctx0.astype(np.int64).copy()
    att_bytes = []
    for r in range(total):
        m = inputs[r][4]
        ctx = ctx + m
        att_bytes.append(attention_bytes(w, ctx, w.B - m))

    lib = co.lib()
    import ctypes
    dims_p = ctypes.byref(sc.dims)
    W_p = ctypes.byref(sc.W)
    st_s, rt_s = co.state(sc.st), co.route(sc.rt)
    st_p, rt_p = ctypes.byref(st_s), ctypes.byref(rt_s)
    # projection scratch first, then the attention area (as carryover_round lays it out)
    ws_ptr, ws_n = sc.ws.data_ptr(), sc.ws_project
    wsa_ptr, wsa_n = ws_ptr + sc.ws_project, sc.ws.numel() - sc.ws_project
    sptr = stream.cuda_stream
    flags = 0

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]

    def step(r, timed_idx=None):
        hidden, q, draft, target, _ = inputs[r]
        out, lse = outs[r & 1]
        rc = lib.carryover_route(dims_p, draft.data_ptr(), target.data_ptr(), flags, st_p, rt_p,
                                 sptr)
        rc |= lib.carryover_project_kv(dims_p, W_p, hidden.data_ptr(), rt_p, st_p, ws_ptr, ws_n,
                                       sptr)
        if timed_idx is not None:
            ev[timed_idx][0].record(stream)
        rc |= lib.drafter_block_attention(dims_p, 0, w.L, q.data_ptr(), st_p, out.data_ptr(),
                                          lse.data_ptr(), flags, wsa_ptr, wsa_n, sptr)
        if timed_idx is not None:
            ev[timed_idx][1].record(stream)
        if rc:
            raise RuntimeError(f"library call failed ({rc})")

    for r in range(args.warmup):
        step(r)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, i)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    status = co.carryover_read_status(sc.st)
    if status:
        raise RuntimeError(f"device status {co.status_string(status)}")

    att_ms = [a.elapsed_time(b) for a, b in ev]
    att_s = float(np.sum(att_ms)) / 1e3
    timed_bytes = float(np.sum(att_bytes[args.warmup:]))
    achieved = timed_bytes / att_s / 1e9
    per_launch = timed_bytes / args.steps

    result = {
        "metric": "drafter rounds/s (block-16) at batch 32",
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
        "roofline": {"bound": "hbm", "kernel": "drafter_block_attention",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes_per_launch": per_launch,
                     "avg_launch_us": att_s / args.steps * 1e6},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w.replace(rounds=w.rounds), args.cpu_baseline_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
