#!/usr/bin/env python3
"""Benchmark of the sparse APML forward + backward on one MI355X.

One step = apml_forward (with plan) + apml_backward (grad_loss = 1) + plan
release, on the synthetic shape-completion workload: B=32 clouds of
N=M=2048 float32 points (primitive surfaces; prediction = permuted reference
+ N(0, 0.05^2)), 10 Sinkhorn iterations. Inputs are resident on the GPU before
the timed region. Prints ONE JSON line.

  --config k     another workload (1..5) for exploration; the reported line
                 is the default one
  --cpu-baseline off   skip the CPU oracle timing
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "APML fwd+bwd point-pairs/s (B=32, N=M=2048 fp32); peak HBM MB"
# MI355X: 256 CUs x 4 SIMD x 16 lanes at 2.4 GHz, one 32-bit VALU operation per
# lane per clock (packed FP32 not used).
VALU_PEAK_OPS = 256 * 64 * 2.4e9
HBM_PEAK = 8.0e12
# Algorithmic VALU operations per pair and direction of the statistics scan:
# 3 subtractions, 1 multiply, 2 fused multiply-adds (squared distance) and
# min + med3 (running minimum and second minimum).
OPS_PER_PAIR_DIR = 8


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--cpu-baseline", choices=["on", "off"], default="on")
    ap.add_argument("--cpu-repeats", type=int, default=3)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (5 times), to scale HBM byte counters")
    return ap.parse_args()


def copy_calibration(mib: int):
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4, "launches": 5}), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures a single GPU: this build has no multi-GPU path "
              "(the loss shards over the batch with no communication). Run with --gpus 1.",
              file=sys.stderr, flush=True)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return

    import numpy as np
    import torch

    import paper_2512_19743_amd as apml
    from workloads import batch, config

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    apml.load()
    w = config(args.config)
    X, Y = batch(w)
    x = torch.from_numpy(X).cuda()
    y = torch.from_numpy(Y).cuda()
    gl = torch.ones(w.B, device="cuda")
    prm = apml.apml_params_default(n_iter=w.n_iter)

    def step():
        loss, plan = apml.apml_forward(x, y, prm)
        gx, _ = apml.apml_backward(plan, x, y, gl)
        plan.close()
        return loss, gx

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # support size of this workload (diagnostic, outside the timed region)
    loss, plan = apml.apml_forward(x, y, prm)
    nnz = plan.nnz()
    stored = plan.info().stored_pairs
    plan.close()

    apml.apml_profile_reset()
    apml.apml_profile_enable(True)
    apml.apml_reset_peak_memory()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    apml.apml_profile_enable(False)
    ms = e0.elapsed_time(e1) / args.steps
    phases = apml.apml_profile_read()
    mem = apml.apml_get_memory_stats()

    pairs = w.B * w.N * w.M
    value = pairs / (ms * 1e-3)
    # dominant kernel: the statistics scan (one launch per step, both directions)
    stats_ms, stats_n = phases["stats"]
    stats_avg = stats_ms / max(stats_n, 1)
    ops = 2 * pairs * OPS_PER_PAIR_DIR
    achieved = ops / (stats_avg * 1e-3)
    support_ms, support_n = phases["support"]
    support_avg = support_ms / max(support_n, 1)

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "point-pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"config {w.cfg} ({w.name}): B={w.B} N={w.N} M={w.M} L={w.n_iter}, "
                               f"{w.reference} reference, {w.prediction} prediction sigma={w.sigma}",
                   "B": w.B, "N": w.N, "M": w.M, "n_iter": w.n_iter, "tau": 1e-8, "p_min": 0.8},
        "roofline": {
            "kernel": "k_top2 (minimum / second minimum scan, rows and columns)",
            "bound": "alu",
            "achieved": achieved / 1e12,
            "peak": VALU_PEAK_OPS / 1e12,
            "unit": "TOP/s",
            "frac": achieved / VALU_PEAK_OPS,
            "traffic": None,
            "avg_launch_ms": stats_avg,
            "ops_per_launch": ops,
        },
        "peak_hbm_mb": mem["peak_in_use"] / 1e6,
        "support": {"nnz_total": int(nnz.sum()), "nnz_per_row": float(nnz.sum()) / (w.B * w.N),
                    "stored_pairs": int(stored)},
        "phases_ms_per_step": {k: v[0] / args.steps for k, v in phases.items()},
        "support_scan": {"avg_launch_ms": support_avg,
                         "frac_valu": pairs * OPS_PER_PAIR_DIR / (support_avg * 1e-3) / VALU_PEAK_OPS},
        "wall_ms_per_step": wall * 1e3 / args.steps,
    }

    if args.cpu_baseline == "on":
        import oracle

        op = oracle.params(n_iter=w.n_iter)
        if args.config == 2:
            idx = list(range(w.B))
            sample = "the full workload: all 32 samples, forward + backward"
        else:
            idx = [0]
            sample = "sample 0 of the workload, forward + backward"
        times = []
        for _ in range(max(1, args.cpu_repeats)):
            t = time.perf_counter()
            oracle.run_batch(X[idx], Y[idx], op, grad=True)
            times.append(time.perf_counter() - t)
        tc = statistics.median(times)
        line["cpu_baseline"] = {"value": len(idx) * w.N * w.M / tc, "unit": "point-pairs/s",
                                "cores": oracle.max_threads(), "kind": "oracle",
                                "sample": f"{sample}; median of {len(times)} runs, {tc:.2f} s each"}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
