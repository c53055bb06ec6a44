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
# MI355X FP32 vector peak, 157.3 TFLOP/s, in 32-bit VALU lane operations: 128
# lanes per CU per clock (256 CUs, 2.4 GHz; an FMA counts two flops). The
# library does not use packed FP32, so one instruction stream reaches half of
# it (64 lanes per CU per clock, measured); v_min co-issues with other VALU
# work, so a mix such as the statistics scan's goes above that half.
VALU_PEAK_OPS = 157.3e12 / 2
HBM_PEAK = 8.0e12
# Algorithmic VALU operations per pair and direction of the statistics scan:
# 3 subtractions, 1 multiply, 2 fused multiply-adds (squared distance) and
# min + med3 (running minimum and second minimum).
OPS_PER_PAIR_DIR = 8


# Algorithmic work of each phase of one step, per launch (the library records
# one HIP event pair per phase on its stream). Dense phases count VALU
# operations per point pair; sparse phases count bytes per stored entry of the
# support (nnz after symmetrization), as the method must move them at least
# once: emission of the row-major structure 16 B, column-major view 32 B,
# softmaxes 24 B, Sinkhorn 8 B per entry and half-step forward (+8 B for the
# loss) and 16 B per entry and half-step in reverse, softmax/temperature
# adjoint 24 B + distance gradient 8 B.
# The dense phases count the pairs their scans evaluate (every pair in the
# full scans; the skipping scans of large samples skip pairs that cannot
# matter and report how many they evaluated).
def _ops(per_pair, which):
    return lambda w, scanned, nnz: per_pair * scanned[which]


def _bytes(per_entry_fn):
    return lambda w, scanned, nnz: per_entry_fn(w) * nnz


PHASE_MODEL = {
    "stats": ("alu", _ops(OPS_PER_PAIR_DIR, 0), "VALU ops",
              {"full": "k_top2: minimum and second minimum of every row and column",
               "skip": "k_spatial_sort + k_cull_top2: curve order, then the minima over the runs that can matter"}),
    "support": ("alu", _ops(OPS_PER_PAIR_DIR, 1), "VALU ops",
                {"full": "k_emit: radius test of every pair, counts and staged hits of the candidate support",
                 "skip": "k_cull_emit: radius test over the runs that can matter, counts and staged hits"}),
    "build": ("hbm", _bytes(lambda w: 16), "bytes",
              {"full": "k_emit_compact_place: row-major structure from the staged hits, placement of the Sinkhorn pieces",
               "skip": "k_cull_order_place: row-major structure from the staged hits, placement of the Sinkhorn pieces"}),
    "softmax": ("hbm", _bytes(lambda w: 32 + 24), "bytes",
                "k_csc_rows + k_col_softmax: column-major view, Eq. 1, Eq. 2, P0 (written into the Sinkhorn pieces)"),
    "sinkhorn": ("hbm", _bytes(lambda w: 2 * w.n_iter * 8 + 8), "bytes",
                 "k_sinkhorn_fwd: L Sinkhorn iterations (Eq. 3, Eq. 4) and the loss"),
    "bwd_sinkhorn": ("hbm", _bytes(lambda w: 2 * w.n_iter * 16), "bytes",
                     "k_sinkhorn_bwd: reverse Sinkhorn sweeps"),
    "bwd_softmax": ("hbm", _bytes(lambda w: 24 + 8), "bytes",
                    "softmax and temperature adjoints, distance gradient (Eq. 5)"),
}

# HBM bytes per launch measured with rocprofv3 counters (FETCH_SIZE and
# WRITE_SIZE, KiB per dispatch, each scaled by the same counter's reading for
# a plain device copy of known size), summed over the phase's kernels. Each
# entry names the source files it was measured on with their SHA-256: once a
# file changes, traffic is reported as null until measured again.
TRAFFIC = {
    "stats": {"sources": {"paper_2512_19743_amd/csrc/dense.hip": "3cb072cf5cb664e8cbe1f5d54d9ee9109ac4162a21dd1abcb1c3bfe4420ac13b", "paper_2512_19743_amd/csrc/apml_internal.h": "b3585ddee1fa29ad500cf288d62b310cc25baf2041eed550aac54c3fdf63837f", "paper_2512_19743_amd/csrc/device_common.h": "4de73120c421b7e0af9f71c422c6f85ac615a9d9154719f1a1158a98c87c89a7"}, "kernels": ["k_top2"], "bytes_per_launch": 32794531},
    "support": {"sources": {"paper_2512_19743_amd/csrc/dense.hip": "3cb072cf5cb664e8cbe1f5d54d9ee9109ac4162a21dd1abcb1c3bfe4420ac13b", "paper_2512_19743_amd/csrc/apml_internal.h": "b3585ddee1fa29ad500cf288d62b310cc25baf2041eed550aac54c3fdf63837f", "paper_2512_19743_amd/csrc/device_common.h": "4de73120c421b7e0af9f71c422c6f85ac615a9d9154719f1a1158a98c87c89a7"}, "kernels": ["k_emit"], "bytes_per_launch": 32857993},
    "build": {"sources": {"paper_2512_19743_amd/csrc/dense.hip": "3cb072cf5cb664e8cbe1f5d54d9ee9109ac4162a21dd1abcb1c3bfe4420ac13b", "paper_2512_19743_amd/csrc/pieces.h": "f583f03e18c705c400d730c1898150e41963388a2bc4895a88aca2cb4a0f625b", "paper_2512_19743_amd/csrc/apml_internal.h": "b3585ddee1fa29ad500cf288d62b310cc25baf2041eed550aac54c3fdf63837f", "paper_2512_19743_amd/csrc/device_common.h": "4de73120c421b7e0af9f71c422c6f85ac615a9d9154719f1a1158a98c87c89a7"}, "kernels": ["k_emit_compact_place"], "bytes_per_launch": 23189412},
    "softmax": {"sources": {"paper_2512_19743_amd/csrc/softmax.hip": "083b4fd2edd2980ac8cfd94a426dbcdb3c2e0009101b2824711be304ce307d34", "paper_2512_19743_amd/csrc/apml_internal.h": "b3585ddee1fa29ad500cf288d62b310cc25baf2041eed550aac54c3fdf63837f", "paper_2512_19743_amd/csrc/device_common.h": "4de73120c421b7e0af9f71c422c6f85ac615a9d9154719f1a1158a98c87c89a7"}, "kernels": ["k_csc_rows", "k_col_softmax"], "bytes_per_launch": 45071558},
    "sinkhorn": {"sources": {"paper_2512_19743_amd/csrc/sinkhorn.hip": "4c802f43f25de7177c72507d1ed13422c43d16c1647567695adad8abc2a7eb9b", "paper_2512_19743_amd/csrc/pieces.h": "f583f03e18c705c400d730c1898150e41963388a2bc4895a88aca2cb4a0f625b", "paper_2512_19743_amd/csrc/apml_internal.h": "b3585ddee1fa29ad500cf288d62b310cc25baf2041eed550aac54c3fdf63837f", "paper_2512_19743_amd/csrc/device_common.h": "4de73120c421b7e0af9f71c422c6f85ac615a9d9154719f1a1158a98c87c89a7"}, "kernels": ["k_sinkhorn_fwd"], "bytes_per_launch": 26081540},
    "bwd_sinkhorn": {"sources": {"paper_2512_19743_amd/csrc/sinkhorn.hip": "4c802f43f25de7177c72507d1ed13422c43d16c1647567695adad8abc2a7eb9b", "paper_2512_19743_amd/csrc/pieces.h": "f583f03e18c705c400d730c1898150e41963388a2bc4895a88aca2cb4a0f625b", "paper_2512_19743_amd/csrc/apml_internal.h": "b3585ddee1fa29ad500cf288d62b310cc25baf2041eed550aac54c3fdf63837f", "paper_2512_19743_amd/csrc/device_common.h": "4de73120c421b7e0af9f71c422c6f85ac615a9d9154719f1a1158a98c87c89a7"}, "kernels": ["k_sinkhorn_bwd"], "bytes_per_launch": 26068935},
    "bwd_softmax": {"sources": {"paper_2512_19743_amd/csrc/softmax.hip": "083b4fd2edd2980ac8cfd94a426dbcdb3c2e0009101b2824711be304ce307d34", "paper_2512_19743_amd/csrc/apml_internal.h": "b3585ddee1fa29ad500cf288d62b310cc25baf2041eed550aac54c3fdf63837f", "paper_2512_19743_amd/csrc/device_common.h": "4de73120c421b7e0af9f71c422c6f85ac615a9d9154719f1a1158a98c87c89a7"}, "kernels": ["k_bwd_col_softmax", "k_bwd_row_softmax"], "bytes_per_launch": 33356621},
}


def _sha(path):
    import hashlib

    with open(os.path.join(ROOT, path), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_for(phase, d):
    t = TRAFFIC.get(phase)
    if not t or any(_sha(src) != h for src, h in t["sources"].items()):
        return None
    return t["bytes_per_launch"]


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--scan", choices=["auto", "full", "skip"], default="auto",
                    help="how the dense scans visit the pairs (identical results)")
    ap.add_argument("--cpu-baseline", choices=["on", "off"], default="on")
    ap.add_argument("--cpu-repeats", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--memory-sweep", action="store_true",
                    help="only measure peak library memory and time of one forward+backward at B=1, "
                         "N=M in 1k..256k (shape-completion generator), one JSON line per size, with the "
                         "stored pairs of 16 seeded samples per size")
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


def memory_sweep():
    """Peak device memory held by the library (plan + scratch) and time of one
    forward+backward at B = 1 as N = M grows; a least-squares line in N + M
    gives the bytes per point."""
    import numpy as np
    import torch

    import paper_2512_19743_amd as apml
    from workloads import custom

    apml.load()
    sizes = [1024, 2048, 4096, 8192, 16384, 32768, 65536, 131072, 262144]
    trials = 16
    pts, peaks = [], []
    for n in sizes:
        X, Y = custom(n, 1, n, n, reference="primitives", prediction="perm_noise", sigma=0.05)
        x = torch.from_numpy(X).cuda()
        y = torch.from_numpy(Y).cuda()
        gl = torch.ones(1, device="cuda")
        prm = apml.apml_params_default(n_iter=10)

        def step():
            loss, plan = apml.apml_forward(x, y, prm)
            apml.apml_backward(plan, x, y, gl)
            nnz = int(plan.nnz().sum())
            plan.close()
            return nnz

        step()
        torch.cuda.synchronize()
        apml.apml_release_cached_memory()
        step()  # warm again with blocks sized for this N only
        torch.cuda.synchronize()
        apml.apml_reset_peak_memory()
        times = []
        for _ in range(3):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            loss, plan = apml.apml_forward(x, y, prm)
            apml.apml_backward(plan, x, y, gl)
            e1.record()
            torch.cuda.synchronize()
            nnz = int(plan.nnz().sum())
            plan.close()
            times.append(e0.elapsed_time(e1))
        peak = apml.apml_get_memory_stats()["peak_in_use"]
        pts.append(2 * n)
        peaks.append(peak)
        # stored pairs over several seeded samples of the same size (one batched forward)
        Xt, Yt = custom(n, trials, n, n, reference="primitives", prediction="perm_noise", sigma=0.05)
        _, plan = apml.apml_forward(torch.from_numpy(Xt).cuda(), torch.from_numpy(Yt).cuda(), prm)
        per = plan.nnz().astype(np.float64)
        plan.close()
        torch.cuda.synchronize()
        apml.apml_release_cached_memory()  # the batch's blocks would inflate the next size's peak
        # one dense fp32 N x M matrix, the least a dense formulation holds
        print(json.dumps({"N": n, "M": n, "B": 1, "nnz": nnz, "peak_library_mb": peak / 1e6,
                          "bytes_per_point": peak / (2 * n), "dense_matrix_mb": 4.0 * n * n / 1e6,
                          "ms_fwd_bwd": statistics.median(times), "trials": trials,
                          "nnz_mean": float(per.mean()), "nnz_std": float(per.std(ddof=1)),
                          "nnz_min": int(per.min()), "nnz_max": int(per.max())}), flush=True)
        del x, y, Xt, Yt
    A = np.vstack([np.asarray(pts, float), np.ones(len(pts))]).T
    slope, icpt = np.linalg.lstsq(A, np.asarray(peaks, float), rcond=None)[0]
    print(json.dumps({"fit": "peak_bytes = a * (N + M) + b", "a_bytes_per_point": slope, "b_bytes": icpt}), flush=True)


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
    if args.memory_sweep:
        memory_sweep()
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
    prm = apml.apml_params_default(n_iter=w.n_iter, dense_scan={"auto": 0, "full": 1, "skip": 2}[args.scan])

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
    info = plan.info()
    stored = info.stored_pairs
    scanned = (int(info.scanned_min), int(info.scanned_support))
    plan.close()

    # timed region: K steps, library profiling off
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
    ms = e0.elapsed_time(e1) / args.steps
    mem = apml.apml_get_memory_stats()

    # per-phase split: the same K steps again with HIP events recorded by the
    # library on its stream around each phase
    apml.apml_profile_reset()
    apml.apml_profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    apml.apml_profile_enable(False)
    phases = apml.apml_profile_read()

    pairs = w.B * w.N * w.M
    value = pairs / (ms * 1e-3)
    scan_mode = "skip" if scanned[0] < 2 * pairs else "full"
    nnz_total = int(nnz.sum())
    kernels = {}
    for name, (tot_ms, n) in phases.items():
        if n == 0 or name not in PHASE_MODEL:
            continue
        bound, per, unit_kind, what = PHASE_MODEL[name]
        if isinstance(what, dict):
            what = what[scan_mode]
        avg = tot_ms / n
        work = per(w, scanned, nnz_total)
        achieved = work / (avg * 1e-3)
        peak = VALU_PEAK_OPS if bound == "alu" else HBM_PEAK
        kernels[name] = {"kernel": what, "bound": bound, "avg_launch_ms": avg, "launches_per_step": n / args.steps,
                         "work_per_launch": work, "work_unit": unit_kind,
                         "achieved": achieved / (1e12 if bound == "alu" else 1e9),
                         "unit": "TOP/s" if bound == "alu" else "GB/s", "frac": achieved / peak,
                         "traffic": traffic_for(name, None)}
    dom = max(kernels, key=lambda k: kernels[k]["avg_launch_ms"] * kernels[k]["launches_per_step"])
    d = kernels[dom]
    roofline = {"bound": d["bound"], "achieved": d["achieved"],
                "peak": VALU_PEAK_OPS / 1e12 if d["bound"] == "alu" else HBM_PEAK / 1e9,
                "unit": d["unit"], "frac": d["frac"], "traffic": traffic_for(dom, d),
                "kernel": d["kernel"], "phase": dom, "avg_launch_ms": d["avg_launch_ms"],
                "work_per_launch": d["work_per_launch"], "work_unit": d["work_unit"]}

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
        "config": {"workload": f"{w.name}: B={w.B} N={w.N} M={w.M} L={w.n_iter}, "
                               f"{w.reference} reference, {w.prediction} prediction sigma={w.sigma}",
                   "B": w.B, "N": w.N, "M": w.M, "n_iter": w.n_iter, "tau": 1e-8, "p_min": 0.8,
                   "dense_scan": scan_mode},
        "roofline": roofline,
        "peak_hbm_mb": mem["peak_in_use"] / 1e6,
        "support": {"nnz_total": nnz_total, "nnz_per_row": nnz_total / (w.B * w.N),
                    "stored_pairs": int(stored),
                    "scanned_fraction_min": scanned[0] / (2 * w.B * w.N * w.M),
                    "scanned_fraction_support": scanned[1] / (w.B * w.N * w.M)},
        "phases_ms_per_step": {k: v[0] / args.steps for k, v in phases.items()},
        "kernels": kernels,
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
        t_start = time.perf_counter()
        # at least cpu_repeats runs and about ten seconds of CPU work
        while len(times) < max(1, args.cpu_repeats) or time.perf_counter() - t_start < args.cpu_seconds:
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
