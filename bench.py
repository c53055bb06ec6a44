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
# MI355X published peaks: FP32 vector 157.3 TFLOP/s (256 CUs x 2.4 GHz x 128
# FMA lanes x 2 flops), HBM3E 8 TB/s.
FP32_PEAK_FLOPS = 157.3e12
HBM_PEAK = 8.0e12
# Algorithmic floating-point work of the dense scans: one evaluation of the
# squared distance per pair covers both directions' statistics (and, in the
# support scan, the row's and the column's radius test): 3 subtractions,
# 3 multiplications, 2 additions = 8 FLOPs per pair. The selects (min, med3,
# compares) are not floating-point arithmetic and are not counted. The full
# statistics scan evaluates every pair once for both directions; the VALU
# issue rate it reaches is measured with counters (VALU instructions per CU
# and clock), not here.
FLOPS_PER_PAIR = 8


# Algorithmic work of each phase of one step, per launch (the library records
# one HIP event pair per phase on its stream). Dense phases count FLOPs per
# point pair evaluated; sparse phases count bytes per stored entry of the
# support (nnz after symmetrization), as the method must move them at least
# once: emission of the row-major structure 16 B, column-major view 32 B,
# softmaxes 24 B, Sinkhorn 8 B per entry and half-step forward (+8 B for the
# loss) and 16 B per entry and half-step in reverse, softmax/temperature
# adjoint 24 B + distance gradient 8 B.
# The dense phases count the pairs their scans evaluate, once per pair (every
# pair in the full scans; the skipping scans of large samples skip pairs that
# cannot matter and report how many they evaluated per direction).
def _flops(which, directions):
    return lambda w, scanned, nnz: FLOPS_PER_PAIR * scanned[which] / directions


def _bytes(per_entry_fn):
    return lambda w, scanned, nnz: per_entry_fn(w) * nnz


PHASE_MODEL = {
    "stats": ("alu", _flops(0, 2), "FLOP",
              {"full": "k_top2_pairs: minimum and second minimum of every row and column, each pair evaluated once",
               "skip": "k_spatial_sort + k_cull_top2: curve order, then the minima over the runs that can matter"}),
    "support": ("alu", _flops(1, 1), "FLOP",
                {"full": "k_emit: radius test of every pair, counts and staged hits of the candidate support",
                 "skip": "k_cull_emit: radius test over the runs that can matter, counts and staged hits"}),
    "build": ("hbm", _bytes(lambda w: 16), "bytes",
              {"full": "k_emit_compact_place: row-major structure from the staged hits, placement of the Sinkhorn pieces",
               "skip": "k_cull_order_place: row-major structure from the staged hits, placement of the Sinkhorn pieces"}),
    "softmax": ("hbm", _bytes(lambda w: 32 + 24), "bytes",
                "k_csc_rows + k_col_softmax: column-major view, Eq. 1, Eq. 2, P0 (written into the Sinkhorn pieces)"),
    "sinkhorn": ("hbm", _bytes(lambda w: 2 * w.n_iter * 8 + 8), "bytes",
                 "k_sinkhorn_fwd (clouds up to 2048 points; larger: the streamed or split kernels, or one launch "
                 "per half-sweep): L Sinkhorn iterations (Eq. 3, Eq. 4) and the loss"),
    "bwd_sinkhorn": ("hbm", _bytes(lambda w: 2 * w.n_iter * 16), "bytes",
                     "k_sinkhorn_bwd (clouds up to 2048 points; larger: the streamed or split kernels, or two "
                     "launches per iteration): reverse Sinkhorn sweeps"),
    "bwd_softmax": ("hbm", _bytes(lambda w: 24 + 8), "bytes",
                    "softmax and temperature adjoints, distance gradient (Eq. 5)"),
}

# HBM bytes per launch measured with rocprofv3 counters (FETCH_SIZE and
# WRITE_SIZE, KiB per dispatch, each scaled by the same counter's reading for
# a plain device copy of known size), summed over the phase's kernels, on the
# workload TRAFFIC_WORKLOAD. Each entry names the source files it was
# measured on with their SHA-256: once a file changes, or on another
# workload, traffic is reported as null.
TRAFFIC_WORKLOAD = 2
TRAFFIC = {
    "stats": {"sources": {"paper_2512_19743_amd/csrc/dense.hip": "b8ad8ac7143c0e550506b6e9f041715acbb53afe58979c162835c46acc143f29", "paper_2512_19743_amd/csrc/apml_internal.h": "9de09b22e2bb70db0e738b837406b4c22d17c6c43878bf853591214bca0bb461", "paper_2512_19743_amd/csrc/device_common.h": "03dc51e197a1281c03edf6f18979a0e66674abec0a0da05b91d1f7efd31020c0"}, "kernels": ["k_top2_pairs", "k_finalize"], "bytes_per_launch": 32933544},
    "support": {"sources": {"paper_2512_19743_amd/csrc/dense.hip": "b8ad8ac7143c0e550506b6e9f041715acbb53afe58979c162835c46acc143f29", "paper_2512_19743_amd/csrc/apml_internal.h": "9de09b22e2bb70db0e738b837406b4c22d17c6c43878bf853591214bca0bb461", "paper_2512_19743_amd/csrc/device_common.h": "03dc51e197a1281c03edf6f18979a0e66674abec0a0da05b91d1f7efd31020c0"}, "kernels": ["k_emit"], "bytes_per_launch": 31271543},
    "build": {"sources": {"paper_2512_19743_amd/csrc/dense.hip": "b8ad8ac7143c0e550506b6e9f041715acbb53afe58979c162835c46acc143f29", "paper_2512_19743_amd/csrc/pieces.h": "f583f03e18c705c400d730c1898150e41963388a2bc4895a88aca2cb4a0f625b", "paper_2512_19743_amd/csrc/apml_internal.h": "9de09b22e2bb70db0e738b837406b4c22d17c6c43878bf853591214bca0bb461", "paper_2512_19743_amd/csrc/device_common.h": "03dc51e197a1281c03edf6f18979a0e66674abec0a0da05b91d1f7efd31020c0"}, "kernels": ["k_emit_compact_place"], "bytes_per_launch": 19027330},
    "softmax": {"sources": {"paper_2512_19743_amd/csrc/softmax.hip": "28183ee496ceedff271bcff0dd2c7514af55af7c0c45ec3fb1acfae43e1015fe", "paper_2512_19743_amd/csrc/apml_internal.h": "9de09b22e2bb70db0e738b837406b4c22d17c6c43878bf853591214bca0bb461", "paper_2512_19743_amd/csrc/device_common.h": "03dc51e197a1281c03edf6f18979a0e66674abec0a0da05b91d1f7efd31020c0"}, "kernels": ["k_csc_rows", "k_col_softmax"], "bytes_per_launch": 47747018},
    "sinkhorn": {"sources": {"paper_2512_19743_amd/csrc/sinkhorn.hip": "6a3a219f06db8722ed82302bacadd7d5d9a8d94492632d4a1c2cf2fc4b99ff33", "paper_2512_19743_amd/csrc/pieces.h": "f583f03e18c705c400d730c1898150e41963388a2bc4895a88aca2cb4a0f625b", "paper_2512_19743_amd/csrc/apml_internal.h": "9de09b22e2bb70db0e738b837406b4c22d17c6c43878bf853591214bca0bb461", "paper_2512_19743_amd/csrc/device_common.h": "03dc51e197a1281c03edf6f18979a0e66674abec0a0da05b91d1f7efd31020c0"}, "kernels": ["k_sinkhorn_fwd"], "bytes_per_launch": 26089219},
    "bwd_sinkhorn": {"sources": {"paper_2512_19743_amd/csrc/sinkhorn.hip": "6a3a219f06db8722ed82302bacadd7d5d9a8d94492632d4a1c2cf2fc4b99ff33", "paper_2512_19743_amd/csrc/pieces.h": "f583f03e18c705c400d730c1898150e41963388a2bc4895a88aca2cb4a0f625b", "paper_2512_19743_amd/csrc/apml_internal.h": "9de09b22e2bb70db0e738b837406b4c22d17c6c43878bf853591214bca0bb461", "paper_2512_19743_amd/csrc/device_common.h": "03dc51e197a1281c03edf6f18979a0e66674abec0a0da05b91d1f7efd31020c0"}, "kernels": ["k_sinkhorn_bwd"], "bytes_per_launch": 26059848},
    "bwd_softmax": {"sources": {"paper_2512_19743_amd/csrc/softmax.hip": "28183ee496ceedff271bcff0dd2c7514af55af7c0c45ec3fb1acfae43e1015fe", "paper_2512_19743_amd/csrc/apml_internal.h": "9de09b22e2bb70db0e738b837406b4c22d17c6c43878bf853591214bca0bb461", "paper_2512_19743_amd/csrc/device_common.h": "03dc51e197a1281c03edf6f18979a0e66674abec0a0da05b91d1f7efd31020c0"}, "kernels": ["k_bwd_col_softmax", "k_bwd_row_softmax"], "bytes_per_launch": 33406536},
}


def _sha(path):
    import hashlib

    with open(os.path.join(ROOT, path), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_for(phase, config_index):
    t = TRAFFIC.get(phase)
    if config_index != TRAFFIC_WORKLOAD or not t or any(_sha(src) != h for src, h in t["sources"].items()):
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
                    help="only the scaling study: stored pairs of --trials seeded samples per size and peak "
                         "memory and time of one forward+backward at B=1, N=M in 1k..256k (shape-completion "
                         "generator), dense path beside it up to 64k; one JSON line per size")
    ap.add_argument("--trials", type=int, default=500, help="samples per size of the memory sweep")
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


SWEEP_SIZES = [1024, 2048, 4096, 8192, 16384, 32768, 65536, 131072, 262144]
SWEEP_CHUNK = 32  # trials per batched forward


def _sweep_inputs(job):
    from workloads import custom

    n, chunk_index, count = job
    return custom(n * 1000 + chunk_index, count, n, n, reference="primitives", prediction="perm_noise", sigma=0.05)


def memory_sweep(trials: int):
    """Stored pairs and loss-side memory of the sparse path against the cloud
    size N = M (B = 1 per sample, shape-completion generator, L = 10), with the
    dense path beside it where its N x M matrices fit.

    Per size: the stored pairs after symmetrization (nnz) of `trials` seeded
    samples (mean, spread, range), computed in batched forwards of 32 samples;
    for one sample, the peak device memory of one forward + backward (the
    library's pool, and PyTorch's caching allocator route) and its time; the
    same for the dense path up to 65536 points. A least-squares line in N + M
    gives the sparse path's bytes per point. Inputs are generated first, in a
    process pool, before the GPU is touched."""
    import concurrent.futures
    import multiprocessing

    import numpy as np

    jobs = {n: [(n, c, min(SWEEP_CHUNK, trials - c * SWEEP_CHUNK)) for c in range((trials + SWEEP_CHUNK - 1) // SWEEP_CHUNK)]
            for n in SWEEP_SIZES}
    inputs = {}
    ctx = multiprocessing.get_context("spawn")
    with concurrent.futures.ProcessPoolExecutor(max_workers=min(16, os.cpu_count() or 1), mp_context=ctx) as ex:
        for n in SWEEP_SIZES:
            t = time.perf_counter()
            inputs[n] = list(ex.map(_sweep_inputs, jobs[n]))
            print(json.dumps({"generated": n, "trials": trials, "seconds": time.perf_counter() - t}), flush=True)

    import torch

    import paper_2512_19743_amd as apml

    apml.load()
    prm = apml.apml_params_default(n_iter=10)
    pts, peaks = [], []
    for n in SWEEP_SIZES:
        X, Y = inputs[n][0]
        x = torch.from_numpy(np.ascontiguousarray(X[:1])).cuda()
        y = torch.from_numpy(np.ascontiguousarray(Y[:1])).cuda()
        gl = torch.ones(1, device="cuda")

        def step():
            loss, plan = apml.apml_forward(x, y, prm)
            apml.apml_backward(plan, x, y, gl)
            plan.close()

        def timed(fn, reps):
            fn()
            torch.cuda.synchronize()
            out = []
            for _ in range(reps):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                fn()
                e1.record()
                torch.cuda.synchronize()
                out.append(e0.elapsed_time(e1))
            return statistics.median(out)

        def pool_peak(fn):
            torch.cuda.synchronize()
            apml.apml_release_cached_memory()
            fn()  # blocks sized for this N only
            torch.cuda.synchronize()
            base = apml.apml_get_memory_stats()["in_use"]
            apml.apml_reset_peak_memory()
            fn()
            torch.cuda.synchronize()
            peak = apml.apml_get_memory_stats()["peak_in_use"] - base
            apml.apml_release_cached_memory()
            return peak

        peak = pool_peak(step)
        ms = timed(step, 3)
        peak_torch = torch_peak_bytes(step)
        pts.append(2 * n)
        peaks.append(peak)
        # stored pairs of every trial, in batched forwards
        nnz = []
        for Xc, Yc in inputs[n]:
            _, plan = apml.apml_forward(torch.from_numpy(Xc).cuda(), torch.from_numpy(Yc).cuda(), prm)
            nnz.extend(plan.nnz().tolist())
            plan.close()
        torch.cuda.synchronize()
        apml.apml_release_cached_memory()
        per = np.asarray(nnz, dtype=np.float64)
        rec = {"N": n, "M": n, "B": 1, "trials": len(nnz), "nnz_mean": float(per.mean()),
               "nnz_std": float(per.std(ddof=1)), "nnz_min": int(per.min()), "nnz_max": int(per.max()),
               "nnz_per_point": float(per.mean() / (2 * n)),
               "peak_library_mb": peak / 1e6, "bytes_per_point": peak / (2 * n),
               "peak_torch_mb": peak_torch / 1e6, "ms_fwd_bwd": ms,
               "dense_model_mb": 16.0 * n * n / 1e6}
        # the dense path (P0 and the plan in float32, the adjoint in float64:
        # 16 bytes per pair) where it fits comfortably
        if 16.0 * n * n < 100e9:
            def dstep():
                loss, plan = apml.apml_dense_forward(x, y, prm)
                apml.apml_dense_backward(plan, x, y, gl)
                plan.close()

            dpeak = pool_peak(dstep)
            dms = timed(dstep, 1 if n >= 32768 else 3)
            apml.apml_release_cached_memory()
            rec.update({"dense_peak_mb": dpeak / 1e6, "dense_ms_fwd_bwd": dms,
                        "memory_ratio_dense_over_sparse": dpeak / peak, "time_ratio_dense_over_sparse": dms / ms})
        print(json.dumps(rec), flush=True)
        del x, y
        inputs[n] = None
    A = np.vstack([np.asarray(pts, float), np.ones(len(pts))]).T
    slope, icpt = np.linalg.lstsq(A, np.asarray(peaks, float), rcond=None)[0]
    print(json.dumps({"fit": "peak_bytes = a * (N + M) + b", "a_bytes_per_point": slope, "b_bytes": icpt}), flush=True)


def torch_peak_bytes(step) -> int:
    """Peak device memory of one step with the library's allocations routed to
    PyTorch's caching allocator: max_memory_allocated after a reset, minus what
    was allocated before (inputs and outputs of the caller included only as far
    as the step allocates them)."""
    import gc

    import torch

    import paper_2512_19743_amd as apml

    gc.collect()
    torch.cuda.synchronize()
    # blocks the library's own pool still caches would otherwise be missing
    # from what PyTorch can allocate
    apml.apml_release_cached_memory()
    apml.apml_set_allocator_torch()
    try:
        step()  # warm the caching allocator's blocks
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        before = torch.cuda.memory_allocated()
        step()
        torch.cuda.synchronize()
        return torch.cuda.max_memory_allocated() - before
    finally:
        gc.collect()
        torch.cuda.synchronize()
        apml.apml_set_allocator_default()


def dense_bytes(B, N, M, L, d=3) -> int:
    """Device memory of one dense forward + backward: P0 and the plan (float32)
    and the plan adjoint (float64) per pair, and an upper bound of the
    per-point vectors (statistics, Sinkhorn sums and their products, column
    partial sums)."""
    return 16 * B * N * M + (96 + 16 * (L + 1) + 8 * d * 64) * B * (N + M)


def dense_baseline(x, y, gl, w, sparse_ms, sparse_peak, steps):
    """Dense APML (every pair materialised, Sec. III-A) forward + backward on
    the same batch: median time of a few steps and peak memory (PyTorch's
    caching allocator route), next to the sparse path's. Skipped, with the
    reason, when its matrices do not fit in the free device memory."""
    import gc

    import torch

    import paper_2512_19743_amd as apml

    prm = apml.apml_params_default(n_iter=w.n_iter)
    need = dense_bytes(w.B, w.N, w.M, w.n_iter)
    gc.collect()
    torch.cuda.synchronize()
    apml.apml_release_cached_memory()
    torch.cuda.empty_cache()
    free = torch.cuda.mem_get_info()[0]
    if need > 0.8 * free:
        return {"skipped": f"needs {need / 1e9:.1f} GB of device memory (16 B per pair), "
                           f"{free / 1e9:.1f} GB free", "model_gb": need / 1e9,
                "memory_ratio_dense_over_sparse_model": need / sparse_peak}

    def dstep():
        loss, plan = apml.apml_dense_forward(x, y, prm)
        apml.apml_dense_backward(plan, x, y, gl)
        plan.close()

    dstep()
    torch.cuda.synchronize()
    n = max(3, min(steps, 10))
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(n):
        dstep()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / n
    peak = torch_peak_bytes(dstep)
    torch.cuda.empty_cache()
    return {"ms_per_step": ms, "peak_hbm_mb": peak / 1e6, "steps": n, "model_gb": need / 1e9,
            "time_ratio_dense_over_sparse": ms / sparse_ms, "memory_ratio_dense_over_sparse": peak / sparse_peak,
            "what": "apml_dense_forward + apml_dense_backward: P0, the plan and its adjoint as N x M matrices"}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def dense_oracle_tiny() -> dict:
    """The dense float64 PyTorch formulation (oracle/dense.py) with autograd on
    the tiny workload (2 clouds of 256 points), forward + backward."""
    import torch

    from oracle.dense import dense_apml
    from workloads import batch, config

    w = config(1)
    X, Y = batch(w)
    times = []
    for _ in range(3):
        t = time.perf_counter()
        for b in range(w.B):
            xb = torch.from_numpy(X[b].astype("float64")).requires_grad_(True)
            yb = torch.from_numpy(Y[b].astype("float64")).requires_grad_(True)
            loss, _ = dense_apml(xb, yb, n_iter=w.n_iter)
            loss.backward()
        times.append(time.perf_counter() - t)
    tc = statistics.median(times)
    return {"value": w.pairs / tc, "unit": "point-pairs/s", "threads": torch.get_num_threads(),
            "sample": f"tiny workload (B=2, N=M=256), forward + backward with autograd; median of 3, {tc:.3f} s"}


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
        memory_sweep(args.trials)
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

    # peak loss-side memory through PyTorch's caching allocator: the library
    # routed to it, peak statistics reset, one step, max_memory_allocated
    # above what was allocated before
    peak_torch = torch_peak_bytes(step)

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
        peak = FP32_PEAK_FLOPS if bound == "alu" else HBM_PEAK
        kernels[name] = {"kernel": what, "bound": bound, "avg_launch_ms": avg, "launches_per_step": n / args.steps,
                         "work_per_launch": work, "work_unit": unit_kind,
                         "achieved": achieved / (1e12 if bound == "alu" else 1e9),
                         "unit": "TFLOP/s" if bound == "alu" else "GB/s", "frac": achieved / peak,
                         "traffic": traffic_for(name, args.config)}
    dom = max(kernels, key=lambda k: kernels[k]["avg_launch_ms"] * kernels[k]["launches_per_step"])
    d = kernels[dom]
    roofline = {"bound": d["bound"], "achieved": d["achieved"],
                "peak": FP32_PEAK_FLOPS / 1e12 if d["bound"] == "alu" else HBM_PEAK / 1e9,
                "unit": d["unit"], "frac": d["frac"], "traffic": traffic_for(dom, args.config),
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
        "peak_hbm_mb": peak_torch / 1e6,
        "peak_hbm_mb_pool": mem["peak_in_use"] / 1e6,
        "support": {"nnz_total": nnz_total, "nnz_per_row": nnz_total / (w.B * w.N),
                    "stored_pairs": int(stored),
                    "scanned_fraction_min": scanned[0] / (2 * w.B * w.N * w.M),
                    "scanned_fraction_support": scanned[1] / (w.B * w.N * w.M)},
        "phases_ms_per_step": {k: v[0] / args.steps for k, v in phases.items()},
        "kernels": kernels,
        "wall_ms_per_step": wall * 1e3 / args.steps,
    }

    # the dense formulation (Sec. III-A) on the same batch: time and peak memory
    line["dense_baseline"] = dense_baseline(x, y, gl, w, ms, peak_torch, args.steps)

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
                                "sample": f"{sample}; median of {len(times)} runs, {tc:.2f} s each",
                                "cpu_model": cpu_model(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
                                "dense_float64_oracle_tiny": dense_oracle_tiny()}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
