#!/usr/bin/env python3
"""Benchmark of one partition's PipeGCN training step on one MI355X.

Default workload: one of 4 partitions of a 233K-node dense-community graph
(58,000 inner nodes, ~30,000 boundary nodes, power-law degree with mean row
length ~495 and max ~18.6K, 602-dim features, 4 GCN layers 602-256-256-256-41,
softmax cross-entropy, fp32 update GEMMs, fp32 aggregation), PipeGCN-GF
(smoothing of stale features and gradients, decay 0.95), stale-buffer
refills on a side stream.  One "step" is one full iteration of Algorithm 1
for the partition: forward, loss, backward, stale-gradient accumulation,
smoothing, packing, refills and the SGD update.

Prints ONE JSON line.  ``value`` = partition train-steps/s with all inputs
resident in HBM.  ``roofline`` is computed for the kernel with the largest
total time, from per-launch durations measured with HIP events recorded on
the launch stream during the timed steps.  ``cpu_baseline`` is the fp64
oracle's per-partition step timed on the host for a bounded sample of the
same workload, scaled to the full partition.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
# fp32 GEMMs by parts: six bf16 part products per fp32 product on the bf16 matrix cores
F32_PARTS_CEILING_TFLOPS = MFMA_PEAK_TFLOPS["bf16"] / 6


def f32_gemm_method() -> str:
    """The library's fp32 GEMM path: exact bf16 parts (default) or the fp32 matrix cores."""
    return "fp32-matrix-cores" if os.environ.get("PGCN_GEMM_F32") == "native" else "bf16-parts-x6"
XGMI_LINK_GBPS = 153.0                   # one xGMI link of MI355X, per direction
VARIANTS = {"PipeGCN": (False, False), "PipeGCN-G": (False, True), "PipeGCN-F": (True, False),
            "PipeGCN-GF": (True, True)}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_work(tr, w, model="gcn"):
    """Per-step algorithmic bytes / flops of each kernel kind.

    Aggregation, compulsory model: every index once, every input feature row
    once, every output row once.  Gather model: every non-zero gathers one
    full input row.  GEMMs: 2*M*N*K flops of the products the layer forms
    (a transform-first GraphSAGE layer adds its self term X_in W_bot over the
    inner rows to P (X W_top) over inner and boundary rows).
    """
    from paper_2203_10428_amd import binding as B
    i = tr.info
    n, b, e = i["n_inner"], i["n_bd"], i["nnz"]
    items, items_t = i["spmm_items"], i["spmmt_items"]
    L, wd = tr.L, tr.widths
    bf16 = w.gemm_dtype == "bf16"
    k = 2 if model == "sage" else 1          # GraphSAGE's update takes CONCAT(z, h): K = 2 f
    f4 = lambda f: (f + 3) // 4 * 4
    out = {k: 0.0 for k in ("agg_fwd", "agg_bwd", "agg_fwd_gather", "agg_bwd_gather", "gemm_fwd", "gemm_dgrad",
                            "gemm_wgrad", "gemm_fwd_bytes", "gemm_dgrad_bytes", "gemm_wgrad_bytes")}
    idx, idx_t = e * 4 + items * 16, e * 4 + items_t * 16
    s = i["n_send"]
    ea = 2 if bf16 else 4                    # bytes per activation element the GEMM reads where a bf16 copy exists
    ew = 2 if bf16 else 4                    # packed weights
    for l in range(1, L + 1):
        f, fo = wd[l - 1], wd[l]
        send = s * fo * 4 if l < L else 0    # the forward GEMM's epilogue also writes the next layer's sent rows
        if tr.order[l] == B.PGCN_ORDER_TRANSFORM:
            # P (H W): the aggregations move f_out-wide rows (Y forward, T = P^T M backward, at every
            # layer), and the GEMMs run over the n + b inner and boundary rows
            out["agg_fwd"] += idx + (n + b) * f4(fo) * 4 + n * f4(fo) * 4
            out["agg_fwd_gather"] += idx + e * f4(fo) * 4 + n * f4(fo) * 4
            out["agg_bwd"] += idx_t + n * f4(fo) * 4 + (n + b) * f4(fo) * 4
            out["agg_bwd_gather"] += idx_t + e * f4(fo) * 4 + (n + b) * f4(fo) * 4
            self_term = 2.0 * n * f * fo if model == "sage" else 0.0
            out["gemm_fwd"] += 2.0 * (n + b) * f * fo + self_term
            out["gemm_wgrad"] += 2.0 * (n + b) * f * fo + self_term
            # compulsory bytes: fp32 operands read once (rounded while staged on the bf16 path), output once
            out["gemm_fwd_bytes"] += (n + b) * f * 4 + k * f * fo * ew + (n + b) * fo * 4
            out["gemm_wgrad_bytes"] += (n + b) * (f + fo) * 4 + f * fo * 4
            if l > 1:
                out["gemm_dgrad"] += 2.0 * (n + b) * f * fo + self_term
                out["gemm_dgrad_bytes"] += (n + b) * (fo + f) * 4 + k * f * fo * ew
            continue
        out["agg_fwd"] += idx + (n + b) * f * 4 + n * f4(f) * (6 if bf16 else 4)
        out["agg_fwd_gather"] += idx + e * f4(f) * 4 + n * f4(f) * (6 if bf16 else 4)
        out["gemm_fwd"] += 2.0 * n * k * f * fo
        out["gemm_wgrad"] += 2.0 * n * k * f * fo
        out["gemm_fwd_bytes"] += n * k * f * ea + k * f * fo * ew + n * fo * 4 + send
        # A, J and the mask source H read once; dW written once; bf16 path with an input gradient
        # also writes the masked operand as bf16
        out["gemm_wgrad_bytes"] += n * k * f * ea + 2 * n * fo * 4 + k * f * fo * 4 + \
            (n * fo * 2 if bf16 and l > 1 else 0)
        if l > 1:
            out["agg_bwd"] += idx_t + n * f * 4 + (n + b) * f4(f) * 4
            out["agg_bwd_gather"] += idx_t + e * f4(f) * 4 + (n + b) * f4(f) * 4
            out["gemm_dgrad"] += 2.0 * n * k * f * fo
            out["gemm_dgrad_bytes"] += n * fo * (2 if bf16 else 8) + k * f * fo * ew + n * k * f * 4
    return out


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per step of `kernel` from committed counter runs, if still valid.

    profiles/traffic_<workload>.json holds FETCH_SIZE and WRITE_SIZE summed over
    the kernel's dispatches of one step, scaled by the same counters on a plain
    copy of known size, and the SHA-256 of the kernel, work-plan and stride sources
    they were taken with.  If a source has changed since, the figure no longer
    applies (None).
    """
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    for name, digest in rec["sources"].items():
        src = os.path.join(ROOT, "paper_2203_10428_amd", "csrc", name)
        if hashlib.sha256(open(src, "rb").read()).hexdigest() != digest:
            return None
    return rec["kernels"].get(kernel)


def cpu_baseline(w, scale: float, model: str = "gcn", order: str = "agg", norm: str = "mean"):
    """Time the fp64 oracle's per-partition step (same layer association and normalisation as the
    GPU run) on the whole partition (scale 1) or on a sample of the same graph law."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle.partition import build_partition, propagation_matrix
    from oracle.pipegcn import Options, partition_step
    from paper_2203_10428_amd import configs

    ws = w if scale == 1.0 else configs.with_inner_scale(w, scale)
    g = configs.make_graph(ws)
    d = configs.make_dense(ws, g.n, model=model)
    p = build_partition(g.n, g.rowptr, g.col, g.owner, 0, g.nparts, self_loop=model == "gcn")
    P = propagation_matrix(p, norm)
    rng = np.random.default_rng(7)
    L = w.layers
    recv_f = {l: rng.standard_normal((p.n_bd, w.widths[l - 1])) for l in range(1, L + 1)}
    recv_g = {l: 1e-3 * rng.standard_normal((len(p.send_idx), w.widths[l - 1])) for l in range(2, L + 1)}
    ema_f = {l: np.zeros_like(v) for l, v in recv_f.items()}
    ema_g = {l: np.zeros_like(v) for l, v in recv_g.items()}
    sf, sg = VARIANTS["PipeGCN-GF"]
    opts = Options(smooth_f=sf, smooth_g=sg, gamma=w.gamma, eta=w.eta, loss=w.loss, loss_scale=w.loss_scale,
                   gemm="bf16" if w.gemm_dtype == "bf16" else "f64", order=order, norm=norm)
    if model == "sage":
        opts = Options(**{**opts.__dict__, "model": "sage", "dropout": w.sage_dropout, "optimizer": "adam",
                          "eta": w.sage_lr})
    y = d.labels[p.inner_gid]
    X_in = d.X[p.inner_gid]
    Ws = [x.astype(np.float64) for x in d.W]
    t0 = time.perf_counter()
    partition_step(p, P, X_in, y, Ws, recv_f, recv_g, ema_f, ema_g, 2, opts)
    sec = time.perf_counter() - t0
    reps = 1
    if sec < 1.0:
        # a short step is dominated by first-call costs: time further steps (at least 2 s of them)
        # after this untimed one and report their mean
        reps = min(200, int(2.0 / max(sec, 1e-4)) + 1)
        t0 = time.perf_counter()
        for _ in range(reps):
            partition_step(p, P, X_in, y, Ws, recv_f, recv_g, ema_f, ema_g, 2, opts)
        sec = (time.perf_counter() - t0) / reps
    blas_threads = max([x.get("num_threads", 1) for x in threadpool_info()] or [1])
    return sec, p.n_inner, p.nnz, blas_threads, reps


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="reddit-like-1of4")
    ap.add_argument("--variant", default="PipeGCN-GF", choices=list(VARIANTS))
    ap.add_argument("--model", default="gcn", choices=["gcn", "sage"],
                    help="gcn: Algorithm 1's GCN layer with SGD; sage: the experiments' GraphSAGE layer with the "
                         "setup table's dropout and Adam learning rate")
    ap.add_argument("--order", default="auto", choices=["agg", "transform", "auto"],
                    help="GCN layer association: (P H) W, P (H W), or P (H W) where the layer narrows")
    ap.add_argument("--norm", default="mean", choices=["mean", "sym"],
                    help="GCN propagation matrix: mean D^-1 (A+I) or symmetric D^-1/2 (A+I) D^-1/2")
    ap.add_argument("--no-fuse-pack", action="store_true",
                    help="pack the sent rows in a pass of their own instead of in the kernel writing the layer output")
    ap.add_argument("--cache-layer1", action="store_true",
                    help="variant: keep layer 1's aggregate across steps (constant input features); it reuses "
                         "outputs across steps, so its line is a variant, not the step's measurement")
    ap.add_argument("--no-copy-modes", action="store_true", help="skip the serial / no-refill comparison")
    ap.add_argument("--refill", default="blit", choices=["dma", "blit"], help="engine of the stale-buffer refills")
    ap.add_argument("--remote", default="device", choices=["device", "host"],
                    help="where the emulated peers' data lives: device memory, or pinned host memory (refills "
                         "cross the host link, as in the paper's CPU-staged exchange)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=float, default=None,
                    help="inner-node fraction timed on the CPU (default 1: one step of the whole partition; "
                         "0.1 for the 2M-row stress partition, whose fp64 step needs ~115 GB; 0.15 for the "
                         "GraphSAGE model, whose oracle also draws the dropout masks)")
    ap.add_argument("--out", default=None, help="also write the JSON line to this file")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run 5 plain device copies of BYTES bytes (counter calibration) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n * 4, "copies": 5}))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one partition on one GPU: runs on more than one GPU are not supported "
              "(the multi-partition exchange over xGMI is a design only).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2203_10428_amd import binding as B
    from paper_2203_10428_amd import configs
    from paper_2203_10428_amd.step import PartitionTrainer, StepOptions

    w = configs.WORKLOADS[args.workload]
    t0 = time.perf_counter()
    g = configs.make_graph(w)
    d = configs.make_dense(w, g.n, model=args.model)
    log(f"workload {w.name}: graph {g.stats} generated in {time.perf_counter() - t0:.1f}s")
    sf, sg = VARIANTS[args.variant]
    so = StepOptions(smooth_f=sf, smooth_g=sg, gamma=w.gamma, eta=w.eta, copy_mode="pipe",
                     refill_dma=args.refill == "dma", remote=args.remote, order=args.order, norm=args.norm,
                     cache_layer1=args.cache_layer1, fuse_pack=not args.no_fuse_pack)
    if args.model == "sage":
        so = StepOptions(**{**so.__dict__, "model": "sage", "dropout": w.sage_dropout, "optimizer": "adam",
                            "eta": w.sage_lr})
    tr = PartitionTrainer(g, d.X, d.labels, d.W, w.widths, w.loss, w.loss_scale, w.gemm_dtype, so)
    del d
    log(f"partition set up: {tr.info}")

    def timed(k, mode, per_step_ms=None):
        """Mean wall-clock ms per step over k steps bracketed by device synchronisations; with
        per_step_ms, also each step's time between events recorded on the compute stream."""
        tr.opts.copy_mode = mode
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(k)] if per_step_ms is not None else None
        torch.cuda.synchronize()
        s = time.perf_counter()
        for i in range(k):
            if evs:
                tr.stream.wait_stream(torch.cuda.current_stream())
                evs[i][0].record(tr.stream)
            tr.step()
            if evs:
                evs[i][1].record(tr.stream)
        torch.cuda.synchronize()
        mean = (time.perf_counter() - s) / k * 1e3
        if evs:
            per_step_ms.extend(a.elapsed_time(b) for a, b in evs)
        return mean

    for _ in range(args.warmup):
        tr.step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    def summarise(records, k):
        kinds = {}
        for name, ms, launches in records:     # an aggregation record spans its back-to-back chunk launches
            c = kinds.setdefault(name, [0, 0.0])
            c[0] += launches
            c[1] += ms
        return {n: {"launches": c[0] / k, "ms_per_step": c[1] / k, "avg_launch_ms": c[1] / c[0]}
                for n, c in kinds.items()}

    # per-kernel breakdown (untimed steps, every kind traced) -> the dominant kernel
    kb = 3
    B.pgcn_trace_enable(kb * 512)
    timed(kb, "pipe")
    breakdown = summarise(B.pgcn_trace_collect(kb * 512), kb)
    B.pgcn_trace_disable()
    compute_kinds = ["agg_fwd", "agg_bwd", "gemm_fwd", "gemm_dgrad", "gemm_wgrad"]
    dominant = max((k for k in compute_kinds if k in breakdown), key=lambda k: breakdown[k]["ms_per_step"])

    # timed region: exactly --steps steps; the dominant kernel's launches are
    # bracketed by HIP events on their launch stream (the roofline's durations;
    # aggregation chunk launches of one column range share one pair)
    B.pgcn_trace_enable(max(1024, args.steps * 256))
    B.pgcn_trace_filter([dominant])
    step_events = []
    ms_per_step = timed(args.steps, "pipe", step_events)
    per_step = summarise(B.pgcn_trace_collect(args.steps * 256), args.steps)
    B.pgcn_trace_disable()
    loss = tr.loss.item()
    step_median = float(np.median(step_events))
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step (wall clock), median {step_median:.3f} ms "
        f"(compute-stream events), loss {loss:.6f}")

    work = algorithmic_work(tr, w, args.model)
    dt = "bf16" if w.gemm_dtype == "bf16" else "f32"
    util = {}
    for k in compute_kinds:
        if k not in breakdown:
            continue
        sec = (per_step if k == dominant else breakdown)[k]["ms_per_step"] / 1e3
        if k.startswith("agg"):
            util[k] = {"GBps_compulsory": work[k] / sec / 1e9, "GBps_gather_model": work[k + "_gather"] / sec / 1e9}
        else:
            # the attainable rate is the lower of the matrix-core peak and the product's arithmetic
            # intensity (flops per compulsory byte) times the HBM peak
            ai = work[k] / max(work[k + "_bytes"], 1.0)
            parts = dt == "f32" and f32_gemm_method() == "bf16-parts-x6"
            attain = min(F32_PARTS_CEILING_TFLOPS if parts else MFMA_PEAK_TFLOPS[dt], ai * HBM_PEAK_GBPS / 1e3)
            util[k] = {"TFLOPs": work[k] / sec / 1e12, "mfma_frac": work[k] / sec / 1e12 / MFMA_PEAK_TFLOPS[dt],
                       "flop_per_byte": ai, "attainable_TFLOPs": attain,
                       "frac_attainable": work[k] / sec / 1e12 / attain}
            if parts:
                # fp32-equivalent rate against the ceiling of the by-parts form
                util[k]["parts_ceiling_TFLOPs"] = F32_PARTS_CEILING_TFLOPS
                util[k]["frac_parts_ceiling"] = work[k] / sec / 1e12 / F32_PARTS_CEILING_TFLOPS
    if dominant.startswith("agg"):
        ach = util[dominant]["GBps_compulsory"]
        tr_bytes = measured_traffic(w.name, dominant)
        roof = {"bound": "hbm", "kernel": dominant, "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": ach / HBM_PEAK_GBPS,
                "traffic": None if tr_bytes is None else tr_bytes / per_step[dominant]["launches"],
                "traffic_GBps": None if tr_bytes is None else tr_bytes / (per_step[dominant]["ms_per_step"] / 1e3) / 1e9,
                # counter-measured HBM-side bytes over the same time, against the same peak
                "traffic_frac": None if tr_bytes is None else
                tr_bytes / (per_step[dominant]["ms_per_step"] / 1e3) / 1e9 / HBM_PEAK_GBPS,
                "gather_model_GBps": util[dominant]["GBps_gather_model"],
                "algorithmic_bytes_per_step": work[dominant],
                "launches_per_step": per_step[dominant]["launches"],
                "avg_launch_ms": per_step[dominant]["avg_launch_ms"]}
    else:
        ach = util[dominant]["TFLOPs"]
        roof = {"bound": "mfma", "kernel": dominant, "achieved": ach, "peak": MFMA_PEAK_TFLOPS[dt],
                "unit": "TFLOP/s", "frac": ach / MFMA_PEAK_TFLOPS[dt], "traffic": None,
                "algorithmic_flops_per_step": work[dominant],
                "launches_per_step": per_step[dominant]["launches"],
                "avg_launch_ms": per_step[dominant]["avg_launch_ms"]}

    copy_modes = None
    if not args.no_copy_modes:
        k2 = max(3, args.steps // 2)
        copy_modes = {m: timed(k2, m) for m in ("none", "serial", "pipe")}
        copy_modes["hidden"] = copy_modes["pipe"] <= 1.03 * copy_modes["none"]
        tr.opts.refill_dma = not tr.opts.refill_dma
        copy_modes["pipe_other_engine"] = timed(k2, "pipe")
        copy_modes["refill_engine"] = args.refill
        tr.opts.refill_dma = not tr.opts.refill_dma
        log(f"copy modes (ms/step): {copy_modes}")

    cpu = None
    if not args.no_cpu_baseline:
        try:
            if args.cpu_sample is None:
                args.cpu_sample = 0.15 if args.model == "sage" else (0.1 if w.graph_kind == "rmat" else 1.0)
            sec, n_s, nnz_s, threads, reps = cpu_baseline(w, args.cpu_sample, args.model, args.order, args.norm)
            scale = tr.info["nnz"] / nnz_s
            what = (f"fp64 oracle per-partition step ({args.model}, PipeGCN-GF, t=2)")
            timing = (f"{sec:.2f}s for one step" if reps == 1 else
                      f"{sec * 1e3:.2f} ms per step, the mean of {reps} steps after an untimed one")
            if args.cpu_sample == 1.0:
                what += (f" on the whole partition ({n_s} inner rows, {nnz_s} nnz): {timing}, "
                         f"not extrapolated")
            else:
                what += (f" on the same graph law at {args.cpu_sample:g} of the inner/pool nodes ({n_s} inner rows, "
                         f"{nnz_s} nnz): {timing}; scaled by the nnz ratio {scale:.2f} to the full partition")
            cpu = {"value": 1.0 / (sec * scale), "unit": "steps/s", "cores": threads, "kind": "oracle",
                   "host_cpus": os.cpu_count(), "blas_threads": threads, "sparse_threads": 1,
                   "sample": what + (f"; SciPy's sparse products run single-threaded, the dense products on "
                                     f"{threads} BLAS threads of the host's {os.cpu_count()} CPUs")}
            log(f"cpu baseline: {cpu}")
        except Exception as exc:  # the baseline must never hide the GPU result
            cpu = {"value": None, "unit": "steps/s", "cores": os.cpu_count(), "kind": "oracle",
                   "sample": f"failed: {exc!r}"}

    i = tr.info
    line = {
        "metric": "partition train-steps/sec (fwd+bwd, 4-layer); SpMM HBM GB/s; GEMM MFMA util",
        "value": 1e3 / ms_per_step,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        # per-step time between events recorded on the compute stream around each timed step
        "ms_per_step_median_events": step_median,
        "ms_per_step_events_min_max": [float(np.min(step_events)), float(np.max(step_events))],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic",
        "config": {"workload": w.name, "variant": args.variant,
                   "layer": "graphsage-concat" if args.model == "sage" else "gcn", "remote": args.remote,
                   "optimizer": so.optimizer, "dropout": so.dropout, "copy_mode": "pipe", "refill": args.refill,
                   "order": args.order, "norm": args.norm, "layer1_cached": args.cache_layer1, "pack_fused": not args.no_fuse_pack,
                   "transform_first_layers": [l for l in range(1, tr.L + 1) if tr.order[l] == B.PGCN_ORDER_TRANSFORM],
                   "widths": list(w.widths),
                   "loss": w.loss, "gemm_dtype": w.gemm_dtype, "aggregation_dtype": "f32",
                   "f32_gemm": f32_gemm_method() if w.gemm_dtype != "bf16" else None,
                   "n_inner": i["n_inner"], "n_bd": i["n_bd"], "n_send": i["n_send"], "nnz": i["nnz"],
                   "max_row_len": i["max_row_len"],
                   # the block of P_i (and of P_i^T) aggregated on the matrix cores: rows, columns, non-zeros
                   "dense_block": [i["spmm_hub_rows"], i["spmm_hub_cols"], i["spmm_hub_nnz"]],
                   "dense_block_t": [i["spmmt_hub_rows"], i["spmmt_hub_cols"], i["spmmt_hub_nnz"]],
                   "parallelism": "1 partition / 1 GPU"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "kernels": breakdown,
        "algorithmic_work_per_step": work,
        "utilisation": util,
        "copy_modes_ms_per_step": copy_modes,
        # what the refills move per step, and the time one xGMI link (~153 GB/s) would take for it
        "refill_bytes_per_step": tr.refill_bytes,
        "xgmi_link_ms_per_step": tr.refill_bytes / XGMI_LINK_GBPS / 1e6,
        "loss": loss,
    }
    print(json.dumps(line), flush=True)
    if args.out:
        os.makedirs(os.path.dirname(os.path.abspath(args.out)), exist_ok=True)
        with open(args.out, "w") as f:
            f.write(json.dumps(line) + "\n")


if __name__ == "__main__":
    main()
