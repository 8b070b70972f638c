"""Benchmark of the MuonBP optimizer step on one MI355X.

Workload: one fused attention QKV weight, 2048 x 6144 bf16 (params, grads,
momentum and NS operands), cut into 8 column shards of 2048 x 768 (the
8-way tensor-parallel shard shape), rank-128 synthetic gradients, K = 5
Newton-Schulz iterations, period P = 5 (steps t = 0, 5, 10, ... are full).

A step is one whole optimizer step: momentum, norms, NS (blockwise or full)
and the weight update, all in the HIP library.  Inputs are resident in HBM
before timing starts.  Printed: ONE JSON line (see the keys below).

    python bench.py [--gpus 1] [--steps 100] [--warmup 5] [--no-cpu-baseline]
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

WORKLOAD = "qkv-2048x6144-bf16"
METRIC = "optimizer steps/sec and NS TFLOP/s (% of bf16 MFMA peak), block vs full"
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA, published
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E, published
LR_FULL = 0.02
MU, WD = 0.95, 0.1
# Gradients live in one fixed buffer per matrix, as a training loop's .grad
# tensors do (the step's cost does not depend on their values).
N_GRAD_BUFFERS = 1


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def ns_unit_flops(S, L, K):
    """Algorithmic NS flops of one S x L unit: Gram and A A counted on their
    distinct (symmetric) entries, B Z in full."""
    return K * (S * (S + 1) * L + S * S * (S + 1) + 2 * S * S * L)


def plan_flops(mats, full, K):
    tot = 0.0
    for r, c, gr, gc in mats:
        units = [(r, c)] if full else [(r // gr, c // gc)] * (gr * gc)
        for p, q in units:
            tot += ns_unit_flops(min(p, q), max(p, q), K)
    return tot


def cpu_baseline(mats, period, rank, sample_steps):
    """The fp64 oracle on the host cores over one period of the workload."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import muonbp_oracle as O
    from paper_2510_16981_amd import workload as W

    specs = [O.MatrixSpec(*m) for m in mats]
    gr, gc = mats[0][2], mats[0][3]
    orc = O.MuonBPOracle(specs, O.OracleConfig(period=period, lr_block=LR_FULL / (gr * gc) ** 0.5,
                                               lr_full=LR_FULL, momentum=MU, weight_decay=WD))
    X = [W.quantize(W.init_param(r, c, 0, k), "bf16").double().numpy()
         for k, (r, c, _, _) in enumerate(mats)]
    Gs = [[W.quantize(W.lowrank_grad(r, c, rank, 0, k, t), "bf16").double().numpy()
           for k, (r, c, _, _) in enumerate(mats)] for t in range(sample_steps)]
    t0 = time.perf_counter()
    for t in range(sample_steps):
        X = orc.step(X, Gs[t], t)
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": sample_steps / dt, "unit": "steps/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{sample_steps} consecutive steps (t=0..{sample_steps - 1}: "
                      f"{sum(1 for t in range(sample_steps) if t % period == 0)} full, "
                      f"{sum(1 for t in range(sample_steps) if t % period)} blockwise) of "
                      f"{WORKLOAD}, numpy float64, {dt:.1f} s",
            "host_cpus": len(os.sched_getaffinity(0)), "cpu": platform.processor() or platform.machine()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(blocks of a sharded matrix are processed as a batch on one GPU).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2510_16981_amd import muonbp as mb
    from paper_2510_16981_amd import workload as W

    wl = W.WORKLOADS[WORKLOAD]
    mats = W.workload_matrices(WORKLOAD)
    period, rank, K = wl["period"], wl["rank"], 5
    gr, gc = mats[0][2], mats[0][3]
    lr_block = LR_FULL / (gr * gc) ** 0.5
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    log(f"workload {WORKLOAD}: generating inputs")
    params = [W.quantize(W.init_param(r, c, 0, k), "bf16").cuda() for k, (r, c, _, _) in enumerate(mats)]
    grads = [[W.quantize(W.lowrank_grad(r, c, rank, 0, k, t), "bf16").cuda()
              for k, (r, c, _, _) in enumerate(mats)] for t in range(N_GRAD_BUFFERS)]
    opt = mb.MuonBP(mats, period, lr_block, LR_FULL, MU, WD, options=mb.options_default(ns_steps=K))
    torch.cuda.synchronize()

    t = 0
    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        opt.step(params, grads[t % N_GRAD_BUFFERS], t)
        t += 1
    torch.cuda.synchronize()

    # Timed region: exactly K steps of the schedule, no profiling events.
    log(f"timing {args.steps} steps")
    t_first = t
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        opt.step(params, grads[t % N_GRAD_BUFFERS], t)
        t += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    n_full = sum(1 for s in range(t_first, t) if s % period == 0)

    # Per-kernel pass: the same K steps again with HIP events around every
    # launch (library profiling), split by step kind.
    log("per-kernel pass")
    per = {}
    for kind in ("block", "full"):
        steps_kind = n_full if kind == "full" else args.steps - n_full
        steps_kind = max(steps_kind, 1)
        opt.profile_enable(True)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(steps_kind):
            while (t % period == 0) != (kind == "full"):
                t += 1
            opt.step(params, grads[t % N_GRAD_BUFFERS], t)
            t += 1
        ev1.record(stream)
        prof = opt.profile_read()
        opt.profile_enable(False)
        torch.cuda.synchronize()
        ns_ms = sum(prof[k][0] for k in mb.NS_KINDS)
        ns_launches = sum(prof[k][1] for k in mb.NS_KINDS)
        flops = plan_flops(mats, kind == "full", K) * steps_kind
        info = mb.describe_plan(mats, kind == "full", opt.options)
        per[kind] = {
            "steps": steps_kind,
            "ms_per_step_profiled": ev0.elapsed_time(ev1) / steps_kind,
            "ns_ms_per_step": ns_ms / steps_kind,
            "ns_tflops": flops / (ns_ms * 1e-3) / 1e12,
            "ns_frac_bf16_peak": flops / (ns_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
            "ns_dense_tflops_paper_count": info.ns_dense_flops * steps_kind / (ns_ms * 1e-3) / 1e12,
            "ns_gemm_launches": ns_launches,
            "kernel_ms_per_step": {k: v[0] / steps_kind for k, v in prof.items()},
            "ns_flops_per_step": flops / steps_kind,
        }
    n_el = sum(r * c for r, c, _, _ in mats)
    ew = {}
    for kind, bpe in (("momentum", 6), ("update", 6)):
        ms = (per["block"]["kernel_ms_per_step"][kind] * per["block"]["steps"]
              + per["full"]["kernel_ms_per_step"][kind] * per["full"]["steps"]) / \
             (per["block"]["steps"] + per["full"]["steps"])
        ew[kind] = {"bytes_per_elem": bpe, "gbs": n_el * bpe / (ms * 1e-3) / 1e9,
                    "frac_hbm_peak": n_el * bpe / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                    "note": "footprint fits the 256 MB last-level cache at this size"}

    # Dominant kernel: the grouped NS GEMM (all three NS products), over the
    # whole schedule of the timed region (block and full steps).
    tot_flops = sum(per[k]["ns_flops_per_step"] * per[k]["steps"] for k in per)
    tot_ms = sum(per[k]["ns_ms_per_step"] * per[k]["steps"] for k in per)
    launches = sum(per[k]["ns_gemm_launches"] for k in per)
    achieved = tot_flops / (tot_ms * 1e-3) / 1e12
    roofline = {"kernel": "k_ns_gemm<bf16>", "bound": "mfma", "achieved": achieved,
                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": achieved / BF16_PEAK_TFLOPS,
                "traffic": None, "launches": launches,
                "avg_launch_us": tot_ms * 1e3 / launches,
                "avg_flops_per_launch": tot_flops / launches}

    ms_per_step = elapsed * 1e3 / args.steps
    out = {
        "metric": METRIC, "value": args.steps / elapsed, "unit": "steps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "matrix": "2048x6144", "grid": "1x8", "block": "2048x768",
                   "period": period, "ns_steps": K, "rank": rank, "full_steps_timed": n_full,
                   "parallelism": "none (1 GPU; 8 shards batched)"},
        "block": per["block"], "full": per["full"], "elementwise": ew,
        "roofline": roofline,
    }
    opt.close()
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(mats, period, rank, 3 * period)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
