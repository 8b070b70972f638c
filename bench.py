"""Benchmark of the MuonBP optimizer step on one MI355X.

Default workload (the one the metric is quoted on): one fused attention QKV
weight, 2048 x 6144 bf16 (params, grads, momentum and NS operands), cut into
8 column shards of 2048 x 768 (the 8-way tensor-parallel shard shape),
rank-128 synthetic gradients, K = 5 Newton-Schulz iterations, period P = 5
(steps t = 0, 5, 10, ... are full).  Other workloads (--workload) are the
larger shapes of the same method: a 16-layer d=2048 model, the 32-layer
8B-shaped model (with a period sweep) and the 4096 x 14336 MLP matrices.

A step is one whole optimizer step: momentum, norms, NS (blockwise or full)
and the weight update, all in the HIP library.  Inputs are resident in HBM
before timing starts.  Printed: ONE JSON line.

    python bench.py [--gpus 1] [--steps 100] [--warmup 5] [--workload NAME]
                    [--period P] [--no-cpu-baseline]
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

DEFAULT_WORKLOAD = "qkv-2048x6144-bf16"
METRIC = "optimizer steps/sec and NS TFLOP/s (% of bf16 MFMA peak), block vs full"
BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA, published
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E, published
LR_FULL = 0.02
MU, WD = 0.95, 0.1
K_NS = 5
# Inputs drawn on the host (exact seeded values) up to this many elements;
# larger models draw timing-only inputs on the GPU.
HOST_INPUT_LIMIT = 64 << 20


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


def cpu_baseline(workload, mats, period, rank, sample_steps):
    """The fp64 oracle on the host cores over `sample_steps` steps of the
    workload (from t = 0, so the sample holds full and block steps)."""
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
    nf = sum(1 for t in range(sample_steps) if period and t % period == 0)
    return {"value": sample_steps / dt, "unit": "steps/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{sample_steps} consecutive steps (t=0..{sample_steps - 1}: {nf} full, "
                      f"{sample_steps - nf} blockwise) of {workload}, numpy float64, {dt:.1f} s",
            "host_cpus": len(os.sched_getaffinity(0)), "cpu": platform.processor() or platform.machine()}


def make_inputs(mats, rank):
    """Params (one per matrix) and grads.  Small workloads: the exact seeded
    host inputs.  Large ones: GPU-drawn timing-only inputs, one gradient
    tensor per distinct shape shared by its matrices (grads are read-only and
    the step's cost does not depend on their values)."""
    import torch
    from paper_2510_16981_amd import workload as W
    n_el = sum(r * c for r, c, _, _ in mats)
    if n_el <= HOST_INPUT_LIMIT:
        params = [W.quantize(W.init_param(r, c, 0, k), "bf16").cuda() for k, (r, c, _, _) in enumerate(mats)]
        grads = [W.quantize(W.lowrank_grad(r, c, rank, 0, k, 0), "bf16").cuda()
                 for k, (r, c, _, _) in enumerate(mats)]
        return params, grads, "synthetic (seeded host draws)"
    params = [W.device_param(r, c, 0, k) for k, (r, c, _, _) in enumerate(mats)]
    by_shape = {}
    grads = []
    for k, (r, c, _, _) in enumerate(mats):
        if (r, c) not in by_shape:
            by_shape[(r, c)] = W.device_grad(r, c, rank, 0, k)
        grads.append(by_shape[(r, c)])
    torch.cuda.synchronize()
    return params, grads, "synthetic (GPU-drawn, one gradient per distinct shape)"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--period", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(blocks of a sharded matrix are processed as a batch on one GPU).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2510_16981_amd import muonbp as mb
    from paper_2510_16981_amd import workload as W

    name = args.workload
    wl = W.WORKLOADS[name]
    mats = W.workload_matrices(name)
    n_el = sum(r * c for r, c, _, _ in mats)
    large = n_el > HOST_INPUT_LIMIT
    steps = args.steps if args.steps is not None else (5 if large else 100)
    warmup = args.warmup if args.warmup is not None else (2 if large else 5)
    period = args.period if args.period is not None else wl["period"]
    rank = wl["rank"]
    gr, gc = mats[0][2], mats[0][3]
    lr_block = LR_FULL / (gr * gc) ** 0.5
    torch.cuda.set_device(0)

    log(f"workload {name}: {len(mats)} matrices, {n_el / 1e6:.1f} M params; generating inputs")
    params, grads, data = make_inputs(mats, rank)
    opt = mb.MuonBP(mats, period, lr_block, LR_FULL, MU, WD, options=mb.options_default(ns_steps=K_NS))
    torch.cuda.synchronize()

    t = 0
    log(f"warmup {warmup} steps")
    for _ in range(warmup):
        opt.step(params, grads, t)
        t += 1
    torch.cuda.synchronize()

    # Timed region: exactly `steps` steps of the schedule, no profiling events.
    log(f"timing {steps} steps")
    t_first = t
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        opt.step(params, grads, t)
        t += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    n_full = sum(1 for s in range(t_first, t) if period > 0 and s % period == 0)

    def next_of_kind(t, full):
        while (period > 0 and t % period == 0) != full:
            t += 1
        return t

    # Step time per kind (no events), then a per-kernel pass with HIP events
    # around every launch (library profiling), per kind.
    per = {}
    for kind in ("block", "full"):
        full = kind == "full"
        if full and period == 0:
            continue
        reps = max(1, min(n_full if full else steps - n_full, 20))
        t = next_of_kind(t, full)
        opt.step(params, grads, t)  # settle after a switch of step kind
        t += 1
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            t = next_of_kind(t, full)
            opt.step(params, grads, t)
            t += 1
        torch.cuda.synchronize()
        ms_step = (time.perf_counter() - t0) * 1e3 / reps
        log(f"per-kernel pass ({kind})")
        opt.profile_enable(True)
        for _ in range(reps):
            t = next_of_kind(t, full)
            opt.step(params, grads, t)
            t += 1
        prof = opt.profile_read()
        opt.profile_enable(False)
        torch.cuda.synchronize()
        ns_ms = sum(prof[k][0] for k in mb.NS_KINDS)
        ns_launches = sum(prof[k][1] for k in mb.NS_KINDS)
        flops = plan_flops(mats, full, K_NS) * reps
        info = mb.describe_plan(mats, full, opt.options)
        per[kind] = {
            "steps": reps,
            "ms_per_step": ms_step,
            "ns_ms_per_step": ns_ms / reps,
            "ns_tflops": flops / (ns_ms * 1e-3) / 1e12,
            "ns_frac_bf16_peak": flops / (ns_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
            "ns_dense_tflops_paper_count": info.ns_dense_flops * reps / (ns_ms * 1e-3) / 1e12,
            "ns_gemm_launches": ns_launches,
            "kernel_ms_per_step": {k: v[0] / reps for k, v in prof.items()},
            "ns_flops_per_step": flops / reps,
            "gemm_tiles": [f"{info.gemm_tile_rows[i]}x{info.gemm_tile_cols[i]}:{info.gemm_tiles[i]}"
                           for i in range(3)],
        }

    kinds = list(per)
    ew = {}
    for kname, bpe in (("momentum", 6), ("update", 6)):
        ms = sum(per[k]["kernel_ms_per_step"][kname] for k in kinds) / len(kinds)
        gbs = n_el * bpe / (ms * 1e-3) / 1e9
        ew[kname] = {"bytes_per_elem": bpe, "gbs": gbs, "frac_hbm_peak": gbs / HBM_PEAK_GBS,
                     "footprint_bytes": n_el * bpe,
                     "note": ("footprint within the 256 MB last-level cache" if n_el * bpe < 256e6
                              else "footprint well beyond the 256 MB last-level cache")}

    # Dominant kernel: the grouped NS GEMM (all three NS products), weighted
    # by the schedule of the timed region (block and full steps).
    wts = {"block": steps - n_full, "full": n_full}
    tot_flops = sum(per[k]["ns_flops_per_step"] * wts[k] for k in kinds)
    tot_ms = sum(per[k]["ns_ms_per_step"] * wts[k] for k in kinds)
    launches = sum(per[k]["ns_gemm_launches"] / per[k]["steps"] * wts[k] for k in kinds)
    achieved = tot_flops / (tot_ms * 1e-3) / 1e12
    roofline = {"kernel": "k_ns_gemm (bf16, all tile shapes)", "bound": "mfma",
                "achieved": achieved, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / BF16_PEAK_TFLOPS, "traffic": None,
                "launches": launches, "avg_launch_us": tot_ms * 1e3 / launches,
                "avg_flops_per_launch": tot_flops / launches}

    out = {
        "metric": METRIC, "value": steps / elapsed, "unit": "steps/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": elapsed * 1e3 / steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": data,
        "config": {"workload": name, "matrices": len(mats), "params": n_el,
                   "grids": sorted({f"{g0}x{g1}" for _, _, g0, g1 in mats}),
                   "period": period, "ns_steps": K_NS, "rank": rank, "full_steps_timed": n_full,
                   "parallelism": "none (1 GPU; shards batched)"},
        "block": per.get("block"), "full": per.get("full"), "elementwise": ew,
        "roofline": roofline,
    }
    if "block" in per and "full" in per:
        tb, tf = per["block"]["ms_per_step"], per["full"]["ms_per_step"]
        out["period_sweep_ms_per_step"] = {
            ("inf" if P == 0 else str(P)): (tb if P == 0 else (tf + (P - 1) * tb) / P)
            for P in W.PERIOD_SWEEP}
        out["period_sweep_note"] = ("(t_full + (P - 1) t_block) / P from the measured block and "
                                    "full step times; P = 1 is Muon, inf is BlockMuon")
    opt.close()
    if not args.no_cpu_baseline and not large:
        log("cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(name, mats, period, rank, 3 * max(period, 1))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
