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

Counter support (the roofline's `traffic`): `--copy-probe MIB` runs only a
streaming kernel of known size, and `--ingest-traffic` turns six rocprofv3
--pmc runs into profiles/k_ns_gemm_traffic_<workload>.md, which later runs
read as long as the kernel sources are unchanged.
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


PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ("kernels.hip", "plan.cpp", "plan.h", "device_types.h", "muonbp_api.cpp")


def kernel_source_digest():
    """sha256 over the sources that decide what the NS GEMM launches read and
    write (kernels, tile plans, descriptors)."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2510_16981_amd", "csrc", f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def traffic_file(workload):
    return os.path.join(PROFILES, f"k_ns_gemm_traffic_{workload}.md")


TRAFFIC_TAG = "traffic-json:"


def measured_traffic(workload, launches_of):
    """HBM bytes per k_ns_gemm launch from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by a copy of known size),
    weighted by this run's launches of each step kind.  None when no summary
    exists or the kernel sources changed since the counters were taken."""
    path = traffic_file(workload)
    if not os.path.exists(path):
        return None, "no counter summary for this workload"
    rec = None
    with open(path) as fh:
        for line in fh:
            if line.startswith(TRAFFIC_TAG):
                rec = json.loads(line[len(TRAFFIC_TAG):])
    if rec is None:
        return None, "counter summary has no traffic record"
    if rec.get("kernel_source_sha256") != kernel_source_digest():
        return None, "kernel sources changed since the counters were taken"
    tot = n = 0
    for kind, cnt in launches_of.items():
        if cnt and kind not in rec["bytes_per_launch"]:
            return None, f"no counters for {kind} steps"
        if cnt:
            tot += rec["bytes_per_launch"][kind] * cnt
            n += cnt
    return (tot / n if n else None), os.path.relpath(path, ROOT)


COPY_KERNEL_MATCH = "neg_kernel"


def copy_probe(mib):
    """Calibration for the HBM byte counters: a streaming kernel that reads
    `mib` MiB and writes `mib` MiB (torch's elementwise negation, fp32;
    a plain device copy may go to the DMA engines and show no dispatch),
    three times."""
    import torch
    n = mib << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "reps": 3, "kernel_match": COPY_KERNEL_MATCH}),
          flush=True)


def _pmc_rows(run_dir):
    """(kernel name, counter, value) rows of a rocprofv3 --pmc csv run."""
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                rows.append((r["Kernel_Name"], r["Counter_Name"], float(r["Counter_Value"])))
    if not rows:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    return rows


def _mean_kib(rows, counter, name_part):
    v = [x for k, c, x in rows if c == counter and name_part in k]
    if not v:
        raise SystemExit(f"no {counter} rows for kernels matching {name_part!r}")
    return sum(v) / len(v), len(v)


def ingest_traffic(workload, dirs, command):
    """Write the traffic summary from six rocprofv3 --pmc runs: FETCH_SIZE and
    WRITE_SIZE of the copy probe, of a run of block steps only (--period 0)
    and of full steps only (--period 1).  dirs: copy_fetch, copy_write,
    block_fetch, block_write, full_fetch, full_write."""
    d = dict(zip(("copy_fetch", "copy_write", "block_fetch", "block_write", "full_fetch",
                  "full_write"), dirs))
    copy_kib = None
    for line in open(os.path.join(d["copy_fetch"], "copy_probe.json")):
        if line.startswith("{"):
            copy_kib = json.loads(line)["copy_probe_bytes"] / 1024.0
    cf, _ = _mean_kib(_pmc_rows(d["copy_fetch"]), "FETCH_SIZE", COPY_KERNEL_MATCH)
    cw, _ = _mean_kib(_pmc_rows(d["copy_write"]), "WRITE_SIZE", COPY_KERNEL_MATCH)
    sf, sw = copy_kib / cf, copy_kib / cw
    per, detail = {}, {}
    for kind in ("block", "full"):
        f, nf = _mean_kib(_pmc_rows(d[f"{kind}_fetch"]), "FETCH_SIZE", "k_ns_gemm")
        w, nw = _mean_kib(_pmc_rows(d[f"{kind}_write"]), "WRITE_SIZE", "k_ns_gemm")
        per[kind] = (f * sf + w * sw) * 1024.0
        detail[kind] = {"fetch_kib_raw": f, "write_kib_raw": w, "dispatches": [nf, nw]}
    rec = {"kernel_source_sha256": kernel_source_digest(), "bytes_per_launch": per,
           "scale": {"fetch": sf, "write": sw}, "copy_kib": copy_kib,
           "copy_raw_kib": {"fetch": cf, "write": cw}, "detail": detail}
    path = traffic_file(workload)
    with open(path, "w") as fh:
        fh.write(f"# k_ns_gemm HBM traffic, {workload}\n\n")
        fh.write("rocprofv3 counter runs (each on its own, FETCH_SIZE then WRITE_SIZE, KiB per "
                 "dispatch), averaged over every k_ns_gemm dispatch of the run and scaled by what "
                 "the same counter reads for a plain copy of known size.\n\n")
        fh.write("Commands:\n\n```\n" + command.strip() + "\n```\n\n")
        fh.write("| | copy probe | block-step launches | full-step launches |\n|---|---|---|---|\n")
        fh.write(f"| FETCH_SIZE KiB/dispatch (raw) | {cf:.0f} | {detail['block']['fetch_kib_raw']:.0f} | "
                 f"{detail['full']['fetch_kib_raw']:.0f} |\n")
        fh.write(f"| WRITE_SIZE KiB/dispatch (raw) | {cw:.0f} | {detail['block']['write_kib_raw']:.0f} | "
                 f"{detail['full']['write_kib_raw']:.0f} |\n")
        fh.write(f"| scale (copy bytes / counter) | fetch {sf:.3f}, write {sw:.3f} | | |\n")
        fh.write(f"| HBM bytes per launch (scaled) | | {per['block']:.4g} | {per['full']:.4g} |\n\n")
        fh.write(TRAFFIC_TAG + " " + json.dumps(rec) + "\n")
    print(path)


def ingest_kernel_trace(workload, run_dir, command):
    """Write profiles/k_ns_gemm_<workload>.md from a rocprofv3 --kernel-trace
    --stats csv run of bench.py (its JSON line saved as bench.json in the
    same folder): the per-kernel statistics, and the k_ns_gemm average over
    the dispatches of the timed region next to bench.py's own figure."""
    import csv
    import glob

    def one(pattern):
        f = glob.glob(os.path.join(run_dir, "**", pattern), recursive=True)
        if not f:
            raise SystemExit(f"no {pattern} under {run_dir}")
        return f[0]

    stats = list(csv.DictReader(open(one("*kernel_stats.csv"))))
    trace = sorted(csv.DictReader(open(one("*kernel_trace.csv"))), key=lambda r: int(r["Start_Timestamp"]))
    bj = None
    for line in open(os.path.join(run_dir, "bench.json")):
        if line.startswith("{"):
            bj = json.loads(line)
    warm, steps = bj["warmup"], bj["steps"]
    # Step boundaries: every step starts with one k_momentum dispatch.
    starts = [i for i, r in enumerate(trace) if "k_momentum" in r["Kernel_Name"]]
    lo, hi = starts[warm], starts[warm + steps]
    ns = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in trace[lo:hi]
          if "k_ns_gemm" in r["Kernel_Name"]]
    avg_trace_us = sum(ns) / len(ns) / 1e3
    span_us = (int(trace[hi - 1]["End_Timestamp"]) - int(trace[lo]["Start_Timestamp"])) / 1e3
    path = os.path.join(PROFILES, f"k_ns_gemm_{workload}.md")
    with open(path, "w") as fh:
        fh.write(f"# Kernel trace, bench.py --workload {workload}\n\n")
        fh.write("Command:\n\n```\n" + command.strip() + "\n```\n\n")
        fh.write(f"bench.py line of the same run: value {bj['value']:.1f} steps/s, "
                 f"roofline achieved {bj['roofline']['achieved']:.1f} TFLOP/s "
                 f"(frac {bj['roofline']['frac']:.3f}), avg_launch_us "
                 f"{bj['roofline']['avg_launch_us']:.2f}.\n\n")
        fh.write(f"k_ns_gemm dispatches of the timed region in the trace ({len(ns)} dispatches, "
                 f"steps {warm}..{warm + steps - 1}): average duration {avg_trace_us:.2f} us; "
                 f"bench.py's HIP-event figure: {bj['roofline']['avg_launch_us']:.2f} us "
                 f"(ratio {bj['roofline']['avg_launch_us'] / avg_trace_us:.3f}).  Timed region "
                 f"in the trace: {span_us / 1e3:.2f} ms for {steps} steps.\n\n")
        fh.write("rocprofv3 --stats (whole run: warm-up, timed region, per-kind passes):\n\n")
        fh.write("| kernel | calls | average us | min us | max us | % of GPU time |\n|---|---|---|---|---|---|\n")
        for r in stats:
            name = r["Name"]
            if len(name) > 90:
                name = name[:87] + "..."
            fh.write(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.2f} |\n")
    print(path)


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
    ap.add_argument("--copy-probe", type=int, metavar="MIB", default=None,
                    help="only run a plain copy of MIB MiB (counter calibration) and exit")
    ap.add_argument("--ingest-traffic", nargs=6, metavar="DIR", default=None,
                    help="write the traffic summary of --workload from six rocprofv3 --pmc "
                         "csv runs: copy FETCH, copy WRITE, block FETCH, block WRITE, full "
                         "FETCH, full WRITE (no GPU use)")
    ap.add_argument("--ingest-kernel-trace", metavar="DIR", default=None,
                    help="write the kernel summary of --workload from a rocprofv3 --kernel-trace "
                         "--stats csv run of bench.py whose JSON line is DIR/bench.json (no GPU use)")
    ap.add_argument("--command", default="", help="with --ingest-*: the commands that made the runs")
    args = ap.parse_args()
    if args.ingest_traffic:
        ingest_traffic(args.workload, args.ingest_traffic, args.command)
        return
    if args.ingest_kernel_trace:
        ingest_kernel_trace(args.workload, args.ingest_kernel_trace, args.command)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(blocks of a sharded matrix are processed as a batch on one GPU).", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe:
        torch.cuda.set_device(0)
        copy_probe(args.copy_probe)
        return
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

    # Timed region: exactly `steps` steps of the schedule.  One pair of HIP
    # events per step on the library's stream (the stream the kernels run
    # on) brackets the step's NS GEMM launches, which run back to back; more
    # markers (one pair per launch) would themselves slow the step.
    log(f"timing {steps} steps")
    t_first = t
    opt.profile_enable(2)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        opt.step(params, grads, t)
        t += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    timed_prof = opt.profile_read(split=True)
    opt.profile_enable(0)
    n_full = sum(1 for s in range(t_first, t) if period > 0 and s % period == 0)
    n_of = {"block": steps - n_full, "full": n_full}

    def next_of_kind(t, full):
        while (period > 0 and t % period == 0) != full:
            t += 1
        return t

    # Per step kind, apart from the timed region: the wall time of a run of
    # that kind only (no events), then a detail pass with events around every
    # launch for the per-kernel split.
    per = {}
    for kind in ("block", "full"):
        full = kind == "full"
        nk = n_of[kind]
        if nk == 0:
            continue
        reps = max(1, min(nk, 20))
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
        log(f"per-kernel detail pass ({kind})")
        opt.profile_enable(1)
        for _ in range(reps):
            t = next_of_kind(t, full)
            opt.step(params, grads, t)
            t += 1
        detail = opt.profile_read()
        opt.profile_enable(0)
        span_ms, span_n = timed_prof[kind]["ns_span"]
        flops = plan_flops(mats, full, K_NS)
        info = mb.describe_plan(mats, full, opt.options)
        per[kind] = {
            "steps_in_timed_region": nk,
            "ms_per_step": ms_step,
            "ms_per_step_reps": reps,
            "ns_ms_per_step": span_ms / nk,
            "ns_tflops": flops * nk / (span_ms * 1e-3) / 1e12,
            "ns_frac_bf16_peak": flops * nk / (span_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
            "ns_dense_tflops_paper_count": info.ns_dense_flops * nk / (span_ms * 1e-3) / 1e12,
            "ns_gemm_launches_per_step": span_n / nk,
            "ns_flops_per_step": flops,
            "detail_kernel_ms_per_step": {k: v[0] / reps for k, v in detail.items()
                                          if k != "ns_span"},
            "detail_launches": {k: v[1] for k, v in detail.items() if k != "ns_span"},
            "gemm_tiles": [f"{info.gemm_tile_rows[i]}x{info.gemm_tile_cols[i]}:{info.gemm_tiles[i]}"
                           for i in range(3)],
        }

    kinds = list(per)
    ew = {}
    for kname, bpe in (("momentum", 6), ("update", 6)):
        n_launch = sum(per[k]["detail_launches"][kname] for k in kinds)
        if n_launch == 0:
            ew[kname] = {"fused": True,
                         "note": "applied inside the last NS product (no kernel of its own)"}
            continue
        ms = (sum(per[k]["detail_kernel_ms_per_step"][kname] * per[k]["ms_per_step_reps"]
                  for k in kinds) / n_launch)
        gbs = n_el * bpe / (ms * 1e-3) / 1e9
        ew[kname] = {"bytes_per_elem": bpe, "gbs": gbs, "frac_hbm_peak": gbs / HBM_PEAK_GBS,
                     "footprint_bytes": n_el * bpe, "timing": "detail pass",
                     "note": ("footprint within the 256 MB last-level cache" if n_el * bpe < 256e6
                              else "footprint well beyond the 256 MB last-level cache")}

    # Dominant kernel: the grouped NS GEMM (all three NS products) over the
    # launches of the timed region (block and full steps as scheduled).
    tot_flops = sum(plan_flops(mats, k == "full", K_NS) * n_of[k] for k in kinds)
    tot_ms = sum(timed_prof[k]["ns_span"][0] for k in kinds)
    launches = sum(timed_prof[k]["ns_span"][1] for k in kinds)
    achieved = tot_flops / (tot_ms * 1e-3) / 1e12
    launches_of = {k: timed_prof[k]["ns_span"][1] for k in kinds}
    traffic, traffic_note = measured_traffic(name, launches_of)
    roofline = {"kernel": "k_ns_gemm (bf16, all tile shapes)", "bound": "mfma",
                "achieved": achieved, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / BF16_PEAK_TFLOPS, "traffic": traffic,
                "traffic_note": traffic_note,
                "launches": launches, "avg_launch_us": tot_ms * 1e3 / launches,
                "avg_flops_per_launch": tot_flops / launches,
                "timing": ("HIP events on the library stream around each step's back-to-back "
                           "NS GEMM launches, over the timed region; avg_launch_us = span / "
                           "launches (includes the gaps between them)")}

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
