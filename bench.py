"""Benchmark of the MuonBP optimizer step on one MI355X.

Default workload: every 2D weight of a 32-layer model with the shapes of the
paper's 8B Llama-style model (Table 5: d = 4096, ffn = 14336, GQA kv width
1024), bf16 params, grads, momentum and NS operands, each matrix cut into
the 8-way Megatron shard grid (column shards 1 x 8 for q, k, v, gate, up;
row shards 8 x 1 for o, down), rank-128 synthetic gradients, K = 5
Newton-Schulz iterations, period P = 5 (steps t = 0, 5, 10, ... are full).
This is the largest configuration that fits one GPU (6.98 B parameters).
Other workloads (--workload) are smaller shapes of the same method: one
2048 x 6144 QKV weight in 8 column shards, a 16-layer d=2048 model and the
4096 x 14336 MLP matrices.

A step is one whole optimizer step: momentum, norms, NS (blockwise or full)
and the weight update, all in the HIP library.  Inputs are resident in HBM
before timing starts.  Printed: ONE JSON line.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload NAME]
                    [--period P] [--no-cpu-baseline]

Counter support (the roofline's `traffic` and MFMA utilisation):
`--copy-probe MIB` runs only a streaming kernel of known size, `--mfma-probe`
only a bf16 product of known flops, and `--ingest-counters` turns nine
rocprofv3 --pmc runs into profiles/counters_<workload>.md, which later runs
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

DEFAULT_WORKLOAD = "llama-32L-d4096-bf16"
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


def gram_space_unit(S, L, K, mode, apply_nn):
    """Whether the library runs an S x L unit's K iterations in Gram space
    (the planner's rule for bf16 NS; mode is the gram_iteration option)."""
    if mode == 1 or not apply_nn or K < 2:
        return False
    return mode == 2 or (S >= 128 and 4 * L >= 5 * S)


GRAM_SEGMENT = 3  # Gram-space iterations per segment (the library's kGramSegment)


def kind_flops(mats, full, K, mode=0, apply_nn=True):
    """Flops of each NS product kind per step as the library computes them
    (symmetric products counted once per distinct entry).  A unit that
    iterates as printed: K Grams, K A A, K applies; a Gram-space unit, per
    segment of n <= 3 iterations: one Gram, 4n - 3 symmetric S x S x S
    products (launched, and profiled, with the polynomial) and one apply."""
    out = {"gram": 0.0, "poly": 0.0, "apply": 0.0}
    segs = [min(GRAM_SEGMENT, K - k0) for k0 in range(0, K, GRAM_SEGMENT)]
    for r, c, gr, gc in mats:
        units = [(r, c)] if full else [(r // gr, c // gc)] * (gr * gc)
        for p, q in units:
            S, L = float(min(p, q)), float(max(p, q))
            g = gram_space_unit(S, L, K, mode, apply_nn)
            out["gram"] += (len(segs) if g else K) * S * (S + 1) * L
            out["poly"] += (sum(4 * n - 3 for n in segs) if g else K) * S * S * (S + 1)
            out["apply"] += (len(segs) if g else K) * 2 * S * S * L
    return out



# Dominant product shapes of the 8B-shaped model: MLP shards 1792 x 4096 on
# block steps (96 of the 224 matrices' 1792 units), whole 4096 x 14336 MLP
# matrices on full steps.
LIBRARY_SHAPES = {
    "block_gram_96x(1792x4096)(4096x1792)": (96, 1792, 4096, 1792),
    "block_poly_96x(1792x1792)^2": (96, 1792, 1792, 1792),
    "block_apply_96x(1792x1792)(1792x4096)": (96, 1792, 1792, 4096),
    "full_gram_(4096x14336)(14336x4096)": (1, 4096, 14336, 4096),
    "full_poly_(4096x4096)^2": (1, 4096, 4096, 4096),
    "full_apply_(4096x4096)(4096x14336)": (1, 4096, 4096, 14336),
}


def library_gemm_reference():
    """The vendor library's bf16 GEMM (torch.matmul / bmm, hipBLASLt) on the
    dominant NS product shapes, dense flops: what a tuned library product
    reaches on this GPU, for comparison with the NS kernels.  Measurement
    only; the optimizer never calls it."""
    import torch
    out = {}
    for name, (b, m, k, n) in LIBRARY_SHAPES.items():
        x = torch.randn(b, m, k, device="cuda", dtype=torch.bfloat16)
        y = torch.randn(b, k, n, device="cuda", dtype=torch.bfloat16)
        fn = (lambda: torch.bmm(x, y)) if b > 1 else (lambda: torch.matmul(x[0], y[0]))
        for _ in range(3):
            fn()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 10
        torch.cuda.synchronize()
        s.record()
        for _ in range(reps):
            fn()
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / reps
        tf = 2.0 * b * m * k * n / (ms * 1e-3) / 1e12
        out[name] = {"ms": ms, "tflops": tf, "frac_bf16_peak": tf / BF16_PEAK_TFLOPS}
        del x, y
    torch.cuda.empty_cache()
    return out


def _oracle_threads():
    from threadpoolctl import threadpool_info
    return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))


def cpu_baseline(workload, mats, period, rank, sample_steps):
    """The fp64 oracle on the host cores over `sample_steps` steps of the
    workload (from t = 0, so the sample holds full and block steps)."""
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
    nf = sum(1 for t in range(sample_steps) if period and t % period == 0)
    return {"value": sample_steps / dt, "unit": "steps/s", "cores": _oracle_threads(),
            "kind": "oracle",
            "sample": f"{sample_steps} consecutive steps (t=0..{sample_steps - 1}: {nf} full, "
                      f"{sample_steps - nf} blockwise) of {workload}, numpy float64, {dt:.1f} s",
            "host_cpus": len(os.sched_getaffinity(0)), "cpu": platform.processor() or platform.machine()}


def _time_oracle_step(O, W, spec, t, period, rank, lr_block, min_s=0.5):
    """Seconds of one MuonBPOracle.step (momentum, NS, update) on one
    matrix, repeated until min_s has passed (small units), averaged."""
    orc = O.MuonBPOracle([spec], O.OracleConfig(period=period, lr_block=lr_block,
                                                lr_full=LR_FULL, momentum=MU, weight_decay=WD))
    X = [W.quantize(W.init_param(spec.rows, spec.cols, 0, 0), "bf16").double().numpy()]
    G = [W.quantize(W.lowrank_grad(spec.rows, spec.cols, rank, 0, 0, t), "bf16").double().numpy()]
    reps, t0 = 0, time.perf_counter()
    while True:
        orc.step(X, G, t)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_s:
            return el / reps


def cpu_baseline_sampled(workload, mats, period, rank):
    """The fp64 oracle on a bounded sample of a workload too large to run
    whole on the host (a full step of the 8B-shaped model is about 666
    TFLOP), scaled to the whole step.  Sample: for every distinct block
    shape, one block run through MuonBPOracle.step as a matrix of its own on
    a block step; for every distinct NS problem of the full plan (S x L,
    S = the smaller side; a tall matrix shares the problem of its transpose),
    one whole matrix through MuonBPOracle.step on a full step.  Each timing
    covers the oracle's momentum, NS and update of that unit.  Block step =
    sum over blocks, full step = sum over matrices; steps/s is averaged over
    the period as P / (t_full + (P - 1) t_block).  Labelled extrapolated."""
    from oracle import muonbp_oracle as O
    from paper_2510_16981_amd import workload as W

    gr0, gc0 = mats[0][2], mats[0][3]
    lr_block = LR_FULL / (gr0 * gc0) ** 0.5
    t_all = time.perf_counter()
    block_t, full_t = {}, {}
    for r, c, gr, gc in mats:
        b = (r // gr, c // gc)
        if b not in block_t:
            block_t[b] = _time_oracle_step(O, W, O.MatrixSpec(b[0], b[1], 1, 1), 1, 0, rank, lr_block)
        f = (min(r, c), max(r, c))
        if f not in full_t:
            # one run of a large matrix is long enough on its own
            full_t[f] = _time_oracle_step(O, W, O.MatrixSpec(r, c, gr, gc), 0, 1, rank, lr_block,
                                          min_s=0.0)
    sample_s = time.perf_counter() - t_all
    t_block = sum(block_t[(r // gr, c // gc)] * gr * gc for r, c, gr, gc in mats)
    t_full = sum(full_t[(min(r, c), max(r, c))] for r, c, _, _ in mats)
    P = max(period, 1)
    value = P / (t_full + (P - 1) * t_block) if period else 1.0 / t_block
    blocks = ", ".join(f"{a}x{b}" for a, b in block_t)
    fulls = ", ".join(f"{a}x{b}" for a, b in full_t)
    return {"value": value, "unit": "steps/s", "cores": _oracle_threads(), "kind": "oracle",
            "extrapolated": True,
            "sample": f"{workload}: one block of each distinct block shape ({blocks}) on a block "
                      f"step and one whole matrix of each distinct full-step NS problem S x L "
                      f"({fulls}) on a full step, each through MuonBPOracle.step (numpy float64), "
                      f"{sample_s:.1f} s in all; scaled by the workload's block and matrix counts "
                      f"to t_block {t_block:.1f} s and t_full {t_full:.1f} s per step, then "
                      f"P / (t_full + (P - 1) t_block) at P = {period} (extrapolated)",
            "t_block_step_s": t_block, "t_full_step_s": t_full,
            "host_cpus": len(os.sched_getaffinity(0)), "cpu": platform.processor() or platform.machine()}


PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ("kernels.hip", "plan.cpp", "plan.h", "device_types.h", "muonbp_api.cpp", "step_core.cpp")


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
    return os.path.join(PROFILES, f"counters_{workload}.md")


TRAFFIC_TAG = "traffic-json:"


def counter_record(workload):
    """The committed rocprofv3 counter record of a workload (written by
    --ingest-counters), or None with the reason: no summary, or the kernel
    sources changed since the counters were taken."""
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
    return rec, os.path.relpath(path, ROOT)


def measured_counters(workload, launches_of):
    """From the counter record, weighted by this run's NS GEMM launches of
    each step kind: HBM bytes per launch (FETCH_SIZE + WRITE_SIZE scaled by a
    copy of known size), executed MFMA flops per launch and the mean MFMA
    utilisation.  (None, None, reason) when no valid record covers the run."""
    rec, note = counter_record(workload)
    if rec is None:
        return None, None, note
    n = sum(launches_of.values())
    for kind, cnt in launches_of.items():
        if cnt and (kind not in rec["bytes_per_launch"] or kind not in rec.get("mfma", {})):
            return None, None, f"no counters for {kind} steps"
    if n == 0:
        return None, None, "no NS GEMM launches"

    def avg(get):
        return sum(get(k) * c for k, c in launches_of.items() if c) / n

    traffic = avg(lambda k: rec["bytes_per_launch"][k])
    mfma = {"executed_flops_per_launch": avg(lambda k: rec["mfma"][k]["executed_flops_per_launch"]),
            "mfma_util_pct": avg(lambda k: rec["mfma"][k]["mfma_util_pct"]),
            "by_step_kind": rec["mfma"], "source": note}
    return traffic, mfma, note


COPY_KERNEL_MATCH = "neg_kernel"
MFMA_PROBE_N = 4096


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


def mfma_probe():
    """Check of the MFMA flop counter: three bf16 products of two 4096 x 4096
    matrices (torch's library GEMM), 2 * 4096^3 flops each."""
    import torch
    n = MFMA_PROBE_N
    a = torch.randn(n, n, device="cuda").to(torch.bfloat16)
    b = torch.randn(n, n, device="cuda").to(torch.bfloat16)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.mm(a, b)
    torch.cuda.synchronize()
    print(json.dumps({"mfma_probe_flops": 2 * n ** 3, "reps": 3}), flush=True)


def launch_products(mats, full, K, mode=0, apply_nn=True):
    """The library's grouped NS GEMM launches of one step, in order, named
    after their products: per iteration the Gram (units as printed; a
    Gram-space unit where its segment starts), the polynomial, the
    Gram-space Q / T products and the A update (Gram-space units), the apply
    (units as printed; a Gram-space unit at its segment's end).  Empty
    launches are skipped, as the library does."""
    flags = []
    for r, c, gr, gc in mats:
        units = [(r, c)] if full else [(r // gr, c // gc)] * (gr * gc)
        flags += [gram_space_unit(min(p, q), max(p, q), K, mode, apply_nn) for p, q in units]
    has_std, has_g = not all(flags), any(flags)
    out = []
    for it in range(K):
        j = it % GRAM_SEGMENT
        n = min(GRAM_SEGMENT, K - it + j)
        if has_std or (has_g and j == 0):
            out.append("gram")
        out.append("poly")
        if has_g and (j > 0 or j < n - 1):
            out.append("gram-space")
        if has_g and j < n - 1:
            out.append("gram-space")
        if has_std or (has_g and j == n - 1):
            out.append("apply")
    return out


def _pmc_dispatches(run_dir, products=None):
    """Dispatches of a rocprofv3 --pmc csv run: {dispatch id: {"name", "ns"
    (duration), counter: value, ...}}.  products: the NS GEMM launches of
    one step in order (launch_products); by default Gram, polynomial and
    apply per iteration."""
    import csv
    import glob
    out = {}
    for f in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                d = out.setdefault((f, int(r["Dispatch_Id"])), {
                    "name": r["Kernel_Name"],
                    "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
                d[r["Counter_Name"]] = float(r["Counter_Value"])
    if not out:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    rows = [out[k] for k in sorted(out)]
    # Name each NS GEMM dispatch after its product: a step launches pack,
    # then its NS GEMM launches in a fixed order, then the update.
    seq = products or ("gram", "poly", "apply")
    i = 0
    for r in rows:
        if "k_pack" in r["name"]:
            i = 0
        elif "k_ns_gemm" in r["name"]:
            r["product"] = seq[i % len(seq)]
            i += 1
    return rows


def _kernel_label(name):
    """Short label of one of the library's kernels (None for others)."""
    import re
    if "muonbp" not in name:
        return None
    m = re.search(r"(k_[a-z_]+)(<[^<>()]*>)?", name)
    return (m.group(1) + (m.group(2) or "").replace(" ", "")) if m else None


def _row_label(r):
    lab = _kernel_label(r["name"])
    return f"{lab} {r['product']}" if lab and "product" in r else lab


def _by_label(rows, counter):
    """Mean counter value and duration per kernel label."""
    acc = {}
    for r in rows:
        lab = _row_label(r)
        if lab is None or counter not in r:
            continue
        a = acc.setdefault(lab, [0.0, 0.0, 0])
        a[0] += r[counter]
        a[1] += r["ns"]
        a[2] += 1
    return {k: {"value": v[0] / v[2], "us": v[1] / v[2] / 1e3, "n": v[2]} for k, v in acc.items()}


def _json_line(path, key):
    for line in open(path):
        if line.startswith("{"):
            rec = json.loads(line)
            if key in rec:
                return rec
    raise SystemExit(f"no JSON line with {key!r} in {path}")


INGEST_DIRS = ("copy_fetch", "copy_write", "mfma_probe", "block_fetch", "block_write",
               "block_mfma", "full_fetch", "full_write", "full_mfma")
MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "MfmaUtil", "GRBM_GUI_ACTIVE")
# Bytes per element the elementwise kernels must move (bf16 storage):
# momentum reads M and G and writes M; pack reads M and writes Z (the apply
# reads Z row-major, so no Z^T; only the units not read in place, the plan's
# pack_elements); update reads X and U and writes X.
ELEMENTWISE_BYTES = {"k_momentum": 6, "k_pack": 4, "k_update": 6}


# Commands that make the runs each summary is ingested from (the default of
# --command; all run from committed files only).
COUNTER_COMMANDS = """\
cd /tmp && export TMPDIR=/tmp   # R = repository root, W = workload
rocprofv3 --pmc FETCH_SIZE -f csv -d $R/gpurun_out/prof/copy_fetch -o run -- python3 $R/bench.py --copy-probe 1024 > $R/gpurun_out/prof/copy_fetch/copy_probe.json
rocprofv3 --pmc WRITE_SIZE -f csv -d $R/gpurun_out/prof/copy_write -o run -- python3 $R/bench.py --copy-probe 1024
rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 MfmaUtil GRBM_GUI_ACTIVE -f csv -d $R/gpurun_out/prof/mfma_probe -o run -- python3 $R/bench.py --mfma-probe > $R/gpurun_out/prof/mfma_probe/mfma_probe.json
# kind=block with P=0, kind=full with P=1; each run's JSON line saved as b.json in its folder
rocprofv3 --pmc FETCH_SIZE -f csv -d $R/gpurun_out/prof/$W/${kind}_fetch -o run -- python3 $R/bench.py --workload $W --period $P --steps 10 --warmup 2 --no-cpu-baseline --no-scalar --no-library-reference
rocprofv3 --pmc WRITE_SIZE -f csv -d $R/gpurun_out/prof/$W/${kind}_write -o run -- python3 $R/bench.py --workload $W --period $P --steps 10 --warmup 2 --no-cpu-baseline --no-scalar --no-library-reference
rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 MfmaUtil GRBM_GUI_ACTIVE -f csv -d $R/gpurun_out/prof/$W/${kind}_mfma -o run -- python3 $R/bench.py --workload $W --period $P --steps 10 --warmup 2 --no-cpu-baseline --no-scalar --no-library-reference
python3 bench.py --workload $W --ingest-counters gpurun_out/prof/{copy_fetch,copy_write,mfma_probe} gpurun_out/prof/$W/{block_fetch,block_write,block_mfma,full_fetch,full_write,full_mfma}
"""
KERNEL_TRACE_COMMANDS = """\
cd /tmp && export TMPDIR=/tmp   # R = repository root
rocprofv3 --kernel-trace --stats -f csv -d $R/gpurun_out/prof/kt -o run -- python3 $R/bench.py --no-cpu-baseline --no-library-reference > $R/gpurun_out/prof/kt/bench.json
python3 bench.py --ingest-kernel-trace gpurun_out/prof/kt
"""


def ingest_counters(workload, dirs, command):
    """Write profiles/counters_<workload>.md from nine rocprofv3 --pmc runs
    (one folder each, in INGEST_DIRS order): FETCH_SIZE and WRITE_SIZE of
    the copy probe; the MFMA counters of the MFMA probe; then FETCH_SIZE,
    WRITE_SIZE and the MFMA counters (MFMA_COUNTERS) of a run of block steps
    only (--period 0) and of full steps only (--period 1), each with its
    bench.py JSON line in b.json.

    Per kernel and step kind: HBM bytes per dispatch (FETCH_SIZE and
    WRITE_SIZE scaled by the copy probe) and the resulting GB/s; executed
    bf16 MFMA flops per dispatch (the counter's unit is 512 flops, checked
    against the probe's known flops) and TFLOP/s; MFMA utilisation (busy
    MFMA cycles over active cycles times SIMDs, rocprofv3's MfmaUtil).
    Durations are those of the counter runs' own dispatches."""
    from paper_2510_16981_amd import muonbp as mb
    from paper_2510_16981_amd import workload as W
    d = dict(zip(INGEST_DIRS, dirs))
    copy_kib = _json_line(os.path.join(d["copy_fetch"], "copy_probe.json"),
                          "copy_probe_bytes")["copy_probe_bytes"] / 1024.0

    def probe_mean(run, counter, pick):
        v = [r[counter] for r in _pmc_dispatches(d[run]) if counter in r and pick(r)]
        if not v:
            raise SystemExit(f"no {counter} dispatches in {d[run]}")
        return v

    cf = probe_mean("copy_fetch", "FETCH_SIZE", lambda r: COPY_KERNEL_MATCH in r["name"])
    cw = probe_mean("copy_write", "WRITE_SIZE", lambda r: COPY_KERNEL_MATCH in r["name"])
    cf, cw = sum(cf) / len(cf), sum(cw) / len(cw)
    sf, sw = copy_kib / cf, copy_kib / cw
    probe_flops = _json_line(os.path.join(d["mfma_probe"], "mfma_probe.json"),
                             "mfma_probe_flops")["mfma_probe_flops"]
    # The probe's product is the dispatch with the most MFMA work.
    pm = max(probe_mean("mfma_probe", "SQ_INSTS_VALU_MFMA_MOPS_BF16", lambda r: True))
    mops_unit = 512.0
    probe_ratio = pm * mops_unit / probe_flops

    tables, per_launch, mfma_rec = {}, {}, {}
    for kind in ("block", "full"):
        bj = _json_line(os.path.join(d[f"{kind}_mfma"], "b.json"), "metric")
        n_el = bj["config"]["params"]
        kstats = bj[kind]
        alg_flops_launch = kstats["ns_flops_per_step"] / kstats["ns_gemm_launches_per_step"]
        mats = W.workload_matrices(workload)
        info = mb.describe_plan(mats, kind == "full", mb.options_default(ns_steps=K_NS))
        prods = launch_products(mats, kind == "full", K_NS, 0, bool(info.apply_nn))
        if len(prods) != info.gemm_launches:
            raise SystemExit("launch order model out of step with the planner")
        fetch = _by_label(_pmc_dispatches(d[f"{kind}_fetch"], prods), "FETCH_SIZE")
        write = _by_label(_pmc_dispatches(d[f"{kind}_write"], prods), "WRITE_SIZE")
        mrows = _pmc_dispatches(d[f"{kind}_mfma"], prods)
        mops = _by_label(mrows, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
        util = _by_label(mrows, "MfmaUtil")
        gui = _by_label(mrows, "GRBM_GUI_ACTIVE")
        rows = []
        for lab in sorted(set(fetch) | set(mops)):
            f, w = fetch.get(lab), write.get(lab)
            byt = (f["value"] * sf + w["value"] * sw) * 1024.0 if f and w else None
            us = f["us"] if f else mops[lab]["us"]
            flops = mops[lab]["value"] * mops_unit if lab in mops else None
            base = lab.split("<")[0]
            n_moved = info.pack_elements if base == "k_pack" else n_el
            alg = (n_moved * ELEMENTWISE_BYTES[base]) if base in ELEMENTWISE_BYTES else None
            rows.append({
                "kernel": lab, "dispatches": f["n"] if f else mops[lab]["n"], "us": us,
                "hbm_bytes": byt, "hbm_gbs": byt / (us * 1e3) if byt else None,
                "alg_bytes": alg, "alg_gbs": alg / (us * 1e3) if alg else None,
                "mfma_flops": flops, "mfma_us": mops[lab]["us"] if lab in mops else None,
                "mfma_tflops": (flops / (mops[lab]["us"] * 1e-6) / 1e12) if flops else None,
                "mfma_util": util[lab]["value"] if lab in util else None,
                "gui_active": gui[lab]["value"] if lab in gui else None})
        tables[kind] = rows
        g = [r for r in rows if r["kernel"].startswith("k_ns_gemm")]
        nf = sum(r["dispatches"] for r in g)
        per_launch[kind] = sum(r["hbm_bytes"] * r["dispatches"] for r in g) / nf
        nm = sum(r["dispatches"] for r in g if r["mfma_flops"] is not None)
        ex = sum(r["mfma_flops"] * r["dispatches"] for r in g if r["mfma_flops"] is not None) / nm
        ut = sum(r["mfma_util"] * r["dispatches"] for r in g if r["mfma_util"] is not None) / nm
        mfma_rec[kind] = {"executed_flops_per_launch": ex, "algorithmic_flops_per_launch":
                          alg_flops_launch, "mfma_util_pct": ut}

    rec = {"kernel_source_sha256": kernel_source_digest(), "bytes_per_launch": per_launch,
           "scale": {"fetch": sf, "write": sw}, "copy_kib": copy_kib,
           "copy_raw_kib": {"fetch": cf, "write": cw}, "mfma": mfma_rec,
           "mfma_probe_ratio": probe_ratio}
    path = traffic_file(workload)

    def fmt(x, spec):
        return "" if x is None else format(x, spec)

    with open(path, "w") as fh:
        fh.write(f"# rocprofv3 counters per kernel, {workload}\n\n")
        fh.write("Counter runs, one counter set per run: FETCH_SIZE, WRITE_SIZE, and the MFMA "
                 "set (SQ_INSTS_VALU_MFMA_MOPS_BF16, MfmaUtil, GRBM_GUI_ACTIVE).  Block steps "
                 "only (--period 0) and full steps only (--period 1); every dispatch of the run "
                 "is averaged per kernel.  Durations are those of the counter runs' dispatches "
                 "(serialised by the counter collection).\n\n")
        fh.write("Commands:\n\n```\n" + command.strip() + "\n```\n\n")
        fh.write("Calibration:\n\n")
        fh.write(f"* HBM bytes: a streaming kernel reading and writing {copy_kib / 1024:.0f} MiB "
                 f"reads FETCH_SIZE {cf:.0f} KiB, WRITE_SIZE {cw:.0f} KiB per dispatch: scale "
                 f"fetch {sf:.3f}, write {sw:.3f}.\n")
        fh.write(f"* MFMA flops: SQ_INSTS_VALU_MFMA_MOPS_BF16 counts units of 512 flops; the "
                 f"{MFMA_PROBE_N}^3 bf16 product of the probe reads {pm * mops_unit:.4g} flops "
                 f"against {probe_flops:.4g} (ratio {probe_ratio:.3f}).\n")
        fh.write("* MfmaUtil = busy MFMA cycles summed over SIMDs / (active GPU cycles x SIMDs), "
                 "in percent.  Its active cycles (GRBM_GUI_ACTIVE) span the counter collection "
                 "window, a few microseconds longer than the dispatch itself (a 3 us kernel "
                 "reads as about 10 us of active cycles at the 2.4 GHz clock), so it understates "
                 "the utilisation of short dispatches; the TFLOP/s column divides the counted "
                 "flops by the dispatch's own duration instead.\n\n")
        for kind in ("block", "full"):
            m = mfma_rec[kind]
            fh.write(f"## {kind} steps\n\n")
            fh.write(f"NS GEMM launches: {per_launch[kind]:.4g} HBM bytes, "
                     f"{m['executed_flops_per_launch']:.4g} executed MFMA flops "
                     f"({m['algorithmic_flops_per_launch']:.4g} algorithmic, ratio "
                     f"{m['executed_flops_per_launch'] / m['algorithmic_flops_per_launch']:.3f}), "
                     f"MfmaUtil {m['mfma_util_pct']:.1f}% per launch on average.\n\n")
            fh.write("| kernel | dispatches | us | HBM MB | HBM GB/s | % of 8 TB/s | algorithmic "
                     "GB/s | MFMA GFLOP | MFMA TFLOP/s | % of 2.5 PF | MfmaUtil % |\n"
                     "|---|---|---|---|---|---|---|---|---|---|---|\n")
            for r in tables[kind]:
                fh.write(f"| `{r['kernel']}` | {r['dispatches']} | {r['us']:.2f} | "
                         f"{fmt(r['hbm_bytes'] and r['hbm_bytes'] / 1e6, '.2f')} | "
                         f"{fmt(r['hbm_gbs'], '.0f')} | "
                         f"{fmt(r['hbm_gbs'] and 100 * r['hbm_gbs'] / HBM_PEAK_GBS, '.1f')} | "
                         f"{fmt(r['alg_gbs'], '.0f')} | "
                         f"{fmt(r['mfma_flops'] and r['mfma_flops'] / 1e9, '.2f')} | "
                         f"{fmt(r['mfma_tflops'], '.0f')} | "
                         f"{fmt(r['mfma_tflops'] and 100 * r['mfma_tflops'] / BF16_PEAK_TFLOPS, '.1f')} | "
                         f"{fmt(r['mfma_util'], '.1f')} |\n")
            fh.write("\n")
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


# Tensors the paper trains with AdamW instead of MuonBP (1D parameters and
# the input embedding, Appendix B), at the 8B-shaped model's sizes: the
# embedding (vocabulary 128256 x d 4096; the paper does not state its
# vocabulary) and 2 RMSNorm vectors per layer plus the final one.
SCALAR_SIZES = [128256 * 4096] + [4096] * (2 * 32 + 1)
SCALAR_WORKLOAD = "adamw-embedding-128256x4096-and-65x4096-norms-bf16"


def scalar_optimizer_bench(steps=20, warmup=3):
    """GB/s of the AdamW step (global-norm clipping on): algorithmic bytes per
    element = gradient read for the norm (2) + params, grads, m, v read (12)
    + params, m, v written (10), bf16 params with fp32 moments."""
    import torch
    from paper_2510_16981_amd import muonbp as mb
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    params = [(0.02 * torch.randn(n, generator=g, device="cuda")).to(torch.bfloat16)
              for n in SCALAR_SIZES]
    grads = [(1e-3 * torch.randn(n, generator=g, device="cuda")).to(torch.bfloat16)
             for n in SCALAR_SIZES]
    opt = mb.AdamW(SCALAR_SIZES)
    for t in range(warmup):
        opt.step(params, grads, t, 1e-3)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(warmup, warmup + steps):
        opt.step(params, grads, t, 1e-3)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    n = sum(SCALAR_SIZES)
    bpe = 24
    gbs = n * bpe / (ms * 1e-3) / 1e9
    opt.close()
    del params, grads
    torch.cuda.empty_cache()
    return {"workload": SCALAR_WORKLOAD, "elements": n, "ms_per_step": ms, "bytes_per_elem": bpe,
            "gbs": gbs, "frac_hbm_peak": gbs / HBM_PEAK_GBS, "steps": steps,
            "timing": "host timer around synchronized back-to-back steps (3 launches each)"}


def ingest_workloads(paths, out_path):
    """Write the larger-workload summary (profiles/steps_larger_workloads.md)
    from bench.py JSON lines, one file per workload run."""
    from paper_2510_16981_amd import workload as W
    kinds = ("momentum", "scale", "pack", "gram", "poly", "apply", "update")
    lines = ["# Step and kernel times: larger workloads (one MI355X)", "",
             "Command for each row (from the repository root), then this summary:", "", "```",
             "python3 bench.py --workload <name> > <name>.json",
             "python3 bench.py --ingest-workloads <name>.json ...", "```", "",
             "`ns TFLOP/s` comes from HIP events around each step's back-to-back NS GEMM launches "
             "in the timed region;", "per-kernel times from the detail pass (events around every "
             "launch); step times from host timers around", "synchronized runs of one step kind.  "
             "Inputs are GPU-drawn timing-only gradients, one per matrix (bench.py make_inputs).",
             ""]
    for path in paths:
        d = None
        for line in open(path):
            if line.startswith("{"):
                d = json.loads(line)
        cfg = d["config"]
        name = cfg["workload"]
        mats = W.workload_matrices(name)
        lines += [f"## {name} ({cfg['matrices']} matrices, {cfg['params'] / 1e9:.3f} B params, "
                  f"grids {', '.join(cfg['grids'])})", "",
                  f"Timed schedule P = {cfg['period']}: {d['value']:.3f} steps/s, "
                  f"{d['ms_per_step']:.2f} ms/step; NS GEMM {d['roofline']['achieved']:.0f} TFLOP/s "
                  f"= {100 * d['roofline']['frac']:.1f}% of {BF16_PEAK_TFLOPS:.0f}.", "",
                  "| Step | ms/step | NS TFLOP/s | % bf16 peak | tiles (Gram, poly, apply) | "
                  + " | ".join(f"{k} ms" for k in kinds) + " |",
                  "|---|---:|---:|---:|---|" + "---:|" * len(kinds)]
        for kind in ("block", "full"):
            b = d.get(kind)
            if not b:
                continue
            det = b["detail_kernel_ms_per_step"]
            lines.append(f"| {kind} | {b['ms_per_step']:.2f} | {b['ns_tflops']:.1f} | "
                         f"{100 * b['ns_frac_bf16_peak']:.1f} | {' '.join(b['gemm_tiles'])} | "
                         + " | ".join(f"{det.get(k, 0.0):.3f}" for k in kinds) + " |")
        ew = d["elementwise"]
        parts = [f"{k} {v['gbs']:.0f} GB/s ({100 * v['frac_hbm_peak']:.0f}% of 8 TB/s)"
                 for k, v in ew.items() if "gbs" in v]
        lines += ["", f"Elementwise (6 B/element each): {', '.join(parts)}; footprint "
                  f"{ew['momentum'].get('note', '')}.".replace("footprint footprint", "footprint"), ""]
        sw = d.get("period_sweep_ms_per_step")
        if sw:
            lines += ["Period sweep, ms/step ((t_full + (P-1) t_block) / P): "
                      + ", ".join(f"P={k}: {v:.1f}" for k, v in sw.items()), ""]
        sc = d.get("scalar_optimizer")
        if sc:
            lines += [f"AdamW pass ({sc['workload']}): {sc['ms_per_step']:.3f} ms/step, "
                      f"{sc['gbs']:.0f} GB/s ({100 * sc['frac_hbm_peak']:.0f}% of 8 TB/s).", ""]
        del mats
    with open(out_path, "w") as fh:
        fh.write("\n".join(lines))
    print(out_path)


def make_inputs(mats, rank):
    """Params and grads, one tensor each per matrix.  Small workloads: the
    exact seeded host inputs.  Large ones: GPU-drawn timing-only inputs (the
    step's cost does not depend on their values).  Every matrix has its own
    gradient in its own memory, so no step reads a gradient another matrix
    has just pulled into the caches."""
    import torch
    from paper_2510_16981_amd import workload as W
    n_el = sum(r * c for r, c, _, _ in mats)
    if n_el <= HOST_INPUT_LIMIT:
        params = [W.quantize(W.init_param(r, c, 0, k), "bf16").cuda() for k, (r, c, _, _) in enumerate(mats)]
        grads = [W.quantize(W.lowrank_grad(r, c, rank, 0, k, 0), "bf16").cuda()
                 for k, (r, c, _, _) in enumerate(mats)]
        return params, grads, "synthetic (seeded host draws)"
    params = [W.device_param(r, c, 0, k) for k, (r, c, _, _) in enumerate(mats)]
    grads = [W.device_grad(r, c, rank, 0, k) for k, (r, c, _, _) in enumerate(mats)]
    torch.cuda.synchronize()
    return params, grads, "synthetic (GPU-drawn, one gradient per matrix)"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--period", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-scalar", action="store_true",
                    help="skip the AdamW measurement (scalar_optimizer)")
    ap.add_argument("--apply-mode", type=int, default=0,
                    help="library option apply_mode (0: apply reads Z row-major, 1: keeps Z^T)")
    ap.add_argument("--k-split", type=int, default=0,
                    help="library option k_split (0: planner's choice)")
    ap.add_argument("--no-library-reference", action="store_true",
                    help="skip timing the vendor library's GEMM on the dominant shapes")
    ap.add_argument("--tile-policy", type=int, default=0,
                    help="library option tile_policy (0: planner's choice)")
    ap.add_argument("--gram-iteration", type=int, default=0,
                    help="library option gram_iteration (0: Gram-space iteration where it saves "
                         "time, 1: every iteration as printed, 2: Gram-space wherever allowed)")
    ap.add_argument("--copy-probe", type=int, metavar="MIB", default=None,
                    help="only run a plain copy of MIB MiB (counter calibration) and exit")
    ap.add_argument("--mfma-probe", action="store_true",
                    help="only run three 4096^3 bf16 products (MFMA counter check) and exit")
    ap.add_argument("--ingest-counters", nargs=9, metavar="DIR", default=None,
                    help="write the per-kernel counter summary of --workload from nine "
                         "rocprofv3 --pmc csv runs: copy FETCH, copy WRITE, MFMA probe, then "
                         "FETCH, WRITE and MFMA counters of block steps and of full steps "
                         "(no GPU use)")
    ap.add_argument("--ingest-kernel-trace", metavar="DIR", default=None,
                    help="write the kernel summary of --workload from a rocprofv3 --kernel-trace "
                         "--stats csv run of bench.py whose JSON line is DIR/bench.json (no GPU use)")
    ap.add_argument("--ingest-workloads", nargs="+", metavar="JSON", default=None,
                    help="write profiles/steps_larger_workloads.md from bench.py JSON outputs "
                         "(no GPU use)")
    ap.add_argument("--command", default=None,
                    help="with --ingest-*: the commands that made the runs (default: the standard ones)")
    args = ap.parse_args()
    if args.ingest_counters:
        ingest_counters(args.workload, args.ingest_counters,
                        COUNTER_COMMANDS if args.command is None else args.command)
        return
    if args.ingest_workloads:
        ingest_workloads(args.ingest_workloads, os.path.join(PROFILES, "steps_larger_workloads.md"))
        return
    if args.ingest_kernel_trace:
        ingest_kernel_trace(args.workload, args.ingest_kernel_trace,
                            KERNEL_TRACE_COMMANDS if args.command is None else args.command)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(blocks of a sharded matrix are processed as a batch on one GPU).", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe or args.mfma_probe:
        torch.cuda.set_device(0)
        if args.copy_probe:
            copy_probe(args.copy_probe)
        else:
            mfma_probe()
        return
    from paper_2510_16981_amd import muonbp as mb
    from paper_2510_16981_amd import workload as W

    name = args.workload
    wl = W.WORKLOADS[name]
    mats = W.workload_matrices(name)
    n_el = sum(r * c for r, c, _, _ in mats)
    large = n_el > HOST_INPUT_LIMIT
    steps = args.steps if args.steps is not None else (20 if large else 100)
    warmup = args.warmup if args.warmup is not None else 5
    period = args.period if args.period is not None else wl["period"]
    rank = wl["rank"]
    gr, gc = mats[0][2], mats[0][3]
    lr_block = LR_FULL / (gr * gc) ** 0.5
    torch.cuda.set_device(0)

    log(f"workload {name}: {len(mats)} matrices, {n_el / 1e6:.1f} M params; generating inputs")
    params, grads, data = make_inputs(mats, rank)
    opt = mb.MuonBP(mats, period, lr_block, LR_FULL, MU, WD,
                    options=mb.options_default(ns_steps=K_NS, apply_mode=args.apply_mode,
                                               k_split=args.k_split, tile_policy=args.tile_policy,
                                               gram_iteration=args.gram_iteration))
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
        info = mb.describe_plan(mats, full, opt.options)
        flops = info.ns_flops
        kf = kind_flops(mats, full, K_NS, args.gram_iteration, bool(info.apply_nn))
        assert abs(sum(kf.values()) - flops) <= 1e-9 * flops, "flop model out of step with the planner"
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
            "detail_gemm_tflops": {k: f * reps / (detail[k][0] * 1e-3) / 1e12
                                   for k, f in kf.items() if detail[k][0] > 0},
            "gram_space_units": int(info.gram_units),
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
    tot_flops = sum(per[k]["ns_flops_per_step"] * n_of[k] for k in kinds)
    tot_ms = sum(timed_prof[k]["ns_span"][0] for k in kinds)
    launches = sum(timed_prof[k]["ns_span"][1] for k in kinds)
    achieved = tot_flops / (tot_ms * 1e-3) / 1e12
    launches_of = {k: timed_prof[k]["ns_span"][1] for k in kinds}
    traffic, mfma_counters, traffic_note = measured_counters(name, launches_of)
    # The same NS work counted as Alg. 2 as printed (K Grams, A A and
    # applies per unit, symmetric products once): the rate the printed
    # schedule would need to match this time.
    printed = sum(sum(kind_flops(mats, k == "full", K_NS, 1).values()) * n_of[k] for k in kinds)
    roofline = {"kernel": "k_ns_gemm (bf16, all tile shapes)", "bound": "mfma",
                "achieved": achieved, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / BF16_PEAK_TFLOPS,
                "flops": "the products as computed (Gram-space segments on wide units)",
                "printed_equivalent_tflops": printed / (tot_ms * 1e-3) / 1e12,
                "traffic": traffic,
                "traffic_note": traffic_note, "mfma_counters": mfma_counters,
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
    del params, grads
    torch.cuda.empty_cache()
    if name == DEFAULT_WORKLOAD and not args.no_library_reference:
        log("library GEMM reference")
        out["library_gemm_reference"] = library_gemm_reference()
    if not args.no_scalar:
        log("scalar optimizer (AdamW) pass")
        out["scalar_optimizer"] = scalar_optimizer_bench()
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        if large:
            out["cpu_baseline"] = cpu_baseline_sampled(name, mats, period, rank)
        else:
            out["cpu_baseline"] = cpu_baseline(name, mats, period, rank, 3 * max(period, 1))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
