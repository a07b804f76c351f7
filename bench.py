#!/usr/bin/env python3
"""Benchmark: dense bf16 GEMM C = A*B (fp32 accumulate, fp32 out), 8192^3, one GPU.

(With --workload gemv<N>_fp32 it measures the fp32 GEMV y = A*x instead and
prints that kernel's line, bound by HBM bandwidth.)

One step is one call of xgemm_run on the 8192 x 8192 x 8192 bf16 workload
(entries uniform on [-1, 1], seed 2), inputs already resident in HBM.  Prints
one JSON line.  ``value`` is the whole-job throughput over the K timed steps,
bracketed by device synchronisation; ``roofline.achieved`` uses the average
duration of the GEMM kernel from two HIP events recorded on the stream the
kernel is launched on around the K steps, during which the stream runs the
kernels back to back (for a call the selector cuts into a body and a band of
C, both launches: ``config.band`` then describes the band).  The paper's own
protocol (5 warm-up + 100 timed iterations, mean of the inter-quartile range;
Section 6) is reported beside it, from a second sample of max(K, 100) calls
with events around each call.  Before the warm-up steps, untimed calls
run for --settle seconds (at least 64 calls): from idle, the GPU's power
controller takes tens of calls to settle, and the first ones run 10-35%
slower than the sustained rate that the timed steps are meant to measure
(``settle`` in the line says how many calls that took).  ``counters`` and
``roofline.traffic`` are not measured by this run: they come from the
committed rocprofv3 summary of the same kernel sources, taken on another box.

Usage: python bench.py [--gpus 1] [--steps 100] [--warmup 5] [--settle 0.5] [--workload NAME] [--no-persistent]
       [--no-cpu-baseline] [--no-comparator] [--copy-calibration BYTES]
       python bench.py --sweep M,N,K [M,N,K ...] [--dtype bf16] [--rounds 5]
       python bench.py --summarize-counters DIR [--workload NAME]   (CPU only)

--sweep times every (tile, split-k) configuration of each shape and reports
the selector's plan against the fastest one (one JSON line per shape; the
configuration selector's validation).

Counters: run this script under ``rocprofv3 --pmc`` (one pass per counter
group, with --copy-calibration 1073741824 on the FETCH_SIZE and WRITE_SIZE
passes), then ``--summarize-counters`` on the output directory writes
profiles/counters_<workload>.json.  The HBM byte counters are scaled by what
they read for a plain 1 GiB device copy (known traffic: 1 GiB read, 1 GiB
written).  The bench line reports the summary while the kernel sources still
hash to the value recorded in it.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2516.6, "fp16": 2516.6}  # MI355X dense MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_HBM_GBS = 8000.0                            # MI355X HBM3E
METRIC = "GEMM TFLOP/s and % of MI355X dense MFMA peak (bf16, 8192³) on 1 GPU"
GEMV_METRIC = "GEMV TFLOP/s and %% of the MI355X HBM-bound GEMV peak (fp32, %d², 2 FLOP per 4-byte element)"
COUNTERS_FILE = os.path.join(ROOT, "profiles", "counters_%s.json")
# device code whose change invalidates committed counters of each kernel
# family (the kernel the counters describe is also named in them)
KERNEL_SOURCES = {"gemm": ("gemm_kernel.hpp", "sk_kernel.hpp"), "gemv": ("gemv_kernel.hpp",)}


def family(workload: str) -> str:
    return "gemv" if workload.startswith("gemv") else "gemm"


def kernel_source_hash(fam: str = "gemm") -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[fam]:
        with open(os.path.join(ROOT, "paper_2609_16389_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_counters(workload: str):
    """Committed rocprofv3 --pmc summary of this workload's kernel, or None
    if there is none or the kernel sources changed since it was taken."""
    path = COUNTERS_FILE % workload
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_source_sha256") != kernel_source_hash(family(workload)):
        return None
    return d


def stored_traffic(workload: str):
    """HBM bytes per launch from the committed counters, or None."""
    d = stored_counters(workload)
    return None if d is None else d.get("hbm_bytes_per_launch")


def _kernel_metrics(med: dict, dur_ns: float, fetch_scale, write_scale) -> dict:
    """Derived figures of one kernel from its median counter values."""
    out = {"median_duration_ns": dur_ns, "counters_median": med}
    if fetch_scale and "FETCH_SIZE" in med:
        out["hbm_read_bytes_per_launch"] = 1024.0 * med["FETCH_SIZE"] * fetch_scale
    if write_scale and "WRITE_SIZE" in med:
        out["hbm_write_bytes_per_launch"] = 1024.0 * med["WRITE_SIZE"] * write_scale
    if "hbm_read_bytes_per_launch" in out and "hbm_write_bytes_per_launch" in out:
        out["hbm_bytes_per_launch"] = out["hbm_read_bytes_per_launch"] + out["hbm_write_bytes_per_launch"]
    if "SQ_VALU_MFMA_BUSY_CYCLES" in med and "GRBM_GUI_ACTIVE" in med:
        # GRBM_GUI_ACTIVE is summed over the 8 XCDs; 1024 SIMDs in all
        per_xcd = med["GRBM_GUI_ACTIVE"] / 8.0
        out["mfma_busy_pct"] = 100.0 * med["SQ_VALU_MFMA_BUSY_CYCLES"] / (per_xcd * 1024.0)
        out["clock_ghz"] = per_xcd / dur_ns
    if "SQ_LDS_BANK_CONFLICT" in med and "SQ_LDS_IDX_ACTIVE" in med:
        out["lds_bank_conflict_pct"] = 100.0 * med["SQ_LDS_BANK_CONFLICT"] / max(1.0, med["SQ_LDS_IDX_ACTIVE"])
    if "TCC_HIT_sum" in med and "TCC_MISS_sum" in med:
        out["l2_hit_pct"] = 100.0 * med["TCC_HIT_sum"] / max(1.0, med["TCC_HIT_sum"] + med["TCC_MISS_sum"])
    return out


def summarize_counters(directory: str, workload: str) -> str:
    """rocprofv3 --pmc CSV output -> profiles/counters_<workload>.json.

    Every kernel of the call is summarised (the GEMM launches, a split-k
    reduction, operand copies); ``kernel`` and the top-level figures are those
    of the GEMM kernel with the largest total time, and ``per_call`` sums the
    HBM bytes and durations of all the call's kernels.  The copy kernel of
    --copy-calibration only provides the byte counters' scale."""
    import csv
    import datetime
    import statistics
    vals, durs = {}, {}
    for path in sorted(glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)):
        with open(path) as f:
            for r in csv.DictReader(f):
                k = r["Kernel_Name"]
                vals.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
                durs.setdefault(k, []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    fam = family(workload)
    copy = [k for k in vals if "copyBuffer" in k or "copy_kernel" in k]
    ours = [k for k in vals if k not in copy and "xgem" in k]
    main_kernels = [k for k in ours if ("%s_kernel" % fam) in k]
    if not main_kernels:
        raise SystemExit("no %s kernel in %s" % (fam.upper(), directory))
    fetch_scale = write_scale = None
    out = {"workload": workload, "kernel_source_sha256": kernel_source_hash(fam),
           "source": {"directory": os.path.basename(os.path.normpath(directory)),
                      "summarized": datetime.date.today().isoformat(),
                      "note": "rocprofv3 --pmc passes of bench.py on one MI355X box; counters perturb "
                              "timing, so durations here run longer than in a kernel trace"}}
    if copy:
        cm = {c: statistics.median(v) for c, v in vals[copy[0]].items()}
        gib_kib = 1024.0 * 1024.0
        if cm.get("FETCH_SIZE"):
            fetch_scale = gib_kib / cm["FETCH_SIZE"]
        if cm.get("WRITE_SIZE"):
            write_scale = gib_kib / cm["WRITE_SIZE"]
        out["copy_calibration"] = {"kernel": copy[0], "bytes": 1 << 30, "counters_median": cm,
                                   "fetch_scale": fetch_scale, "write_scale": write_scale}
    per = {}
    for k in ours:
        med = {c: statistics.median(v) for c, v in vals[k].items()}
        per[k] = _kernel_metrics(med, statistics.median(durs[k]), fetch_scale, write_scale)
        per[k]["dispatches"] = len(durs[k]) // max(1, len(vals[k]))
    main = max(main_kernels, key=lambda n: per[n]["median_duration_ns"])
    out["kernel"] = main
    out["dispatches"] = per[main]["dispatches"]
    out.update({k: v for k, v in per[main].items() if k != "dispatches"})
    out["kernels"] = per
    # kernels of one call: dispatched once per call like the GEMM kernel (the
    # GEMM launches, the reduction, operand copies); kernels dispatched less
    # often are one-time set-up (zeroing a new workspace's counters)
    calls = per[main]["dispatches"]
    in_call = {k: p for k, p in per.items() if p["dispatches"] >= calls}
    out["per_call"] = {
        "kernels": len(in_call),
        "median_duration_ns": sum(p["median_duration_ns"] * p["dispatches"] / calls for p in in_call.values()),
        "setup_kernels": sorted(k for k in per if k not in in_call),
    }
    if all("hbm_bytes_per_launch" in p for p in in_call.values()):
        out["per_call"]["hbm_bytes"] = sum(p["hbm_bytes_per_launch"] * p["dispatches"] / calls
                                           for p in in_call.values())
    path = COUNTERS_FILE % workload
    with open(path, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
    return path


def settle(step, seconds: float, min_calls: int = 64) -> dict:
    """Run `step` until the GPU has reached its sustained clock under the
    power cap: at least min_calls calls and `seconds` of wall time (the host
    waits for the GPU every 16 calls, so the time is the GPU's).  From idle,
    the first tens of large GEMMs run 10-35% slower than the sustained rate
    while the power controller settles (8192^3: 823, 773, 933, 1029, 1004,
    946 ... us, then 734 us from about the 50th call on)."""
    import torch
    t0 = time.perf_counter()
    n = 0
    while n < min_calls or time.perf_counter() - t0 < seconds:
        step()
        n += 1
        if n % 16 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    return {"calls": n, "seconds": round(time.perf_counter() - t0, 3)}


def timed_region(step, steps: int, stream):
    """Exactly `steps` calls, bracketed by device synchronisation: the wall
    time, and the time between two HIP events recorded on the launch stream
    around them (the GPU is busy with the calls back to back in between, so
    that time over `steps` is the average duration of one call's kernels).
    Events between the calls would cost time of their own (0.8% at 8192^3,
    8% at 4096^3), so they are left to the per-call sample below."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, e0.elapsed_time(e1) * 1e-3


def per_call_times(step, calls: int, stream) -> np.ndarray:
    """Durations (s) of `calls` more calls, each between two HIP events: the
    sample of the paper's protocol (mean of the inter-quartile range)."""
    import torch
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(calls)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(calls)]
    torch.cuda.synchronize()
    for i in range(calls):
        starts[i].record(stream)
        step()
        ends[i].record(stream)
    torch.cuda.synchronize()
    return np.array([a.elapsed_time(b) for a, b in zip(starts, ends)]) * 1e-3


def iqr_mean(per: np.ndarray) -> float:
    srt = np.sort(per)
    q = len(srt) // 4
    return float(srt[q:len(srt) - q].mean()) if len(srt) >= 4 else float(srt.mean())


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), for the baseline's record."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, A, B, budget_s: float = 12.0):
    """The oracle, untuned, on a bounded sample: the first R rows of C."""
    import oracle
    oracle.build(force=False)
    cores = oracle.thread_count()
    # two probes separate the per-call cost (decoding B) from the per-row cost
    t0 = time.perf_counter()
    oracle.gemm_rows(A, B, w.dtype, np.arange(cores))
    t1 = time.perf_counter()
    oracle.gemm_rows(A, B, w.dtype, np.arange(4 * cores))
    t2 = time.perf_counter()
    per_row = max((t2 - t1) - (t1 - t0), 1e-4) / (3 * cores)
    rows = int(min(w.M, max(cores, budget_s / per_row)))
    t0 = time.perf_counter()
    oracle.gemm_rows(A, B, w.dtype, np.arange(rows))
    t = time.perf_counter() - t0
    flops = 2.0 * rows * w.N * w.K
    return {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": "rows 0..%d of C (%d x %d outputs, K=%d) of the %s workload, fp64, including "
                      "decoding B; %.1f s" % (rows - 1, rows, w.N, w.K, w.name, t)}


def gemv_cpu_baseline(w, A, x, budget_s: float = 10.0):
    """The oracle, untuned, on the whole GEMV workload, repeated for about
    budget_s seconds."""
    import oracle
    oracle.build(force=False)
    cores = oracle.thread_count()
    t0 = time.perf_counter()
    oracle.gemv(A, x)
    one = time.perf_counter() - t0
    reps = max(1, int(budget_s / max(one, 1e-3)))
    t0 = time.perf_counter()
    for _ in range(reps):
        oracle.gemv(A, x)
    t = (time.perf_counter() - t0) / reps
    return {"value": round(w.flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": "the whole %s workload (%d x %d), fp64, %d repetitions of %.3f s" % (w.name, w.M, w.K, reps, t)}


def bench_gemv(args, w):
    """The fp32 GEMV line: y = A x, one xgemv_run per step."""
    import torch
    from paper_2609_16389_amd import workloads as wl
    from paper_2609_16389_amd import xgemm as xg
    print("bench: workload %s M=%d K=%d fp32" % (w.name, w.M, w.K), file=sys.stderr, flush=True)
    A_np, x_np = wl.gemv_workload_inputs(w)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    A = torch.from_numpy(A_np).to(dev)
    x = torch.from_numpy(x_np).to(dev)
    y = torch.empty(w.M, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    h = xg.handle(0, stream)
    cfg = xg.xgemv_select_config(w.M, w.K, torch.cuda.get_device_properties(dev).multi_processor_count)

    def step():
        rc = xg.xgemv_run(h, w.M, w.K, A.data_ptr(), w.K, x.data_ptr(), y.data_ptr(), stream.cuda_stream)
        if rc != xg.XGEMM_OK:
            raise xg.XgemmError(rc, xg.xgemm_last_error(h))

    settled = settle(step, args.settle)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    wall, ev = timed_region(step, args.steps, stream)
    per = per_call_times(step, max(args.steps, 100), stream)
    value = w.flops * args.steps / wall / 1e12
    achieved_gbs = w.alg_bytes / (ev / args.steps) / 1e9
    peak_tflops = PEAK_HBM_GBS * 1e9 * 2 / 4 / 1e12
    iqr = iqr_mean(per)
    if args.copy_calibration:
        n = args.copy_calibration // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
    comparator = None
    if not args.no_comparator:
        for _ in range(3):
            torch.mv(A, x)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(20):
            torch.mv(A, x)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) * 1e-3 / 20
        comparator = {"name": "torch.mv (rocBLAS/hipBLASLt)", "tflops": round(w.flops / t / 1e12, 3),
                      "gbs": round(w.alg_bytes / t / 1e9, 1)}
    counters = stored_counters(w.name)
    out = {
        "metric": GEMV_METRIC % w.M,
        "value": round(value, 4),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle": settled,
        "ms_per_step": round(wall / args.steps * 1e3, 5),
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic (seeded uniform[-1,1], seed %d)" % w.seed,
        "config": {"workload": w.name, "M": w.M, "K": w.K, "rows": cfg.rows, "unroll": cfg.unroll},
        "pct_of_peak": round(100.0 * value / peak_tflops, 2),
        "paper_protocol_iqr_mean_tflops": round(w.flops / iqr / 1e12, 4),
        "roofline": {"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved_gbs / PEAK_HBM_GBS, 4),
                     "traffic": None if counters is None else counters.get("hbm_bytes_per_launch")},
        "comparator": comparator,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        print("bench: cpu baseline (oracle)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = gemv_cpu_baseline(w, A_np, x_np)
    print(json.dumps(out), flush=True)


SWEEP_MAX_WORKGROUPS = 4096  # configurations with more workgroups than this are not swept


def sweep_candidates(M: int, N: int, K: int, selected: tuple, xg) -> list:
    """(tile, split) pairs the sweep times for one shape: every tile with
    split-k 1, 2, 4, 8 and 16 where each split keeps 3 K steps and the launch
    has at most SWEEP_MAX_WORKGROUPS workgroups, plus the selected one."""
    out = {tuple(selected)}
    for tile in range(xg.XGEMM_TILE_COUNT):
        bm, bn, bk, _ = xg.xgemm_tile_info(tile)
        for split in (1, 2, 4, 8, 16):
            if split > 1 and K // split < 3 * bk:
                continue
            if -(-M // bm) * -(-N // bn) * split > SWEEP_MAX_WORKGROUPS:
                continue
            out.add((tile, split))
    return sorted(out)


def sweep_shape(M: int, N: int, K: int, dtype: str = "bf16", rounds: int = 5) -> dict:
    """Median time of every candidate configuration (and of xgemm_run's plan
    when it cuts C into a body and a band) on seeded uniform[-1, 1] inputs
    drawn on the device; configurations timed in shuffled order, several
    calls per timing."""
    import random
    import statistics
    import torch
    from paper_2609_16389_amd import xgemm as xg
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float16
    code = xg.XGEMM_BF16 if dtype == "bf16" else xg.XGEMM_FP16
    g = torch.Generator(device="cuda").manual_seed(M + N + K)
    A = (torch.rand(M, K, device="cuda", generator=g) * 2 - 1).to(tdt)
    B = (torch.rand(K, N, device="cuda", generator=g) * 2 - 1).to(tdt)
    C = torch.empty(M, N, device="cuda", dtype=torch.float32)
    stream = torch.cuda.current_stream()
    h = xg.handle(torch.cuda.current_device(), stream)
    cu = torch.cuda.get_device_properties(0).multi_processor_count
    sel = xg.xgemm_select_config(M, N, K, code, cu)
    band = xg.xgemm_select_band(M, N, K, code, cu)
    runs = []
    if band.axis != xg.XGEMM_BAND_NONE:
        def call_band():
            rc = xg.xgemm_run(h, M, N, K, A.data_ptr(), K, B.data_ptr(), N, C.data_ptr(), N, code, stream.cuda_stream)
            if rc != xg.XGEMM_OK:
                raise xg.XgemmError(rc)
        call_band()
        runs.append(("band", call_band))
    cands = [(t, sp, 0) for t, sp in sweep_candidates(M, N, K, (sel.tile, sel.split_k), xg)]
    sk = xg.xgemm_config(tile=xg.XGEMM_TILE_256x256, split_k=1, group_m=sel.group_m, stream_k=1)
    if xg.xgemm_kernel_family(M, N, K, A.data_ptr(), K, B.data_ptr(), N, sk) == xg.XGEMM_KERNEL_PERSISTENT:
        cands.append((xg.XGEMM_TILE_256x256, 1, 1))
    for tile, split, stream_k in cands:
        cfg = xg.xgemm_config(tile=tile, split_k=split, group_m=sel.group_m, stream_k=stream_k)

        def call(cfg=cfg):
            rc = xg.xgemm_run_config(h, M, N, K, A.data_ptr(), K, B.data_ptr(), N, C.data_ptr(), N, code,
                                     stream.cuda_stream, cfg)
            if rc != xg.XGEMM_OK:
                raise xg.XgemmError(rc)
        call()
        runs.append(("sk" if stream_k else (tile, split), call))
    torch.cuda.synchronize()
    reps = max(3, min(50, int(2e8 / max(1.0, 2.0 * M * N * K / 1e3))))
    times: dict = {k: [] for k, _ in runs}
    for _ in range(rounds):
        random.shuffle(runs)
        for key, call in runs:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            call()
            e0.record(stream)
            for _ in range(reps):
                call()
            e1.record(stream)
            torch.cuda.synchronize()
            times[key].append(e0.elapsed_time(e1) / reps * 1e3)
    med = {k: statistics.median(v) for k, v in times.items()}
    best = min(med, key=med.get)
    chosen = "band" if band.axis != xg.XGEMM_BAND_NONE else ("sk" if band.body.stream_k else (sel.tile, sel.split_k))
    name = lambda k: k if isinstance(k, str) else list(k)
    out = {"shape": [M, N, K], "dtype": dtype, "selected": name(chosen), "selected_us": round(med[chosen], 2),
           "best": name(best), "best_us": round(med[best], 2), "loss": round(med[chosen] / med[best], 3),
           "all_us": {(k if isinstance(k, str) else "%d:%d" % k): round(v, 1)
                      for k, v in sorted(med.items(), key=lambda kv: (isinstance(kv[0], str), str(kv[0])))}}
    if band.axis != xg.XGEMM_BAND_NONE:
        out["band"] = {"axis": "columns" if band.axis == xg.XGEMM_BAND_COLUMNS else "rows",
                       "body_extent": band.extent, "body": [band.body.tile, band.body.split_k],
                       "band": [band.band.tile, band.band.split_k]}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle", type=float, default=0.5,
                    help="seconds of untimed calls before the warmup steps, so that the timed steps run at "
                         "the GPU's sustained clock (0: only the minimum of 64 calls)")
    ap.add_argument("--workload", default="gemm8192_bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-comparator", action="store_true")
    ap.add_argument("--no-persistent", action="store_true",
                    help="switch the persistent kernel off for the bench handle (xgemm_set_persistent): the plan "
                         "xgemm_run takes without it, to compare the two")
    ap.add_argument("--copy-calibration", type=int, default=0,
                    help="also run a plain device copy of this many bytes (counter calibration)")
    ap.add_argument("--batch", type=int, default=0,
                    help="time xgemm_run_strided_batched on this many independent problems of the "
                         "workload's shape instead of one xgemm_run (one JSON line, no baselines)")
    ap.add_argument("--summarize-counters", metavar="DIR", default=None,
                    help="write profiles/counters_<workload>.json from rocprofv3 --pmc output and exit")
    ap.add_argument("--sweep", nargs="+", metavar="M,N,K", default=None,
                    help="time every (tile, split-k) configuration of these shapes against the selector's plan")
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "fp16"], help="--sweep: input type")
    ap.add_argument("--rounds", type=int, default=5, help="--sweep: timing rounds per configuration")
    args = ap.parse_args()

    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters, args.workload))
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this GEMM is not sharded across GPUs "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_16389_amd import workloads as wl
    from paper_2609_16389_amd import xgemm as xg

    if args.sweep:
        for shape in args.sweep:
            M, N, K = (int(v) for v in shape.split(","))
            print(json.dumps(sweep_shape(M, N, K, args.dtype, args.rounds)), flush=True)
        return
    if args.workload in wl.GEMV_WORKLOADS:
        bench_gemv(args, wl.GEMV_WORKLOADS[args.workload])
        return
    w = wl.WORKLOADS[args.workload]
    print("bench: workload %s M=%d N=%d K=%d %s" % (w.name, w.M, w.N, w.K, w.dtype), file=sys.stderr, flush=True)
    A_bits, B_bits = wl.workload_inputs(w)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float16
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    A = torch.from_numpy(A_bits.view(np.int16)).to(dev).view(tdt)
    B = torch.from_numpy(B_bits.view(np.int16)).to(dev).view(tdt)
    C = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    h = xg.handle(0, stream)
    if args.no_persistent and xg.xgemm_set_persistent(h, 0) != xg.XGEMM_OK:
        raise SystemExit("xgemm_set_persistent failed")
    code = xg.XGEMM_BF16 if w.dtype == "bf16" else xg.XGEMM_FP16
    plan = xg.xgemm_select_plan(w.M, w.N, w.K, code, torch.cuda.get_device_properties(dev).multi_processor_count,
                                0 if args.no_persistent else 1)
    cfg = plan.body  # the whole call's configuration, or the body's when C is cut in two
    kernel_family = xg.xgemm_kernel_family(w.M, w.N, w.K, A.data_ptr(), w.K, B.data_ptr(), w.N, cfg)

    def step():
        rc = xg.xgemm_run(h, w.M, w.N, w.K, A.data_ptr(), w.K, B.data_ptr(), w.N, C.data_ptr(), w.N,
                          code, stream.cuda_stream)
        if rc != xg.XGEMM_OK:
            raise xg.XgemmError(rc, xg.xgemm_last_error(h))

    if args.batch > 0:
        # independent problems: the workload's A and B followed by re-seeded copies
        L = args.batch
        Ab = torch.empty((L, w.M, w.K), dtype=tdt, device=dev)
        Bb = torch.empty((L, w.K, w.N), dtype=tdt, device=dev)
        for b in range(L):
            if b == 0:
                Ab[0].copy_(A)
                Bb[0].copy_(B)
            else:
                a_bits, b_bits = wl.make_inputs(w.M, w.N, w.K, w.dtype, w.dist, w.seed + 1000 * b, w.param)
                Ab[b].copy_(torch.from_numpy(a_bits.view(np.int16)).to(dev).view(tdt))
                Bb[b].copy_(torch.from_numpy(b_bits.view(np.int16)).to(dev).view(tdt))
        Cb = torch.empty((L, w.M, w.N), dtype=torch.float32, device=dev)
        settled = settle(lambda: xg.bmm(Ab, Bb, out=Cb), args.settle)
        for _ in range(args.warmup):
            xg.bmm(Ab, Bb, out=Cb)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            xg.bmm(Ab, Bb, out=Cb)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) * 1e-3 / args.steps
        print(json.dumps({"metric": "strided batched GEMM TFLOP/s", "value": round(L * w.flops / t / 1e12, 2),
                          "unit": "TFLOP/s", "batch": L, "ms_per_step": round(t * 1e3, 4), "dtype": w.dtype,
                          "settle": settled,
                          "config": {"workload": w.name, "M": w.M, "N": w.N, "K": w.K}}), flush=True)
        return

    settled = settle(step, args.settle)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("bench: settled (%d calls, %.2f s), warmup done" % (settled["calls"], settled["seconds"]),
          file=sys.stderr, flush=True)

    # timed region: exactly K steps, bracketed by synchronisation, with two
    # HIP events on the launch stream around them (the kernels' average
    # duration); then a per-call sample for the paper's protocol
    wall, ev = timed_region(step, args.steps, stream)
    print("bench: timed %d steps in %.3f s" % (args.steps, wall), file=sys.stderr, flush=True)
    per = per_call_times(step, max(args.steps, 100), stream)

    flops = float(w.flops)
    ms_per_step = wall / args.steps * 1e3
    value = flops * args.steps / wall / 1e12
    achieved = flops / (ev / args.steps) / 1e12
    iqr = iqr_mean(per)
    peak = PEAK_TFLOPS[w.dtype]

    if args.copy_calibration:
        n = args.copy_calibration // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    comparator = None
    if not args.no_comparator:
        # torch.matmul (hipBLASLt) on the same inputs, bf16/fp16 output; context only
        for _ in range(3):
            torch.matmul(A, B)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(20):
            torch.matmul(A, B)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) * 1e-3 / 20
        comparator = {"name": "torch.matmul (hipBLASLt), 16-bit output", "tflops": round(flops / t / 1e12, 1)}

    traffic = stored_traffic(w.name)
    counters = stored_counters(w.name)
    out = {
        # the headline metric for the 8192^3 workload; the same quantity,
        # named for its shape, for the others
        "metric": METRIC if w.name == "gemm8192_bf16" else
        "GEMM TFLOP/s and %% of MI355X dense MFMA peak (%s, %dx%dx%d) on 1 GPU" % (w.dtype, w.M, w.N, w.K),
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle": settled,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded uniform[-1,1], seed %d)" % w.seed if w.dist == "uniform"
                else "synthetic (seeded normal(0,%g), seed %d)" % (w.param, w.seed),
        "config": dict({"workload": w.name, "M": w.M, "N": w.N, "K": w.K, "out": "fp32",
                        "tile": cfg.tile, "split_k": cfg.split_k,
                        "kernel": "persistent" if kernel_family == xg.XGEMM_KERNEL_PERSISTENT else
                        "pipelined" if kernel_family == xg.XGEMM_KERNEL_PIPELINED else "general"},
                       **({} if plan.axis == xg.XGEMM_BAND_NONE else {"band": {
                           "axis": "columns" if plan.axis == xg.XGEMM_BAND_COLUMNS else "rows",
                           "body_extent": plan.extent, "tile": plan.band.tile,
                           "split_k": plan.band.split_k}})),
        "pct_of_peak": round(100.0 * value / peak, 2),
        "paper_protocol_iqr_mean_tflops": round(flops / iqr / 1e12, 2),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4),
                     "traffic": traffic},
        "comparator": comparator,
        # counters and roofline.traffic are not measured by this run: they
        # come from the committed rocprofv3 --pmc summary of the same kernel
        # sources, taken on another MI355X
        "counters": None if counters is None else dict({
            k: counters.get(k) for k in ("mfma_busy_pct", "clock_ghz", "lds_bank_conflict_pct",
                                         "hbm_read_bytes_per_launch", "hbm_write_bytes_per_launch")},
            source="committed profile profiles/counters_%s.json (another box; kernel sources %s)"
                   % (w.name, counters.get("kernel_source_sha256"))),
        "traffic_source": None if traffic is None else "committed profile profiles/counters_%s.json" % w.name,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        print("bench: cpu baseline (oracle)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, A_bits, B_bits)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
