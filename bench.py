#!/usr/bin/env python3
"""Benchmark: achieved HBM GB/s of OptCC schedule execution on one MI355X.

One step = one call of optcc_allreduce_emulate over a whole workload: every
step of the OptCC schedule for p rank buffers resident in HBM (one fused
kernel launch).  Prints one JSON line.  The headline is the p = 8 workload
(one of eight NICs lost on one rank); the default run also measures every
headline configuration the same way (p4_f32, p8_f32, p8_i32, p16_bf16,
p64_f32, p128_f32) and reports them under "configs".

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload p8_f32]
    python bench.py --trace-summary kernel_trace.csv --line bench_line.json
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
METRIC = "achieved HBM GB/s of OptCC schedule execution (1 GPU) and % of peak BW"
PEAK_GBPS = 8000.0  # MI355X HBM3E
NIC_BYTES_PER_S = 25e9  # one healthy 200 Gb/s NIC, for the model times in seconds
# device code of the executor (kernels, table layouts, launch choices)
KERNEL_SRCS = [os.path.join(ROOT, "paper_2606_01680_amd", "csrc", f)
               for f in ("optcc_kernels.hpp", "optcc_internal.hpp", "optcc_launch.hpp",
                         "optcc_exec.hip", "optcc_kern_f32.hip", "optcc_kern_bf16.hip",
                         "optcc_kern_i32.hip", "optcc_kern_f16.hip",
                         "optcc_kern_f32_g58.hip", "optcc_kern_bf16_g58.hip",
                         "optcc_kern_i32_g58.hip", "optcc_kern_f16_g58.hip")]


def _code_only(text: str) -> str:
    """C/C++ source without comments and with whitespace collapsed, so that
    comment and layout edits keep the hash; string and character literals
    are kept as they are."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":  # literal: copy through its closing quote
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            i = text.find("\n", i)
            i = n if i < 0 else i
        elif text.startswith("/*", i):
            i = text.find("*/", i + 2)
            i = n if i < 0 else i + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_hash() -> str:
    """sha256 (first 16 hex digits) of the device code, comments excluded."""
    h = hashlib.sha256()
    for f in KERNEL_SRCS:
        h.update(_code_only(open(f, encoding="utf-8").read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, launches: int):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they
    were taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    d = json.load(open(path))
    if d.get("kernel_sha256_16") != kernel_hash() or d.get("launches", 1) != launches:
        return None
    return d.get("bytes_per_launch")


# what each stage slot of the executor runs (one GPU per server; several)
SLOT_NAMES = ["S3 of ordering 2: stragglers' values into the chain start",
              "S1 reduce-scatter chain", "S2 upload; P2P up", "S3 download; P2P down",
              "S4 allgather", "S2 of ordering 2: global sum to the stragglers"]
SERVER_SLOT_NAMES = ["N3 collect on the straggler server (type 2)",
                     "N1 collect on the healthy servers", "S3 into the chain start (type 2)",
                     "S1 reduce-scatter chain", "S2 straggler leader adds (type 1)",
                     "N2 fold on the straggler server (type 1)",
                     "N3 copy back on the straggler server (type 1)",
                     "S3 download (type 1)", "S4 allgather", "N4 distribute",
                     "S2 download to the straggler leader (type 2)",
                     "N2 distribute on the straggler server (type 2)"]


def stage_breakdown(torch, optcc, x, w, plan, steps, warmup):
    """Each stage slot timed on its own (one launch of that slot: a lane
    loads the state its first step needs), with its algorithmic bytes."""
    names = SERVER_SLOT_NAMES if w.g > 1 else SLOT_NAMES
    E = torch.cuda.Event
    out = []
    for s in range(plan.num_slots):
        rd, wr = plan.traffic(w.dtype, s, s + 1, 1)
        if rd + wr == 0:
            continue

        def run():
            optcc.optcc_allreduce_emulate_slots(x, w.p, w.n, w.dtype, plan, s, s + 1, 1)

        for _ in range(warmup):
            run()
        evs = [(E(enable_timing=True), E(enable_timing=True)) for _ in range(steps)]
        for a, b in evs:
            a.record()
            run()
            b.record()
        torch.cuda.synchronize()
        ms = statistics.median(a.elapsed_time(b) for a, b in evs)
        out.append({"slot": s, "stage": names[s], "ms_median": round(ms, 5),
                    "bytes": rd + wr, "GBps": round((rd + wr) / (ms * 1e-3) / 1e9, 2)})
    return out


def host_info():
    """CPU model, logical CPUs of the host and CPUs this process may use."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        usable = os.cpu_count()
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cpus": usable}


def oracle_threads():
    """Threads for the all-cores leg: OMP_NUM_THREADS when set (the CPU
    share of the process), else every CPU this process may use."""
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return int(env)
    return host_info()["usable_cpus"]


def cpu_leg(w, x0, plan, traffic_bytes, budget_s, threads):
    """The oracle, untuned, on a bounded sample of whole segments, reported in
    the metric's unit (algorithmic bytes of the sample / oracle time).
    threads = 1: the serial C executor; otherwise the same steps on
    `threads` OpenMP threads (bit-identical results).  When the whole
    workload runs in less than the budget it is run again (inputs restored,
    untimed) until the budget is spent, and the mean is reported."""
    import numpy as np
    import oracle

    off, ln, _ = plan.segments()
    total = plan.num_segments
    host = None

    def run(nseg):
        nonlocal host
        end = int(off[nseg - 1] + ln[nseg - 1])
        if host is None or host.shape[1] < end:
            host = np.empty((w.p, w.n), dtype=oracle.NP_DTYPES[w.dtype])
        src = x0[:, :end].cpu()
        if w.dtype in ("bf16", "f16"):
            import torch
            host[:, :end] = src.view(torch.int16).numpy().view(np.uint16)
        else:
            host[:, :end] = src.numpy()
        if w.g > 1:
            sched = oracle.Schedule.servers(w.q, w.g, w.bandwidths, w.n, w.k, seg_lo=0, seg_hi=nseg)
        else:
            sched = oracle.Schedule(w.p, w.bandwidths, w.n, w.k, seg_lo=0, seg_hi=nseg)
        t = time.perf_counter()
        if threads == 1:
            oracle.run(sched, w.dtype, host)
        else:
            oracle.run_parallel(sched, w.dtype, host, threads)
        return time.perf_counter() - t, end

    first = min(total, threads)  # at least one segment per thread
    t1, _ = run(first)
    nseg = int(max(first, min(total, first * budget_s / max(t1, 1e-6))))
    times = []
    while not times or (nseg == total and sum(times) < budget_s and len(times) < 20):
        t, elems = run(nseg)
        times.append(t)
    t = sum(times) / len(times)
    bytes_sample = traffic_bytes * elems / w.n
    how = "serial C oracle" if threads == 1 else f"the oracle's steps on {threads} OpenMP threads"
    return {"value": round(bytes_sample / t / 1e9, 4), "unit": "GB/s", "cores": threads,
            "sample": f"first {nseg} of {total} segments ({elems} of {w.n} elements per rank), "
                      f"{how}, mean of {len(times)} run(s) of {t:.3f} s"}


def brute_leg(w, x0, budget_s):
    """The definition of the result timed on the host: every coordinate's
    sum over the ranks in fp64 (int64 wrapped to int32), numpy, on leading
    coordinates of the workload (whole vector if it fits the budget).  The
    rate counts the input bytes it reads."""
    import numpy as np
    import oracle

    def run(end):
        src = x0[:, :end].cpu()
        if w.dtype in ("bf16", "f16"):
            import torch
            host = src.view(torch.int16).numpy().view(np.uint16)
        else:
            host = src.numpy()
        t = time.perf_counter()
        oracle.brute_sum(w.dtype, host)
        return time.perf_counter() - t

    end = min(w.n, 1 << 16)
    t = run(end)
    end = int(min(w.n, max(end, end * budget_s / max(t, 1e-6))))
    t = run(end)
    in_bytes = w.p * end * (2 if w.dtype in ("bf16", "f16") else 4)
    return {"value": round(in_bytes / t / 1e9, 4), "unit": "GB/s of input read", "cores": 1,
            "seconds": round(t, 4),
            "sample": f"first {end} of {w.n} elements per rank, all {w.p} ranks",
            "kind": "brute force: fp64 (int64 for int32) sum over the ranks, numpy "
                    "(the definition of the result, not the schedule)"}


def cpu_baseline(w, x0, plan, traffic_bytes, serial_s, parallel_s):
    """Two legs: the serial oracle on one core, and the same executor on all
    the cores this process may use; beside them the brute-force sum."""
    serial = cpu_leg(w, x0, plan, traffic_bytes, serial_s, 1)
    threads = oracle_threads()
    par = cpu_leg(w, x0, plan, traffic_bytes, parallel_s, threads)
    out = dict(serial)
    out["kind"] = "oracle"
    out["all_cores"] = dict(par, kind="oracle, OpenMP over segments (bit-identical to serial)")
    out["brute_force"] = brute_leg(w, x0, min(2.0, parallel_s))
    out.update(host_info())
    return out


def copy_rate(torch, nbytes, steps, warmup):
    """(ms, GB/s read + write) of torch's plain device-to-device copy of
    nbytes: the streaming ceiling of one read and one write stream."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    del src, dst
    return ms, 2 * nbytes / (ms * 1e-3) / 1e9


def copy_bench(torch, args):
    """A plain copy of a known size: reads and writes copy_bytes each."""
    ms, gbps = copy_rate(torch, args.copy_bytes, args.steps, args.warmup)
    print(json.dumps({"copy_bytes": args.copy_bytes, "ms": round(ms, 5),
                      "GBps_read_plus_write": round(gbps, 2)}), flush=True)


BASELINE_CONFIGS = ["p4_f32", "p8_f32", "p8_i32", "p16_bf16", "p64_f32", "p128_f32"]


def full_check(torch, w, x, x0):
    """Properties at full size: all ranks bitwise identical, and every element
    within the error bound of the exact sum (exactly the wrapped sum for
    int32).  x holds the result of one AllReduce of x0."""
    iv = x.view(torch.int16) if x.element_size() == 2 else x.view(torch.int32)
    ok = all(torch.equal(iv[r], iv[0]) for r in range(1, w.p))
    chunk = max(1 << 16, (1 << 28) // w.p)
    for c0 in range(0, w.n, chunk):
        c1 = min(w.n, c0 + chunk)
        if w.dtype == "i32":
            want = x0[:, c0:c1].to(torch.int64).sum(0)
            ok &= torch.equal(x[0, c0:c1], ((want + 2**31) % 2**32 - 2**31).to(torch.int32))
        else:
            xs = x0[:, c0:c1].to(torch.float64)
            u = {"f32": 2.0 ** -24, "f16": 2.0 ** -11, "bf16": 2.0 ** -8}[w.dtype]
            err = (x[0, c0:c1].to(torch.float64) - xs.sum(0)).abs()
            ok &= bool((err <= w.p * u * xs.abs().sum(0)).all())
    return "pass" if ok else "FAIL"


def model_times(optcc, w, plan):
    """Model times of the paper's bandwidth model, in units of N element-times."""
    n = w.n
    t_model = optcc.optcc_model_time(plan) / n
    if w.g > 1:
        lb = optcc.optcc_lower_bound_servers(w.q, w.g, w.bandwidths, n) / n
    else:
        lb = optcc.optcc_lower_bound(w.p, w.bandwidths, n) / n
    t0_ring = 2.0 * (w.p - 1) / (w.g * w.p)  # fault-free optimum with g GPUs per server
    # the same flows timed in the paper's network model (the pattern overlay of
    # Sec. 4.2 and App. D; list scheduling for several GPUs per server)
    evaluated = None
    if plan.num_flows <= (1 << 24):
        evaluated = round(plan.timeline(with_flows=False)[0] / n, 6)
    return {"optcc": round(t_model, 6), "evaluated_schedule": evaluated,
            "fault_free_ring_T0": round(t0_ring, 6), "lower_bound": round(lb, 6),
            "degraded_ring": round(float(max(plan.slowdowns)) * t0_ring, 6)}


def measure(torch, optcc, w, args, check=True):
    """Time args.steps back-to-back AllReduces of workload w (after
    args.warmup untimed ones) between one pair of HIP events, then time the
    same number again with an event pair around each step (the spread of
    the step times; events between launches cost a few microseconds per
    step, so they stay out of the timed region), then check one more at
    full size.  Returns the record and what the CPU baseline needs;
    `launches` counts the executor's kernel launches issued."""
    from paper_2606_01680_amd.workloads import make_inputs

    x = make_inputs(w, device="cuda:0")
    x0 = x.clone()
    if w.g > 1:  # q servers of g GPUs (App. E)
        plan = optcc.optcc_plan_servers(w.q, w.g, w.bandwidths, w.n, w.k)
    else:
        plan = optcc.optcc_plan(w.p, w.bandwidths, w.n, w.k)
    nslots = plan.num_slots
    rd, wr = plan.traffic(w.dtype, 0, nslots, args.launches)
    alg_bytes = rd + wr
    per_call = 1 if args.launches == 1 else nslots

    def step():
        optcc.optcc_allreduce_emulate_slots(x, w.p, w.n, w.dtype, plan, 0, nslots, args.launches)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    E = torch.cuda.Event
    t0, t1 = E(enable_timing=True), E(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record()
    for _ in range(args.steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / args.steps
    # the mean launch time over the timed region (per_call launches a step)
    ms_launch = ms_step
    evs = [(E(enable_timing=True), E(enable_timing=True)) for _ in range(args.steps)]
    for a, b in evs:
        a.record()
        step()
        b.record()
    torch.cuda.synchronize()
    launch_ms = [a.elapsed_time(b) for a, b in evs]
    launches = (args.warmup + 2 * args.steps) * per_call

    stages = None
    if args.stages:
        stages = stage_breakdown(torch, optcc, x, w, plan, args.steps, args.warmup)
        launches += len(stages) * (args.steps + args.warmup)

    result = "skipped"
    if check:  # the timed path computes the sum: properties at full size
        x.copy_(x0)
        step()
        torch.cuda.synchronize()
        launches += per_call
        result = full_check(torch, w, x, x0)
    del x

    # torch's device copy of as many bytes as the rank buffers hold, timed
    # in the same run: a reference rate of one read and one write stream
    buf_bytes = w.p * w.n * (2 if w.dtype in ("bf16", "f16") else 4)
    copy_ms, copy_gbps = copy_rate(torch, buf_bytes, max(args.steps, 5), 2)
    torch.cuda.empty_cache()

    achieved = alg_bytes / (ms_launch * 1e-3) / 1e9
    # counter traffic was taken at the workload's own N
    traffic = measured_traffic(w.name, args.launches) if args.n is None else None
    rec = {
        "workload": w.name, "p": w.p, "N": w.n, "n_chunks": w.k, "dtype": w.dtype,
        "gpus_per_server": w.g,
        "stragglers": {str(int(r)): float(w.bandwidths[int(r)]) for r in plan.stragglers},
        "values": w.values, "plan_kind": plan.kind, "launches_per_step": per_call,
        "ms_per_step": round(ms_step, 5),
        "GBps": round(alg_bytes / (ms_step * 1e-3) / 1e9, 2),
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_GBPS, "unit": "GB/s",
            "frac": round(achieved / PEAK_GBPS, 4),
            "basis": "achieved and frac: algorithmic bytes (every rank input read once, "
                     "every step's destination written) per mean step time of the timed "
                     "region (kernel_ms); traffic_GBps and traffic_frac: rocprofv3 "
                     "FETCH_SIZE + WRITE_SIZE bytes (L2 to memory fabric) per step; "
                     "kernel_ms_median and kernel_ms_min: a second pass with an event pair "
                     "around each step",
            "traffic": traffic,
            "traffic_GBps": None if traffic is None else round(traffic / (ms_launch * 1e-3) / 1e9, 2),
            "traffic_frac": None if traffic is None else round(
                traffic / (ms_launch * 1e-3) / 1e9 / PEAK_GBPS, 4),
            "algorithmic_bytes": alg_bytes, "read_bytes": rd, "write_bytes": wr,
            "kernel_ms": round(ms_launch, 5),
            "kernel_ms_median": round(statistics.median(launch_ms), 5),
            "kernel_ms_min": round(min(launch_ms), 5), "kernel": "optcc_exec_kernel",
        },
        "copy_reference": {
            "kernel": "torch copy_ (the runtime's blit kernel)", "bytes": buf_bytes,
            "ms": round(copy_ms, 5), "GBps_read_plus_write": round(copy_gbps, 2),
            "achieved_over_copy": round(achieved / copy_gbps, 4),
            "traffic_over_copy": None if traffic is None else round(
                traffic / (ms_launch * 1e-3) / 1e9 / copy_gbps, 4),
        },
        "model_time_over_N": model_times(optcc, w, plan),
        "check": result,
        "wall_s_timed": round(wall, 4),
        "executor_launches": launches,
    }
    if stages is not None:
        rec["stages"] = stages
    return rec, x0, plan, alg_bytes


def trace_summary(csv_path, line_path):
    """Split a rocprofv3 kernel trace of one bench run by workload: the
    executor's dispatches, in dispatch order, belong to the workloads in the
    order the bench line lists them (dispatch_order), so each workload's
    average kernel duration can be set beside its line figures."""
    import csv

    line = None
    for text in open(line_path):
        text = text.strip()
        if text.startswith("{") and '"metric"' in text:
            line = json.loads(text)
    if line is None:
        raise SystemExit(f"no bench line in {line_path}")
    rows = []
    with open(csv_path, newline="") as f:
        for r in csv.DictReader(f):
            if "optcc_exec_kernel" in r["Kernel_Name"]:
                rows.append((int(r["Dispatch_Id"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"]),
                             r["Kernel_Name"]))
    rows.sort()
    order = line["dispatch_order"]
    if sum(n for _, n in order) != len(rows):
        raise SystemExit(f"trace has {len(rows)} executor dispatches, the line lists "
                         f"{sum(n for _, n in order)}")
    recs = dict(line.get("configs", {}))
    recs.setdefault(line["config"]["workload"], {"roofline": line["roofline"]})
    print("| Workload | Kernel | Dispatches | Avg ns | Min ns | Max ns | bench kernel_ms | "
          "alg. GB/s at the trace average | frac |")
    print("|---|---|---|---|---|---|---|---|---|")
    at = 0
    for name, n in order:
        part = rows[at:at + n]
        at += n
        ns = [d for _, d, _ in part]
        names = sorted(set(k for _, _, k in part))
        roof = recs[name]["roofline"]
        avg = sum(ns) / len(ns)
        rate = roof["algorithmic_bytes"] / avg
        print(f"| {name} | {' / '.join(names)} | {n} | {avg:,.0f} | {min(ns):,} | {max(ns):,} | "
              f"{roof['kernel_ms']} | {rate:,.1f} | {rate / PEAK_GBPS:.4f} |")


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None,
                    help="one workload only (default: the p8_f32 headline plus every "
                         "headline configuration under \"configs\")")
    ap.add_argument("--launches", type=int, default=1, choices=[0, 1],
                    help="1: fused (default); 0: one launch per stage slot")
    ap.add_argument("--stages", action="store_true",
                    help="also time every stage slot on its own (per-stage breakdown)")
    ap.add_argument("--no-configs", action="store_true",
                    help="measure the headline (or --workload) only")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-check", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="budget of the headline's serial oracle leg (the all-cores leg gets "
                         "half, every other configuration a fifth per leg)")
    ap.add_argument("--copy-only", action="store_true",
                    help="time torch's plain device-to-device copy instead (the reference "
                         "kernel for scaling rocprofv3 byte counters)")
    ap.add_argument("--copy-bytes", type=int, default=1 << 30)
    ap.add_argument("--n", type=int, default=None,
                    help="elements per rank instead of the workload's own N (message-size "
                         "sweeps); the line then reports that N and no counter traffic")
    ap.add_argument("--trace-summary", metavar="CSV", default=None,
                    help="split a rocprofv3 kernel trace of a bench run by workload (no GPU)")
    ap.add_argument("--line", metavar="FILE", default=None,
                    help="the bench run's output, holding its JSON line (with --trace-summary)")
    args = ap.parse_args()
    if args.trace_summary:
        if not args.line:
            ap.error("--trace-summary needs --line")
        trace_summary(args.trace_summary, args.line)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the OptCC emulation runs the p logical ranks on ONE GPU; "
              "it takes --gpus 1 only.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_01680_amd import optcc
    from paper_2606_01680_amd.workloads import ESIZE, WORKLOADS

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_only:
        copy_bench(torch, args)
        return
    sweep = args.workload is None and args.n is None and not args.no_configs
    w = WORKLOADS[args.workload or "p8_f32"]
    if args.n is not None:
        import dataclasses
        if args.n < 1:
            print("bench.py: --n must be >= 1", file=sys.stderr)
            sys.exit(2)
        w = dataclasses.replace(w, n=args.n)

    rec, x0, plan, alg_bytes = measure(torch, optcc, w, args, check=not args.no_check)
    order = [[w.name, rec["executor_launches"]]]
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, x0, plan, alg_bytes, args.cpu_seconds, args.cpu_seconds / 2)
    del x0
    torch.cuda.empty_cache()
    n = w.n
    times = rec["model_time_over_N"]
    out = {
        "metric": METRIC,
        "value": rec["GBps"],
        "unit": "GB/s",
        "value_basis": "algorithmic bytes of the AllReduce's steps / ms_per_step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": rec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": w.name, "p": w.p, "N": w.n, "n_chunks": w.k,
            "gpus_per_server": w.g, "stragglers": rec["stragglers"], "values": w.values,
            "launches_per_step": rec["launches_per_step"], "plan_kind": plan.kind,
        },
        "roofline": rec["roofline"],
        "copy_reference": rec["copy_reference"],
        "model_time_over_N": times,
        # the same model times in seconds for this message on healthy
        # 200 Gb/s NICs (25 GB/s, the paper's ConnectX-6 HDR setting)
        "model_seconds_at_25GBps_nic": {
            k: round(times[key] * n * ESIZE[w.dtype] / NIC_BYTES_PER_S, 6)
            for k, key in (("optcc", "optcc"), ("fault_free_ring_T0", "fault_free_ring_T0"),
                           ("lower_bound", "lower_bound"))},
        "check": rec["check"],
        "kernel_sha256_16": kernel_hash(),
        "wall_s_timed": rec["wall_s_timed"],
    }
    if "stages" in rec:
        out["stages"] = rec["stages"]
    if cpu is not None:
        out["cpu_baseline"] = cpu
    failed = rec["check"] == "FAIL"
    if sweep:
        configs = {}
        for name in BASELINE_CONFIGS:
            if name == w.name:
                r = {k: v for k, v in rec.items() if k not in ("executor_launches", "stages")}
                if cpu is not None:
                    r["cpu_baseline"] = {"serial": {k: cpu[k] for k in ("value", "cores", "sample")},
                                         "all_cores": cpu["all_cores"],
                                         "brute_force": cpu["brute_force"]}
                configs[name] = r
                continue
            print(f"bench: measuring {name}", file=sys.stderr, flush=True)
            wc = WORKLOADS[name]
            r, xc, pc, bc = measure(torch, optcc, wc, args, check=not args.no_check)
            order.append([name, r.pop("executor_launches")])
            if not args.no_cpu_baseline:
                legs = args.cpu_seconds / 5
                r["cpu_baseline"] = {"serial": cpu_leg(wc, xc, pc, bc, legs, 1),
                                     "all_cores": cpu_leg(wc, xc, pc, bc, legs, oracle_threads()),
                                     "brute_force": brute_leg(wc, xc, min(1.0, legs))}
            del xc
            torch.cuda.empty_cache()
            failed |= r["check"] == "FAIL"
            configs[name] = r
        out["configs"] = configs
    out["dispatch_order"] = order
    print(json.dumps(out), flush=True)
    if failed:
        sys.exit(3)


if __name__ == "__main__":
    main()
