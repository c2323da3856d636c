"""Benchmark of the clairvoyant planning path on one MI355X.

One step = the whole path on one job: access streams -> access stats ->
next reuse -> tier plan, with inputs (sizes) resident in HBM and outputs
preallocated; by default one nopfs_plan_job call (--path staged: the four
stage calls). The metric is planned sample-accesses per second: the number of
reads the job issues (A = N * E * L) over the device time of one step.

After the timed steps, the per-tier prefetch queues and the staging
schedule of the planned job (the step's outputs as inputs, the workload's
staging-buffer capacity as d0) are timed the same way and reported under
"schedule", the performance model's fetch sources and consumption times
(the simulated cluster's parameters) under "model", and the clairvoyant
buffer replay (the staging capacity) under "buffer", and the simulator's
four data-loading policies (Perfect, Naive, StagingBuffer, NoPFS) under
"policies"; they are not part of the step.

The later calls, timed after the step, warm up with at most 2 calls of their
own.

Prints ONE JSON line. Per-kernel durations come from HIP events recorded by
the library around each of its launches, on the stream it launches on, over
the timed steps. The dominant kernel's roofline uses the algorithmic bytes of
its stage (the bytes the stage must read and write given the C ABI's dense
layouts), and the HBM traffic measured by rocprofv3 counters (summary under
profiles/) when that summary matches the current kernel sources.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "planned sample-accesses/sec (E×F×stats+plan) and % of HBM peak, 1 MI355X"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
DEFAULT_WORKLOAD = "imagenet22k"


def algorithmic_bytes(job, M_w, D, fused):
    """Bytes each kernel must move given the C ABI's dense layouts, per
    launch: A reads, N*F cells, D distinct (worker, sample) cells read. In the
    fused call the counting pass also lists the D read cells (4 B each: the
    cell's bin and offset) and the tier plan reads that list instead of the
    dense count/first tables."""
    A = int(sum(M_w))
    NF = job.N * job.F
    out = {
        # streams: write R (4 B per read)
        "stream_sort": 4 * A,
        # stats: read R (partitioned), write count (1 B) and first (4 B) per cell
        "stats_tile": 4 * A + 5 * NF + (4 * D if fused else 0),
        # next: read R, write next
        "next_unpartition": 8 * A,
        "seg_partition": 8 * A,
        "next_tile": 8 * A,
        "stream_scatter": 8 * job.E * job.F,
    }
    if fused:
        # list entry and the size of each read cell; tier bytes for every cell
        out["plan_hist"] = 12 * D
        out["plan_write"] = 4 * D + NF
    else:
        # read count and first (and sizes), write tier
        out["plan_hist"] = 5 * NF + 8 * job.F
        out["plan_write"] = 5 * NF + NF
    return out, A


def schedule_algorithmic_bytes(job, M, M_w):
    """Bytes the two schedule calls must move given the C ABI's dense
    layouts, attributed to the kernel that moves them: A reads, N*F cells,
    M_max positions per row. The prefetch order reads R once (its first reads
    are R's), the tier of every cell, and writes the whole order table; the
    staging schedule reads R once, each sample's size once and writes the
    whole fill table. Everything else (the partition of R, codes and sizes in
    partitioned order, per-chunk counts, scans and prefix sums, and the
    second read of R for the queued samples) is the implementation's own
    scratch traffic."""
    A = int(sum(M_w))
    NF = job.N * job.F
    NM = job.N * M
    prefetch = {"seg_partition": 4 * A, "pf_tile": NF, "pf_write": 4 * NM}
    staging = {"seg_partition": 4 * A, "st_tile": 8 * job.F, "st_fill": 4 * NM}
    return prefetch, staging


def model_algorithmic_bytes(job, M, M_w):
    """Bytes the performance-model call must move given the dense layouts:
    R once, every worker's tier of every sample (the holders of each sample)
    and each sample's size once, and the source (2 B) and time (8 B) of
    every position."""
    A = int(sum(M_w))
    return {"seg_partition": 4 * A, "fm_holders": job.N * job.F + 8 * job.F,
            "fm_final": 10 * job.N * M}


def kernel_source_hash():
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_2101_08734_amd", "csrc", "*"))):
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def committed_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary, or None if absent or taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    for line in open(path):
        line = line.strip()
        if line.startswith("{"):
            d = json.loads(line)
            if d.get("source_hash") != kernel_source_hash():
                return None
            k = d.get("kernels", {}).get(kernel)
            return None if k is None else k.get("hbm_bytes_per_launch")
    return None


POLICY_NAMES = ("perfect", "naive", "staging", "nopfs")
SEQUENTIAL_NOTE = ("sequential per worker (each read depends on every earlier one), one wave "
                   "per worker: bound by the wave's instruction issue and latency, not by HBM; "
                   "frac is the HBM fraction for reference")


def _kernel_short_name(full):
    """'ns::(anonymous namespace)::plan_hist<true>(args...)' -> 'plan_hist';
    the policy kernel keeps its policy: 'ps_sim<2>(...)' -> 'ps_sim_staging'."""
    import re
    m = re.findall(r"(\w+)(?:<([^>()]*)>)?\(", full)
    if not m:
        return full
    name, targ = m[-1]
    if name == "ps_sim" and targ.strip().isdigit() and int(targ) < len(POLICY_NAMES):
        return f"ps_sim_{POLICY_NAMES[int(targ)]}"
    return name


def rocprof_summary(d, workload):
    """Summarises rocprofv3 output under d (kt/ kernel trace with --stats,
    fetch/ and write/ counter runs of FETCH_SIZE and WRITE_SIZE), all made by
    this script's benchmark command. Counters are scaled by what they read
    for the calibration copy (1 GiB read + 1 GiB written). Prints a Markdown
    report ending with one JSON line that the benchmark reads back."""
    import collections
    import csv
    stats = {}
    for path in glob.glob(os.path.join(d, "kt", "*kernel_stats.csv")):
        for r in csv.DictReader(open(path)):
            stats[_kernel_short_name(r["Name"])] = (int(r["Calls"]), float(r["AverageNs"]) / 1e6,
                                                    float(r["Percentage"]))
    ctr = collections.defaultdict(lambda: collections.defaultdict(list))
    for sub in ("fetch", "write"):
        for path in glob.glob(os.path.join(d, sub, "*counter_collection.csv")):
            for r in csv.DictReader(open(path)):
                ctr[_kernel_short_name(r["Kernel_Name"])][r["Counter_Name"]].append(
                    float(r["Counter_Value"]))
    cal = ctr.get("calibration_copy_kernel", {})
    gib_kib = float(1 << 20)
    ff = gib_kib / (sum(cal["FETCH_SIZE"]) / len(cal["FETCH_SIZE"])) if cal.get("FETCH_SIZE") else None
    wf = gib_kib / (sum(cal["WRITE_SIZE"]) / len(cal["WRITE_SIZE"])) if cal.get("WRITE_SIZE") else None
    out = {"source_hash": kernel_source_hash(), "workload": workload,
           "fetch_factor": ff, "write_factor": wf, "kernels": {}}
    lines = [f"| kernel | calls | avg ms | % time | HBM read GB/launch | HBM write GB/launch | GB/s |",
             "|---|---|---|---|---|---|---|"]
    for k, (calls, avg_ms, pct) in sorted(stats.items(), key=lambda x: -x[1][2]):
        c = ctr.get(k, {})
        rd = wr = None
        if c.get("FETCH_SIZE") and ff:
            rd = sum(c["FETCH_SIZE"]) / len(c["FETCH_SIZE"]) * 1024 * ff
        if c.get("WRITE_SIZE") and wf:
            wr = sum(c["WRITE_SIZE"]) / len(c["WRITE_SIZE"]) * 1024 * wf
        tot = (rd or 0) + (wr or 0)
        out["kernels"][k] = {"calls": calls, "avg_ms": round(avg_ms, 5),
                             "hbm_read_bytes_per_launch": rd, "hbm_write_bytes_per_launch": wr,
                             "hbm_bytes_per_launch": tot if rd is not None and wr is not None else None}
        gbs = f"{tot / (avg_ms * 1e-3) / 1e9:.0f}" if avg_ms > 0 and tot else ""
        lines.append(f"| {k} | {calls} | {avg_ms:.4f} | {pct:.2f} | "
                     f"{'' if rd is None else f'{rd / 1e9:.3f}'} | "
                     f"{'' if wr is None else f'{wr / 1e9:.3f}'} | {gbs} |")
    print("\n".join(lines))
    print()
    print(f"Counter scaling from the calibration copy: FETCH_SIZE x {ff}, WRITE_SIZE x {wf}.")
    print()
    print(json.dumps(out))


def cpu_baseline(w, sizes, caps, epochs=2, workers=2):
    """The oracle on a bounded sample of the same workload: `epochs` of the E
    epochs sorted and sharded for all workers, and stats, next use and plan
    for `workers` of the N workers on those streams; each stage's time is
    scaled linearly to the full job (streams by E/epochs, per-worker stages
    by N/workers)."""
    import numpy as np
    from oracle import ref
    ref.build()
    job = ref.make_job(w.F, epochs, w.N, w.B, w.drop_last, w.seed)
    full = ref.make_job(*w.job_tuple())
    _, _, Mw = ref.stream_shape(full)
    A = int(Mw.sum())
    t0 = time.perf_counter()
    R = ref.access_streams(job)
    t1 = time.perf_counter()
    count, first = ref.access_stats_rows(job, R[:workers], 0)
    t2 = time.perf_counter()
    ref.reuse_next_rows(job, R[:workers], 0)
    t3 = time.perf_counter()
    ref.tier_plan(full, count, first, sizes, np.asarray(caps, np.int64))
    t4 = time.perf_counter()
    est = (t1 - t0) * (w.E / epochs) + (t4 - t1) * (w.N / workers)
    return {
        "value": A / est,
        "unit": "accesses/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{w.name}: {epochs} of {w.E} epochs sorted+sharded for all {w.N} workers "
                   f"({t1 - t0:.1f}s), stats {t2 - t1:.2f}s + next {t3 - t2:.2f}s + plan "
                   f"{t4 - t3:.1f}s for {workers} of {w.N} workers; scaled x{w.E // epochs} "
                   f"(streams) and x{w.N // workers} (per-worker stages) to {est:.0f}s for the "
                   f"full job; single-threaded, {os.cpu_count()} host cores present"),
    }


def buffer_algorithmic_bytes(job, M, M_w):
    """Bytes the clairvoyant-buffer replay must move given the dense layouts:
    R and next once, each sample's size once, and a hit flag per position."""
    A = int(sum(M_w))
    return {"bs_sim": 8 * A + 8 * job.F + job.N * M + 16 * job.N}


def policy_algorithmic_bytes(job, M, M_w, policy):
    """Bytes a policy simulation must move given the dense layouts: R once,
    each size once, the sources (NoPFS) and the staging windows (staging
    policies), and every consumption time."""
    A = int(sum(M_w))
    b = 4 * A + 8 * job.F + 8 * job.N * M
    if policy >= 2:
        b += 4 * A
    if policy == 3:
        b += 2 * A
    return {f"ps_sim_{POLICY_NAMES[policy]}": b}


def roofline_of(workload, kernel, alg_bytes, avg_ms):
    achieved = alg_bytes / (avg_ms * 1e-3) / 1e9
    return {"bound": "hbm", "kernel": kernel, "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": committed_traffic(workload, kernel), "algorithmic_bytes": alg_bytes,
            "avg_ms": round(avg_ms, 4)}


def time_calls(nopfs, torch, w, calls, algs, steps, warmup, stream, out):
    """Each call timed over `steps` calls with HIP events on the stream the
    library launches on; per-kernel times from the library's own events."""
    for _ in range(warmup):
        for f in calls.values():
            f()
    torch.cuda.synchronize()
    for name, f in calls.items():
        alg = algs[name]
        nopfs.profile_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            f()
        e1.record(stream)
        torch.cuda.synchronize()
        nopfs.profile_enable(False)
        ms = e0.elapsed_time(e1) / steps
        kern = {k: {"ms_per_call": t / steps, "avg_ms": t / n}
                for k, (n, t) in nopfs.profile_results().items()}
        for k, v in kern.items():
            if k in alg:
                v["alg_GBps"] = round(alg[k] / (v["avg_ms"] * 1e-3) / 1e9, 1)
        # the roofline is that of the slowest kernel carrying algorithmic bytes
        # (the bytes the call must move are attributed to the kernels that
        # move them); the slowest kernel overall is reported beside it
        slowest = max(kern, key=lambda k: kern[k]["ms_per_call"])
        own = [k for k in kern if k in alg]
        dominant = max(own, key=lambda k: kern[k]["ms_per_call"]) if own else slowest
        total_alg = sum(alg.values())
        out[name] = {
            "ms_per_call": round(ms, 4),
            "alg_bytes": total_alg,
            "alg_GBps": round(total_alg / (ms * 1e-3) / 1e9, 1),
            "slowest_kernel": slowest,
            "kernels": {k: {kk: round(vv, 4) for kk, vv in v.items()} for k, v in kern.items()},
            "roofline": (roofline_of(w.name, dominant, alg[dominant], kern[dominant]["avg_ms"])
                         if dominant in alg else {"kernel": dominant, "algorithmic_bytes": 0}),
        }
        print(f"[bench] {name}: {ms:.3f} ms/call, dominant {dominant}", file=sys.stderr,
              flush=True)
    return out


def time_schedule(nopfs, torch, w, job, M, M_w, R, tier, sizes, caps, steps, warmup, stream):
    """The per-tier prefetch queues and the staging schedule of the planned
    job (the planning step's own outputs as inputs)."""
    J = len(caps)
    d0 = int(w.staging)
    dev = R.device
    order = torch.empty((job.N, M), dtype=torch.int32, device=dev)
    qlen = torch.empty((job.N, J), dtype=torch.int64, device=dev)
    fill = torch.empty((job.N, M), dtype=torch.int32, device=dev)
    calls = {
        "prefetch_order": lambda: nopfs.prefetch_order(job, R, tier, J, order, qlen,
                                                       stream=stream),
        "staging_schedule": lambda: nopfs.staging_schedule(job, R, sizes, d0, fill, stream=stream),
    }
    pf_alg, st_alg = schedule_algorithmic_bytes(job, M, M_w)
    out = time_calls(nopfs, torch, w, calls, {"prefetch_order": pf_alg, "staging_schedule": st_alg},
                     steps, warmup, stream, {"J": J, "d0_bytes": d0})
    out["queued"] = int(qlen.sum())
    return out


def time_model(nopfs, torch, wl, w, job, M, M_w, R, tier, sizes, steps, warmup, stream):
    """Fetch sources and consumption times of the planned job under the
    performance model with the simulated cluster's parameters."""
    dev = R.device
    src = torch.empty((job.N, M), dtype=torch.int16, device=dev)
    t = torch.empty((job.N, M), dtype=torch.float64, device=dev)
    model = nopfs.make_model(**wl.LASSEN_MODEL)
    calls = {"fetch_model": lambda: nopfs.fetch_model(job, R, tier, sizes, model, src, t,
                                                      stream=stream)}
    out = time_calls(nopfs, torch, w, calls, {"fetch_model": model_algorithmic_bytes(job, M, M_w)},
                     steps, warmup, stream, {"params": dict(wl.LASSEN_MODEL)})
    out["params"]["r"] = list(out["params"]["r"])
    out["params"]["p"] = list(out["params"]["p"])
    # per worker: last consumption; over workers the slowest decides
    last = t.max(dim=1).values
    out["slowest_worker_s"] = round(float(last.max()), 3)
    out["sources"] = {"pfs": int((src == 0).sum()), "remote": int(((src >= 128) & (src < 256)).sum()),
                      "own": int((src >= 256).sum())}
    return out


def time_buffer(nopfs, torch, w, job, M, M_w, R, nxt, sizes, steps, warmup, stream):
    """The clairvoyant buffer replay of the planned job's streams with the
    staging buffer's capacity (a sequential replay per worker, so fewer
    calls are timed)."""
    d0 = int(w.staging)
    dev = R.device
    hit = torch.empty((job.N, M), dtype=torch.int8, device=dev)
    hits = torch.empty((job.N, 2), dtype=torch.int64, device=dev)
    calls = {"buffer_sim": lambda: nopfs.buffer_sim(job, R, nxt, sizes, d0, hit, hits,
                                                    stream=stream)}
    out = time_calls(nopfs, torch, w, calls, {"buffer_sim": buffer_algorithmic_bytes(job, M, M_w)},
                     max(1, min(steps, 3)), min(warmup, 1), stream, {"d0_bytes": d0})
    h = hits.cpu()
    A = int(sum(M_w))
    out["hits"] = int(h[:, 0].sum())
    out["hit_rate"] = round(int(h[:, 0].sum()) / A, 4)
    out["hit_bytes"] = int(h[:, 1].sum())
    out["reads_per_s_per_worker"] = round(A / job.N / (out["buffer_sim"]["ms_per_call"] * 1e-3), 1)
    out["buffer_sim"]["roofline"]["note"] = SEQUENTIAL_NOTE
    return out


def time_policies(nopfs, torch, wl, w, job, M, M_w, R, tier, sizes, steps, warmup, stream):
    """The four data-loading policies of the simulator on the planned job:
    its streams and placement, the fetch model's sources (the simulated
    cluster's parameters) and the staging schedule of the workload's
    staging buffer. Each policy is one sequential replay per worker."""
    dev = R.device
    d0 = int(w.staging)
    model = nopfs.make_model(**wl.LASSEN_MODEL)
    fill = torch.empty((job.N, M), dtype=torch.int32, device=dev)
    nopfs.staging_schedule(job, R, sizes, d0, fill, stream=stream)
    src, _ = nopfs.fetch_model(job, R, tier, sizes, model, stream=stream)
    t = torch.empty((job.N, M), dtype=torch.float64, device=dev)
    fin = torch.empty(job.N, dtype=torch.float64, device=dev)
    io = torch.empty((job.N, 1 + 2 * model.J), dtype=torch.float64, device=dev)
    out = {"d0_bytes": d0}
    for pol, name in enumerate(POLICY_NAMES):
        calls = {name: lambda pol=pol: nopfs.policy_sim(job, R, sizes, model, pol, src=src,
                                                        fill=fill, t=t, finish=fin, io=io,
                                                        stream=stream)}
        time_calls(nopfs, torch, w, calls,
                   {name: policy_algorithmic_bytes(job, M, M_w, pol)},
                   max(1, min(steps, 3)), min(warmup, 1), stream, out)
        f = fin.cpu()
        tot = io.sum(dim=0).cpu()
        J = model.J
        out[name]["slowest_worker_s"] = round(float(f.max()), 3)
        out[name]["mean_worker_s"] = round(float(f.mean()), 3)
        out[name]["roofline"]["note"] = SEQUENTIAL_NOTE
        out[name]["fetch_s"] = {"pfs": round(float(tot[0]), 1),
                                "remote": round(float(tot[1:1 + J].sum()), 1),
                                "own": round(float(tot[1 + J:].sum()), 1)}
    del fill, src, t
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--path", choices=["fused", "staged"], default="fused",
                    help="fused: one nopfs_plan_job call per step; staged: the four stage calls")
    ap.add_argument("--no-schedule", action="store_true",
                    help="skip timing the schedule, model, buffer and policy calls")
    ap.add_argument("--calibrate-bytes", type=int, default=1 << 30,
                    help="size of the calibration copy run after the timed steps")
    ap.add_argument("--rocprof-summary", metavar="DIR",
                    help="summarise rocprofv3 output of this benchmark (no GPU needed)")
    args = ap.parse_args()
    if args.rocprof_summary:
        rocprof_summary(args.rocprof_summary, args.workload)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py plans all N workers of a job on one GPU; it does not run on more "
              "than one GPU (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2101_08734_amd import nopfs
    from paper_2101_08734_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    job = nopfs.Job(*w.job_tuple())
    T, M, M_w = nopfs.stream_shape(job)
    sizes_h = wl.sizes(w)
    caps = [int(c) for c in wl.caps(w)]
    dev = torch.device("cuda:0")
    sizes = torch.from_numpy(sizes_h).to(dev)
    R = torch.empty((job.N, M), dtype=torch.int32, device=dev)
    count = torch.empty((job.N, job.F), dtype=torch.uint8, device=dev)
    first = torch.empty((job.N, job.F), dtype=torch.int32, device=dev)
    nxt = torch.empty((job.N, M), dtype=torch.int32, device=dev)
    tier = torch.empty((job.N, job.F), dtype=torch.int8, device=dev)
    used = torch.empty((job.N, len(caps)), dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()

    out = dict(R=R, count=count, first=first, next=nxt, tier=tier, used=used)

    def step():
        if args.path == "fused":
            nopfs.plan_job(job, sizes, caps, out, stream=stream)
            return
        nopfs.access_streams(job, R, stream=stream)
        nopfs.access_stats(job, R, count, first, stream=stream)
        nopfs.reuse_next(job, R, nxt, stream=stream)
        nopfs.tier_plan(job, count, first, sizes, caps, tier, used, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] {w.name}: warmup done", file=sys.stderr, flush=True)

    nopfs.profile_enable(True)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    nopfs.profile_enable(False)
    kernels = nopfs.profile_results()
    dev_ms = ev0.elapsed_time(ev1)
    ms_per_step = dev_ms / args.steps
    print(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step (wall {wall:.2f}s)",
          file=sys.stderr, flush=True)

    # calibration copy (known traffic) for the counter runs
    if args.calibrate_bytes > 0:
        a = torch.empty(args.calibrate_bytes, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        nopfs.calibration_copy(a, b, args.calibrate_bytes, stream=stream)
        torch.cuda.synchronize()
        del a, b

    D = int((count != 0).sum())  # distinct (worker, sample) cells read
    alg, A = algorithmic_bytes(job, M_w, D, args.path == "fused")
    per_kernel = {k: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps,
                      "avg_ms": ms / n} for k, (n, ms) in kernels.items()}
    dominant = max(per_kernel, key=lambda k: per_kernel[k]["ms_per_step"])
    dom = per_kernel[dominant]
    roofline = None
    if dominant in alg:
        roofline = roofline_of(w.name, dominant, alg[dominant], dom["avg_ms"])
    for k, v in per_kernel.items():
        if k in alg:
            v["alg_GBps"] = round(alg[k] / (v["avg_ms"] * 1e-3) / 1e9, 1)
    print("[bench] kernels: " + json.dumps(per_kernel), file=sys.stderr, flush=True)

    schedule = model = buffer = policies = None
    if not args.no_schedule:
        later_warmup = min(args.warmup, 2)
        schedule = time_schedule(nopfs, torch, w, job, M, M_w, R, tier, sizes, caps, args.steps,
                                 later_warmup, stream)
        model = time_model(nopfs, torch, wl, w, job, M, M_w, R, tier, sizes, args.steps,
                           later_warmup, stream)
        buffer = time_buffer(nopfs, torch, w, job, M, M_w, R, nxt, sizes, args.steps,
                             args.warmup, stream)
        policies = time_policies(nopfs, torch, wl, w, job, M, M_w, R, tier, sizes, args.steps,
                                 args.warmup, stream)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on a bounded sample ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, sizes_h, caps)

    line = {
        "metric": METRIC,
        "value": A / (ms_per_step * 1e-3),
        "unit": "accesses/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": w.name, "path": args.path, "F": w.F, "E": w.E, "N": w.N, "B": w.B,
                   "drop_last": w.drop_last, "seed": w.seed, "accesses": A,
                   "tier_caps_bytes": caps, "parallelism": "none (all N workers on one GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "schedule": schedule,
        "model": model,
        "buffer": buffer,
        "policies": policies,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
