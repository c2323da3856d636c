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


# The planning path's stages and the kernels each one launches (library
# launch names). The counting and next-use passes share one partition of R in
# the fused call; its kernels are counted with the counting stage.
STAGES = {
    "streams": ("stream_count", "stream_offsets", "stream_scan", "stream_scatter", "stream_split",
                "stream_sort", "stream_pad"),
    "stats": ("seg_partition", "offsets_transpose", "stats_tile", "fill_stats_empty"),
    "next": ("next_tile", "next_unpartition", "pad_rows"),
    "plan": ("plan_classes", "plan_binsum", "plan_hist", "plan_cut", "plan_btier", "plan_write",
             "plan_resolve", "plan_exact", "fill_u64", "fill_i32"),
}


def stage_bytes(job, M_w):
    """Algorithmic bytes of each stage per step for the C ABI's dense layouts
    (A reads, N*F cells): streams write R (4A; the key/id exchange allowance 16*E*F is
    reported beside it), stats read R and write count + first (4A + 5NF),
    next reads R and writes next (8A), the plan reads count, first and sizes
    and writes tier (6NF + 8F)."""
    A = int(sum(M_w))
    NF = job.N * job.F
    return {"streams": 4 * A, "stats": 4 * A + 5 * NF, "next": 8 * A,
            "plan": 6 * NF + 8 * job.F}, A, 16 * job.E * job.F


def kernel_bytes(job, M_w):
    """Algorithmic bytes per launch of the kernel that carries each stage's
    output: the stage's bytes (stage_bytes) attributed to its final kernel."""
    sb, A, _ = stage_bytes(job, M_w)
    return {"stream_sort": sb["streams"], "stats_tile": sb["stats"],
            "next_unpartition": sb["next"], "plan_write": sb["plan"]}


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
    staging = {"seg_partition": 4 * A, "st_gather": 8 * job.F, "st_fill": 4 * NM}
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
SEQUENTIAL_NOTE = ("sequential per worker (each read depends on every earlier one), one "
                   "workgroup per worker whose waves split the chains: bound by instruction "
                   "issue and latency on the chain, not by HBM; frac is the HBM fraction for "
                   "reference")


def _kernel_short_name(full):
    """'ns::(anonymous namespace)::plan_hist<true>(args...)' -> 'plan_hist';
    the policy kernels keep their policy: 'ps_sim<1>(...)' -> 'ps_sim_naive',
    'ps_staged<2>(...)' -> 'ps_sim_staging' (the names the library launches them by), and
    the staging schedule's 8-byte-size unpartition its launch name 'st_unpart8'."""
    import re
    m = re.findall(r"(\w+)(?:<([^>()]*)>)?\(", full)
    if not m:
        return full
    name, targ = m[-1]
    if name in ("ps_sim", "ps_staged") and targ.strip().isdigit() and int(targ) < len(POLICY_NAMES):
        return f"ps_sim_{POLICY_NAMES[int(targ)]}"
    if name == "st_unpart" and targ.strip() == "true":  # the 8-byte-size form, launched as such
        return "st_unpart8"
    return name


# rocprofv3 counter passes of the profile summary (one run each; every pass
# stays within the per-block counter limits of one run).
PMC_PASSES = {
    "rd": ["TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum", "TCC_EA0_RDREQ_128B_sum",
           "TCC_EA0_RDREQ_sum"],
    "wr": ["TCC_EA0_WRREQ_sum", "TCC_EA0_WRREQ_64B_sum"],
    "sq": ["VALUBusy", "LDSBankConflict", "OccupancyPercent", "LdsUtil", "SQ_INSTS_VALU",
           "SQ_INSTS_LDS", "SQ_WAVES"],
}


def rocprof_summary(d, workload):
    """Summarises rocprofv3 output under d: kt/ (kernel trace with --stats),
    rd/ and wr/ (L2-to-memory read and write requests by size), sq/ (VALU
    busy, LDS bank conflicts, LDS utilisation, occupancy, instruction and
    wave counts), all made by this script's benchmark command.

    Read bytes are counted per request size, 32 x (32 B requests) + 64 x
    (64 B) + 128 x (128 B); write bytes 32 x (32 B) + 64 x (64 B). Each is
    then scaled by what the same sum reads for the calibration copy (1 GiB
    read + 1 GiB written), and the factors are printed. Prints a Markdown
    report ending with one JSON line that the benchmark reads back."""
    import collections
    import csv
    stats = {}
    for path in glob.glob(os.path.join(d, "kt", "*kernel_stats.csv")):
        for r in csv.DictReader(open(path)):
            stats[_kernel_short_name(r["Name"])] = (int(r["Calls"]), float(r["AverageNs"]) / 1e6,
                                                    float(r["Percentage"]))
    ctr = collections.defaultdict(lambda: collections.defaultdict(list))
    for sub in PMC_PASSES:
        for path in glob.glob(os.path.join(d, sub, "*counter_collection.csv")):
            for r in csv.DictReader(open(path)):
                ctr[_kernel_short_name(r["Kernel_Name"])][r["Counter_Name"]].append(
                    float(r["Counter_Value"]))

    def mean(c, name):
        v = c.get(name)
        return sum(v) / len(v) if v else None

    def raw_read(c):
        n32, n64, n128, n = (mean(c, k) for k in PMC_PASSES["rd"])
        if None in (n32, n64, n128, n):
            return None, None
        return 32 * n32 + 64 * n64 + 128 * n128, n - n32 - n64 - n128

    def raw_write(c):
        n, n64 = (mean(c, k) for k in PMC_PASSES["wr"])
        if None in (n, n64):
            return None
        return 32 * (n - n64) + 64 * n64

    cal = ctr.get("calibration_copy_kernel", {})
    cr, _ = raw_read(cal)
    cw = raw_write(cal)
    gib = float(1 << 30)
    rf = gib / cr if cr else None
    wf = gib / cw if cw else None
    out = {"source_hash": kernel_source_hash(), "workload": workload,
           "read_factor": rf, "write_factor": wf, "kernels": {}}
    lines = ["| kernel | calls | avg ms | % time | HBM read GB/launch | HBM write GB/launch | GB/s "
             "| VALU busy % | LDS bank conflict % | LDS util % | occupancy % | VALU inst/wave "
             "| LDS inst/wave |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    fmt = lambda v, f: "" if v is None else format(v, f)  # noqa: E731
    for k, (calls, avg_ms, pct) in sorted(stats.items(), key=lambda x: -x[1][2]):
        c = ctr.get(k, {})
        r, other = raw_read(c)
        wr = raw_write(c)
        rd = r * rf if r is not None and rf else None
        wr = wr * wf if wr is not None and wf else None
        tot = (rd or 0) + (wr or 0)
        waves = mean(c, "SQ_WAVES")
        sq = {"valu_busy_pct": mean(c, "VALUBusy"), "lds_bank_conflict_pct": mean(c, "LDSBankConflict"),
              "lds_util_pct": mean(c, "LdsUtil"), "occupancy_pct": mean(c, "OccupancyPercent"),
              "valu_insts_per_wave": (mean(c, "SQ_INSTS_VALU") / waves) if waves else None,
              "lds_insts_per_wave": (mean(c, "SQ_INSTS_LDS") / waves) if waves else None,
              "waves": waves}
        out["kernels"][k] = {"calls": calls, "avg_ms": round(avg_ms, 5),
                             "hbm_read_bytes_per_launch": rd, "hbm_write_bytes_per_launch": wr,
                             "hbm_bytes_per_launch": tot if rd is not None and wr is not None else None,
                             "read_requests_of_other_sizes": other, **sq}
        gbs = f"{tot / (avg_ms * 1e-3) / 1e9:.0f}" if avg_ms > 0 and tot else ""
        lines.append(f"| {k} | {calls} | {avg_ms:.4f} | {pct:.2f} | {fmt(rd and rd / 1e9, '.3f')} | "
                     f"{fmt(wr and wr / 1e9, '.3f')} | {gbs} | {fmt(sq['valu_busy_pct'], '.1f')} | "
                     f"{fmt(sq['lds_bank_conflict_pct'], '.2f')} | {fmt(sq['lds_util_pct'], '.1f')} | "
                     f"{fmt(sq['occupancy_pct'], '.1f')} | {fmt(sq['valu_insts_per_wave'], '.0f')} | "
                     f"{fmt(sq['lds_insts_per_wave'], '.0f')} |")
    print("\n".join(lines))
    print()
    print(f"Counter scaling from the calibration copy (1 GiB read, 1 GiB written): read bytes x {rf}, "
          f"write bytes x {wf}.")
    print()
    print(json.dumps(out))


def cpu_model():
    """The host CPU's model name: lscpu's "Model name", else the first
    "model name" of /proc/cpuinfo."""
    import subprocess
    try:
        r = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10)
        for line in r.stdout.splitlines():
            if line.strip().startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, sizes, caps, epochs=2, workers=2):
    """The oracle, single-threaded, on a bounded sample of the same workload:
     - `epochs` of the E epochs generated, sorted and sharded for all N
       workers, scaled by E/epochs;
     - for `workers` of the N workers, rows of the full length (E epochs: the
       sampled epochs' streams repeated, so each row has the full job's reads
       and the same access pattern), counted, linked (next use) and planned,
       scaled by N/workers."""
    import numpy as np
    from oracle import ref
    ref.build()
    job = ref.make_job(w.F, epochs, w.N, w.B, w.drop_last, w.seed)
    full = ref.make_job(*w.job_tuple())
    _, M_full, Mw = ref.stream_shape(full)
    _, _, Mw_s = ref.stream_shape(job)
    A = int(Mw.sum())
    t0 = time.perf_counter()
    R = ref.access_streams(job)
    t1 = time.perf_counter()
    rows = np.full((workers, M_full), -1, np.int32)
    for i in range(workers):
        L = int(Mw_s[i]) // epochs
        for e in range(w.E):
            rows[i, e * L:(e + 1) * L] = R[i, (e % epochs) * L:(e % epochs + 1) * L]
    del R
    t2 = time.perf_counter()
    count, first = ref.access_stats_rows(full, rows, 0)
    t3 = time.perf_counter()
    ref.reuse_next_rows(full, rows, 0)
    t4 = time.perf_counter()
    ref.tier_plan(full, count, first, sizes, np.asarray(caps, np.int64))
    t5 = time.perf_counter()
    scale_e, scale_n = w.E / epochs, w.N / workers
    est = (t1 - t0) * scale_e + (t5 - t2) * scale_n
    return {
        "value": A / est,
        "unit": "accesses/s",
        "cores": 1,
        "kind": "oracle",
        "cpu": cpu_model(),
        "sample": (f"{w.name}: streams of {epochs} of {w.E} epochs generated, sorted and sharded "
                   f"for all {w.N} workers ({t1 - t0:.1f}s, x{scale_e:g}); for {workers} of "
                   f"{w.N} workers, full-length rows ({w.E} epochs, the sampled epochs' streams "
                   f"repeated): stats {t3 - t2:.2f}s + next {t4 - t3:.2f}s + plan {t5 - t4:.1f}s "
                   f"(x{scale_n:g}); {est:.0f}s estimated for the full job; single-threaded "
                   f"(1 of {os.cpu_count()} host cores), {cpu_model()}"),
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


def copy_ceiling(nopfs, torch, nbytes, stream, calls=10):
    """A plain device copy of nbytes (read nbytes, write nbytes) with the
    library's calibration kernel, timed with HIP events on `stream`: the
    measured HBM ceiling of a streaming kernel on this part. The same kernel
    calibrates the byte counters of the rocprofv3 runs."""
    dev = torch.device("cuda:0")
    a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    for _ in range(3):
        nopfs.calibration_copy(a, b, nbytes, stream=stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(calls):
        nopfs.calibration_copy(a, b, nbytes, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / calls
    del a, b
    gbs = 2 * nbytes / (ms * 1e-3) / 1e9
    return {"bytes_read": nbytes, "bytes_written": nbytes, "ms": round(ms, 4),
            "GBps": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4)}


def measure(nopfs, torch, wl, w, path, steps, warmup, stream, keep=False):
    """One workload: `warmup` untimed steps, then `steps` timed steps of the
    whole planning path (fused: one nopfs_plan_job call; staged: the four
    stage calls), device time from HIP events on `stream`, per-kernel times
    from the library's own events. Returns the result dict (and the outputs
    when keep)."""
    job = nopfs.Job(*w.job_tuple())
    T, M, M_w = nopfs.stream_shape(job)
    caps = [int(c) for c in wl.caps(w)]
    dev = torch.device("cuda:0")
    sizes = torch.from_numpy(wl.sizes(w)).to(dev)
    out = dict(R=torch.empty((job.N, M), dtype=torch.int32, device=dev),
               count=torch.empty((job.N, job.F), dtype=torch.uint8, device=dev),
               first=torch.empty((job.N, job.F), dtype=torch.int32, device=dev),
               next=torch.empty((job.N, M), dtype=torch.int32, device=dev),
               tier=torch.empty((job.N, job.F), dtype=torch.int8, device=dev),
               used=torch.empty((job.N, len(caps)), dtype=torch.int64, device=dev))

    def step():
        if path == "fused":
            nopfs.plan_job(job, sizes, caps, out, stream=stream)
            return
        nopfs.access_streams(job, out["R"], stream=stream)
        nopfs.access_stats(job, out["R"], out["count"], out["first"], stream=stream)
        nopfs.reuse_next(job, out["R"], out["next"], stream=stream)
        nopfs.tier_plan(job, out["count"], out["first"], sizes, caps, out["tier"], out["used"],
                        stream=stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    nopfs.profile_enable(True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    nopfs.profile_enable(False)
    kernels = nopfs.profile_results()
    ms_per_step = ev0.elapsed_time(ev1) / steps
    print(f"[bench] {w.name} ({path}): {steps} steps, {ms_per_step:.3f} ms/step "
          f"(wall {wall:.2f}s)", file=sys.stderr, flush=True)

    sb, A, exch = stage_bytes(job, M_w)
    kb = kernel_bytes(job, M_w)
    per_kernel = {k: {"launches_per_step": n / steps, "ms_per_step": ms / steps, "avg_ms": ms / n}
                  for k, (n, ms) in kernels.items()}
    for k, v in per_kernel.items():
        if k in kb:
            v["alg_GBps"] = round(kb[k] / (v["avg_ms"] * 1e-3) / 1e9, 1)
    stages = {}
    for st, names in STAGES.items():
        ms = sum(per_kernel[k]["ms_per_step"] for k in names if k in per_kernel)
        gbs = sb[st] / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
        stages[st] = {"ms_per_step": round(ms, 4), "alg_bytes": sb[st], "alg_GBps": round(gbs, 1),
                      "frac": round(gbs / HBM_PEAK_GBS, 4),
                      "kernels": [k for k in names if k in per_kernel]}
        if st == "streams" and ms > 0:
            b = sb[st] + exch
            stages[st]["alg_bytes_with_exchange"] = b
            stages[st]["frac_with_exchange"] = round(b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
    # the roofline is that of the slowest kernel carrying a stage's bytes; the
    # slowest kernel overall is named beside it
    slowest = max(per_kernel, key=lambda k: per_kernel[k]["ms_per_step"])
    dominant = max((k for k in per_kernel if k in kb), key=lambda k: per_kernel[k]["ms_per_step"])
    roofline = roofline_of(w.name, dominant, kb[dominant], per_kernel[dominant]["avg_ms"])
    roofline["slowest_kernel"] = slowest
    res = {
        "value": A / (ms_per_step * 1e-3),
        "unit": "accesses/s",
        "ms_per_step": round(ms_per_step, 4),
        "config": {"workload": w.name, "path": path, "F": w.F, "E": w.E, "N": w.N, "B": w.B,
                   "drop_last": w.drop_last, "seed": w.seed, "accesses": A,
                   "tier_caps_bytes": caps},
        "roofline": roofline,
        "stages": stages,
        "kernels": {k: {kk: round(vv, 4) for kk, vv in v.items()} for k, v in per_kernel.items()},
    }
    if path == "fused":
        # the read-cell list the counting pass writes for the tier plan (4 B
        # per distinct (worker, sample) cell read): the implementation's own
        # scratch traffic, reported beside the stage bytes, not in them
        D = int((out["count"] != 0).sum())
        res["read_cells"] = D
        res["read_cell_list_bytes"] = 4 * D
    if keep:
        return res, job, M, M_w, sizes, caps, out
    del out, sizes
    torch.cuda.empty_cache()
    return res


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
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other full-size workloads (reported under \"configs\")")
    ap.add_argument("--calibrate-bytes", type=int, default=1 << 30,
                    help="bytes read (and written) by the copy-ceiling / calibration kernel")
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

    stream = torch.cuda.current_stream()
    w = wl.WORKLOADS[args.workload]
    res, job, M, M_w, sizes, caps, out = measure(nopfs, torch, wl, w, args.path, args.steps,
                                                 args.warmup, stream, keep=True)
    R, nxt, tier = out["R"], out["next"], out["tier"]
    del out["count"], out["first"]
    torch.cuda.empty_cache()

    ceiling = None
    if args.calibrate_bytes > 0:
        ceiling = copy_ceiling(nopfs, torch, args.calibrate_bytes, stream)
        print(f"[bench] copy ceiling {ceiling['GBps']} GB/s", file=sys.stderr, flush=True)

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
    del out, R, nxt, tier, sizes
    torch.cuda.empty_cache()

    configs = None
    if not args.no_configs:
        configs = {}
        for name in wl.ORDER:
            if name in (w.name, "small"):
                continue
            configs[name] = measure(nopfs, torch, wl, wl.WORKLOADS[name], args.path,
                                    max(args.steps, 20), args.warmup, stream)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on a bounded sample ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, wl.sizes(w), caps)

    line = {
        "metric": METRIC,
        "value": res["value"],
        "unit": "accesses/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": dict(res["config"], parallelism="none (all N workers on one GPU)"),
        "roofline": res["roofline"],
        "cpu_baseline": cpu,
        "stages": res["stages"],
        "read_cells": res.get("read_cells"),
        "read_cell_list_bytes": res.get("read_cell_list_bytes"),
        "copy_ceiling": ceiling,
        "kernels": res["kernels"],
        "configs": configs,
        "schedule": schedule,
        "model": model,
        "buffer": buffer,
        "policies": policies,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
