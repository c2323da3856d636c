"""The oracle's results for a full-size job, computed in a host thread pool and
compared with device outputs in chunks of worker rows.

Test infrastructure only. Every value here comes from the oracle's own C
functions (``oracle/ref.py``), called from several host threads: ctypes
releases the GIL during a call and the oracle keeps no state between calls.
Nothing is taken from the device path except the outputs being checked.

 - permutations: each epoch's (key, id) sort (the shuffle of section 2) in
   its own task;
 - per chunk of worker rows: the oracle's strided shard of those rows (the
   batch partition of section 4), then their counts and first reads
   (section 3.1), next uses (section 3) and tier plan (section 5.1).
"""
from __future__ import annotations

import os
import threading
from concurrent.futures import ThreadPoolExecutor

import numpy as np

OUTPUTS = ("R", "count", "first", "next", "tier", "used")


def pool_threads() -> int:
    """Worker threads: the host's cores, at most 16 (the CPU share of a
    one-GPU host)."""
    return max(1, min(16, os.cpu_count() or 1))


def oracle_perms(ref, rj, threads=None):
    """perms [E][F]: every epoch's permutation, one task per epoch."""
    threads = threads or pool_threads()
    perms = np.empty((rj.E, rj.F), np.int32)

    def one(e):
        perms[e] = ref.epoch_perm(rj, e)

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(one, range(rj.E)))
    return perms


def oracle_rows(ref, rj, perms, sizes, caps, i0, i1):
    """R, count, first, next, tier, used of workers [i0, i1) from the
    oracle's permutations."""
    rows = ref.streams_rows(rj, perms, i0, i1)
    count, first = ref.access_stats_rows(rj, rows, i0)
    nxt = ref.reuse_next_rows(rj, rows, i0)
    tier, used = ref.tier_plan(rj, count, first, sizes, caps)
    return {"R": rows, "count": count, "first": first, "next": nxt, "tier": tier, "used": used}


def compare_all_rows(ref, rj, sizes, caps, device_outputs, chunk=4, threads=None, perms=None,
                     log=None, rows=None):
    """Compares every element of every output in `device_outputs` (a dict
    name -> {output name: torch tensor on the device}) with the oracle for
    the workers in `rows` = (i0, i1) (default all), in chunks of `chunk`
    worker rows processed by a thread pool. Returns a list of mismatch
    descriptions (empty when everything is equal)."""
    r0, r1 = (0, rj.N) if rows is None else rows
    threads = threads or pool_threads()
    if perms is None:
        perms = oracle_perms(ref, rj, threads)
    sizes = np.ascontiguousarray(sizes, np.int64)
    caps = np.ascontiguousarray(caps, np.int64)
    mism = []
    lock = threading.Lock()
    done = [0]

    def task(i0):
        i1 = min(i0 + chunk, r1)
        exp = oracle_rows(ref, rj, perms, sizes, caps, i0, i1)
        for path, outs in device_outputs.items():
            for name in OUTPUTS:
                got = outs[name][i0:i1].cpu().numpy()
                if not np.array_equal(got, exp[name]):
                    bad = np.argwhere(got != exp[name])
                    with lock:
                        mism.append(f"{path}: {name} rows {i0}..{i1 - 1}: {len(bad)} cells differ, "
                                    f"first at {tuple(int(x) + (i0 if k == 0 else 0) for k, x in enumerate(bad[0]))}")
        with lock:
            done[0] += i1 - i0
            if log and (done[0] % max(chunk, (r1 - r0) // 8) < chunk or done[0] == r1 - r0):
                log(f"{done[0]}/{r1 - r0} workers compared")

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(task, range(r0, r1, chunk)))
    return mism
