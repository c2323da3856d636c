"""ctypes wrapper of the CPU oracle (``oracle/liboracle.so``).

TEST INFRASTRUCTURE: only the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this module. The product path (the
``paper_2101_08734_amd`` package) never imports it.

All arrays are numpy arrays on the host. Functions raise ``OracleError`` on a
negative return code.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "nopfs_ref.c")
# NOPFS_ORACLE_SANITIZE=1 selects a build with AddressSanitizer and
# UndefinedBehaviorSanitizer (every report aborts); the sanitizer runtimes
# must then be preloaded into the interpreter (oracle/run_sanitized_tests.sh).
SANITIZE = os.environ.get("NOPFS_ORACLE_SANITIZE") == "1"
_LIB = os.path.join(_HERE, "liboracle_san.so" if SANITIZE else "liboracle.so")

GCC_CMD = (["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra"]
           + (["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
               "-fno-sanitize-recover=all"] if SANITIZE else [])
           + ["-o", _LIB, _SRC])


class OracleError(RuntimeError):
    pass


class RefJob(ctypes.Structure):
    _fields_ = [("F", ctypes.c_int64), ("E", ctypes.c_int32),
                ("N", ctypes.c_int32), ("B", ctypes.c_int32),
                ("drop_last", ctypes.c_int32), ("seed", ctypes.c_uint64)]


class RefModel(ctypes.Structure):
    _fields_ = [("c", ctypes.c_double), ("beta", ctypes.c_double), ("b_c", ctypes.c_double),
                ("pfs_t", ctypes.c_double), ("pfs_gamma", ctypes.c_double),
                ("w0", ctypes.c_double), ("p0", ctypes.c_double),
                ("J", ctypes.c_int32), ("pad_", ctypes.c_int32),
                ("r", ctypes.c_double * 32), ("p", ctypes.c_double * 32)]


def make_model(c, beta, b_c, pfs_t, pfs_gamma, w0, p0, r, p) -> RefModel:
    """Model parameters in bytes, bytes/s; r and p per cache tier."""
    m = RefModel()
    m.c, m.beta, m.b_c = float(c), float(beta), float(b_c)
    m.pfs_t, m.pfs_gamma, m.w0, m.p0 = float(pfs_t), float(pfs_gamma), float(w0), float(p0)
    m.J = len(r)
    for j, (rj, pj) in enumerate(zip(r, p)):
        m.r[j], m.p[j] = float(rj), float(pj)
    return m


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain C, no GPU code)."""
    if force or not os.path.exists(_LIB) or \
            os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        subprocess.run(GCC_CMD, check=True)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        jp = ctypes.POINTER(RefJob)
        L.nopfs_ref_philox4x32_10.argtypes = [P, P, P]
        L.nopfs_ref_philox4x32_10.restype = None
        L.nopfs_ref_stream_shape.argtypes = [jp, P, P, P]
        L.nopfs_ref_epoch_keys.argtypes = [jp, ctypes.c_int32, P]
        L.nopfs_ref_epoch_perm.argtypes = [jp, ctypes.c_int32, P]
        L.nopfs_ref_streams_from_perms.argtypes = [jp, P, P]
        L.nopfs_ref_streams_rows.argtypes = [jp, P, ctypes.c_int64, ctypes.c_int64, P]
        L.nopfs_ref_access_streams.argtypes = [jp, P]
        L.nopfs_ref_access_stats.argtypes = [jp, P, P, P]
        L.nopfs_ref_reuse_next.argtypes = [jp, P, P]
        L.nopfs_ref_access_stats_rows.argtypes = [jp, P, ctypes.c_int64, ctypes.c_int64, P, P]
        L.nopfs_ref_reuse_next_rows.argtypes = [jp, P, ctypes.c_int64, ctypes.c_int64, P]
        L.nopfs_ref_tier_plan.argtypes = [jp, P, P, P, P, ctypes.c_int32, P, P]
        L.nopfs_ref_sample_columns.argtypes = [jp, P, ctypes.c_int64, P, P, P,
                                               P, P, P]
        L.nopfs_ref_prefetch_order.argtypes = [jp, P, P, P, ctypes.c_int32, P, P]
        L.nopfs_ref_staging_schedule.argtypes = [jp, P, P, ctypes.c_int64, P]
        L.nopfs_ref_fetch_model_rows.argtypes = [jp, P, P, P, ctypes.POINTER(RefModel),
                                                 ctypes.c_int64, ctypes.c_int64, P, P]
        L.nopfs_ref_buffer_sim.argtypes = [jp, P, P, P, ctypes.c_int64, P, P]
        L.nopfs_ref_buffer_sim_rows.argtypes = [jp, P, ctypes.c_int64, ctypes.c_int64, P, P,
                                                ctypes.c_int64, P, P]
        L.nopfs_ref_policy_sim_rows.argtypes = [jp, P, P, P, P, ctypes.POINTER(RefModel),
                                                ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
                                                P, P, P]
        for name in ("nopfs_ref_stream_shape", "nopfs_ref_epoch_keys",
                     "nopfs_ref_epoch_perm", "nopfs_ref_streams_from_perms", "nopfs_ref_streams_rows",
                     "nopfs_ref_access_streams", "nopfs_ref_access_stats",
                     "nopfs_ref_reuse_next", "nopfs_ref_tier_plan",
                     "nopfs_ref_sample_columns", "nopfs_ref_access_stats_rows",
                     "nopfs_ref_reuse_next_rows", "nopfs_ref_prefetch_order",
                     "nopfs_ref_staging_schedule", "nopfs_ref_fetch_model_rows",
                     "nopfs_ref_buffer_sim", "nopfs_ref_buffer_sim_rows",
                     "nopfs_ref_policy_sim_rows"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def make_job(F, E, N, B, drop_last=1, seed=42) -> RefJob:
    return RefJob(int(F), int(E), int(N), int(B), int(drop_last), int(seed))


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what} returned {rc}")


def philox4x32_10(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().nopfs_ref_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def stream_shape(job: RefJob):
    T = np.zeros(1, np.int64)
    Mmax = np.zeros(1, np.int64)
    Mw = np.zeros(job.N, np.int64)
    _check(lib().nopfs_ref_stream_shape(ctypes.byref(job), _ptr(T), _ptr(Mmax),
                                        _ptr(Mw)), "stream_shape")
    return int(T[0]), int(Mmax[0]), Mw


def epoch_keys(job: RefJob, e: int) -> np.ndarray:
    keys = np.empty(job.F, np.uint32)
    _check(lib().nopfs_ref_epoch_keys(ctypes.byref(job), e, _ptr(keys)),
           "epoch_keys")
    return keys


def epoch_perm(job: RefJob, e: int) -> np.ndarray:
    perm = np.empty(job.F, np.int32)
    _check(lib().nopfs_ref_epoch_perm(ctypes.byref(job), e, _ptr(perm)),
           "epoch_perm")
    return perm


def streams_from_perms(job: RefJob, perms: np.ndarray) -> np.ndarray:
    _, Mmax, _ = stream_shape(job)
    perms = np.ascontiguousarray(perms, dtype=np.int32)
    assert perms.shape == (job.E, job.F)
    R = np.empty((job.N, Mmax), np.int32)
    _check(lib().nopfs_ref_streams_from_perms(ctypes.byref(job), _ptr(perms),
                                              _ptr(R)), "streams_from_perms")
    return R


def streams_rows(job: RefJob, perms: np.ndarray, i0: int, i1: int) -> np.ndarray:
    """Rows [i0, i1) of streams_from_perms(job, perms), sharded row by row."""
    _, Mmax, _ = stream_shape(job)
    perms = np.ascontiguousarray(perms, dtype=np.int32)
    assert perms.shape == (job.E, job.F)
    R = np.empty((i1 - i0, Mmax), np.int32)
    _check(lib().nopfs_ref_streams_rows(ctypes.byref(job), _ptr(perms), int(i0), int(i1),
                                        _ptr(R)), "streams_rows")
    return R


def access_streams(job: RefJob) -> np.ndarray:
    _, Mmax, _ = stream_shape(job)
    R = np.empty((job.N, Mmax), np.int32)
    _check(lib().nopfs_ref_access_streams(ctypes.byref(job), _ptr(R)),
           "access_streams")
    return R


def access_stats(job: RefJob, R: np.ndarray):
    R = np.ascontiguousarray(R, dtype=np.int32)
    count = np.empty((job.N, job.F), np.uint8)
    first = np.empty((job.N, job.F), np.int32)
    _check(lib().nopfs_ref_access_stats(ctypes.byref(job), _ptr(R),
                                        _ptr(count), _ptr(first)),
           "access_stats")
    return count, first


def access_stats_rows(job: RefJob, R_rows: np.ndarray, i0: int):
    """Stats of workers [i0, i0 + len(R_rows)) only."""
    R_rows = np.ascontiguousarray(R_rows, dtype=np.int32)
    n = R_rows.shape[0]
    count = np.empty((n, job.F), np.uint8)
    first = np.empty((n, job.F), np.int32)
    _check(lib().nopfs_ref_access_stats_rows(ctypes.byref(job), _ptr(R_rows), i0, i0 + n,
                                             _ptr(count), _ptr(first)), "access_stats_rows")
    return count, first


def reuse_next_rows(job: RefJob, R_rows: np.ndarray, i0: int) -> np.ndarray:
    R_rows = np.ascontiguousarray(R_rows, dtype=np.int32)
    nxt = np.empty_like(R_rows)
    _check(lib().nopfs_ref_reuse_next_rows(ctypes.byref(job), _ptr(R_rows), i0,
                                           i0 + R_rows.shape[0], _ptr(nxt)), "reuse_next_rows")
    return nxt


def reuse_next(job: RefJob, R: np.ndarray) -> np.ndarray:
    R = np.ascontiguousarray(R, dtype=np.int32)
    nxt = np.empty_like(R)
    _check(lib().nopfs_ref_reuse_next(ctypes.byref(job), _ptr(R), _ptr(nxt)),
           "reuse_next")
    return nxt


def tier_plan(job: RefJob, count, first, sizes, caps):
    count = np.ascontiguousarray(count, dtype=np.uint8)
    first = np.ascontiguousarray(first, dtype=np.int32)
    sizes = np.ascontiguousarray(sizes, dtype=np.int64)
    caps = np.ascontiguousarray(caps, dtype=np.int64)
    rows = count.shape[0]
    sub = RefJob(job.F, job.E, rows, job.B, job.drop_last, job.seed)
    tier = np.empty((rows, job.F), np.int8)
    used = np.empty((rows, len(caps)), np.int64)
    _check(lib().nopfs_ref_tier_plan(ctypes.byref(sub), _ptr(count),
                                     _ptr(first), _ptr(sizes), _ptr(caps),
                                     len(caps), _ptr(tier), _ptr(used)),
           "tier_plan")
    return tier, used


def prefetch_order(job: RefJob, R, first, tier, J):
    """order[N][M_max] (tier 0's queue, tier 1's, ..., then -1), qlen[N][J]."""
    R = np.ascontiguousarray(R, dtype=np.int32)
    first = np.ascontiguousarray(first, dtype=np.int32)
    tier = np.ascontiguousarray(tier, dtype=np.int8)
    order = np.empty_like(R)
    qlen = np.empty((job.N, J), np.int64)
    _check(lib().nopfs_ref_prefetch_order(ctypes.byref(job), _ptr(R), _ptr(first), _ptr(tier),
                                          int(J), _ptr(order), _ptr(qlen)), "prefetch_order")
    return order, qlen


def staging_schedule(job: RefJob, R, sizes, d0):
    """fill[N][M_max]: first position from which the sample at h may be staged."""
    R = np.ascontiguousarray(R, dtype=np.int32)
    sizes = np.ascontiguousarray(sizes, dtype=np.int64)
    fill = np.empty_like(R)
    _check(lib().nopfs_ref_staging_schedule(ctypes.byref(job), _ptr(R), _ptr(sizes), int(d0),
                                            _ptr(fill)), "staging_schedule")
    return fill


def fetch_model(job: RefJob, R, tier, sizes, model: RefModel, rows=None):
    """(src, t) for the given workers (default all): src int16 fetch source
    (0 PFS, 128 + j remote tier j, 256 + j own tier j, -1 padding), t float64
    consumption time in seconds (-1 in padding). R holds those workers' rows;
    tier is the placement of all N workers."""
    _, M, _ = stream_shape(job)
    i0, i1 = (0, job.N) if rows is None else rows
    R = np.ascontiguousarray(R, dtype=np.int32)
    tier = np.ascontiguousarray(tier, dtype=np.int8)
    sizes = np.ascontiguousarray(sizes, dtype=np.int64)
    assert R.shape == (i1 - i0, M) and tier.shape == (job.N, job.F)
    src = np.empty((i1 - i0, M), np.int16)
    t = np.empty((i1 - i0, M), np.float64)
    _check(lib().nopfs_ref_fetch_model_rows(ctypes.byref(job), _ptr(R), _ptr(tier), _ptr(sizes),
                                            ctypes.byref(model), int(i0), int(i1), _ptr(src),
                                            _ptr(t)), "fetch_model")
    return src, t


def buffer_sim(job: RefJob, R, nxt, sizes, d0, rows=None):
    """(hit [N][M_max] int8: 1 hit, 0 miss, -1 padding; hits [N][2]: hit count
    and hit bytes) of a clairvoyant buffer of d0 bytes per worker. With rows =
    (i0, i1), R and nxt hold only those workers' rows and so do the results."""
    R = np.ascontiguousarray(R, dtype=np.int32)
    nxt = np.ascontiguousarray(nxt, dtype=np.int32)
    sizes = np.ascontiguousarray(sizes, dtype=np.int64)
    i0, i1 = (0, job.N) if rows is None else rows
    hit = np.empty(R.shape, np.int8)
    hits = np.empty((i1 - i0, 2), np.int64)
    if R.shape[0] != i1 - i0 or nxt.shape != R.shape:
        raise ValueError("R and nxt must hold the rows asked for")
    _check(lib().nopfs_ref_buffer_sim_rows(ctypes.byref(job), _ptr(R), i0, i1, _ptr(nxt),
                                           _ptr(sizes), int(d0), _ptr(hit), _ptr(hits)),
           "buffer_sim")
    return hit, hits


PERFECT, NAIVE, STAGING, NOPFS = 0, 1, 2, 3


def policy_sim(job: RefJob, R, sizes, model: RefModel, policy, src=None, fill=None, rows=None):
    """(t, finish, io) of a policy (PERFECT, NAIVE, STAGING, NOPFS) for the
    given workers (default all): t float64 [rows][M_max] consumption times
    (-1 padding), finish float64 [rows], io float64 [rows][1 + 2J] fetch time
    per source class. R, src and fill hold those workers' rows."""
    _, M, _ = stream_shape(job)
    i0, i1 = (0, job.N) if rows is None else rows
    R = np.ascontiguousarray(R, dtype=np.int32)
    sizes = np.ascontiguousarray(sizes, dtype=np.int64)
    if R.shape != (i1 - i0, M):
        raise ValueError("R must hold the rows asked for")
    if src is not None:
        src = np.ascontiguousarray(src, dtype=np.int16)
        assert src.shape == R.shape
    if fill is not None:
        fill = np.ascontiguousarray(fill, dtype=np.int32)
        assert fill.shape == R.shape
    t = np.empty((i1 - i0, M), np.float64)
    finish = np.empty(i1 - i0, np.float64)
    io = np.empty((i1 - i0, 1 + 2 * model.J), np.float64)
    _check(lib().nopfs_ref_policy_sim_rows(
        ctypes.byref(job), _ptr(R), _ptr(sizes), None if src is None else _ptr(src),
        None if fill is None else _ptr(fill), ctypes.byref(model), int(policy), i0, i1, _ptr(t),
        _ptr(finish), _ptr(io)), "policy_sim")
    return t, finish, io


def sample_columns(job: RefJob, samples):
    samples = np.ascontiguousarray(samples, dtype=np.int32)
    S = len(samples)
    E, N = job.E, job.N
    pos = np.empty((E, S), np.int64)
    occ_worker = np.empty((E, S), np.int32)
    occ_f = np.empty((E, S), np.int32)
    occ_next = np.empty((E, S), np.int32)
    col_count = np.empty((N, S), np.uint8)
    col_first = np.empty((N, S), np.int32)
    _check(lib().nopfs_ref_sample_columns(
        ctypes.byref(job), _ptr(samples), S, _ptr(pos), _ptr(occ_worker),
        _ptr(occ_f), _ptr(occ_next), _ptr(col_count), _ptr(col_first)),
        "sample_columns")
    return dict(pos=pos, occ_worker=occ_worker, occ_f=occ_f,
                occ_next=occ_next, col_count=col_count, col_first=col_first)


def full_pipeline(job: RefJob, sizes, caps):
    """All four stages, in order, on the host."""
    R = access_streams(job)
    count, first = access_stats(job, R)
    nxt = reuse_next(job, R)
    tier, used = tier_plan(job, count, first, sizes, caps)
    return dict(R=R, count=count, first=first, next=nxt, tier=tier, used=used)
