"""Python binding of libnopfs.so (argument marshalling only).

Every computation runs in the library's HIP kernels; this module only turns
torch tensors (device memory) and torch's current stream into the C ABI's
pointers. It raises ``NopfsError`` for a non-zero status and ``RuntimeError``
if the compiled library is missing: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch  # loads the HIP runtime before the library does

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnopfs.so")

NOPFS_OK, NOPFS_EINVAL, NOPFS_ERANGE, NOPFS_ENOMEM, NOPFS_EDEVICE = 0, -1, -2, -3, -4


class NopfsError(RuntimeError):
    def __init__(self, code: int, what: str, detail: str):
        super().__init__(f"{what}: status {code} ({detail})")
        self.code = code


class _Job(ctypes.Structure):
    _fields_ = [("F", ctypes.c_int64), ("E", ctypes.c_int32),
                ("N", ctypes.c_int32), ("B", ctypes.c_int32),
                ("drop_last", ctypes.c_int32), ("seed", ctypes.c_uint64)]


@dataclass(frozen=True)
class Job:
    """A training job as the paper states it: F samples, E epochs, N workers,
    per-worker batch B, drop_last, shuffle seed."""
    F: int
    E: int
    N: int
    B: int
    drop_last: int = 1
    seed: int = 42

    def c(self) -> _Job:
        return _Job(int(self.F), int(self.E), int(self.N), int(self.B),
                    int(self.drop_last), int(self.seed) & ((1 << 64) - 1))

    def epochs(self, e_begin: int, e_end: int) -> "Job":
        """The shape of epochs [e_begin, e_end) of this job: what
        access_streams_range writes, and what the stats, next-use and plan
        calls take for those epochs' streams. (Its own access_streams would
        draw epochs 0.., not e_begin..: use access_streams_range.)"""
        return Job(self.F, int(e_end) - int(e_begin), self.N, self.B, self.drop_last, self.seed)


class Model(ctypes.Structure):
    """Parameters of the performance model (nopfs_model): bytes, bytes/s,
    seconds; r and p per cache tier."""
    _fields_ = [("c", ctypes.c_double), ("beta", ctypes.c_double), ("b_c", ctypes.c_double),
                ("pfs_t", ctypes.c_double), ("pfs_gamma", ctypes.c_double),
                ("w0", ctypes.c_double), ("p0", ctypes.c_double),
                ("J", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("r", ctypes.c_double * 32), ("p", ctypes.c_double * 32)]


def make_model(c, beta, b_c, pfs_t, pfs_gamma, w0, p0, r, p) -> Model:
    m = Model()
    m.c, m.beta, m.b_c = float(c), float(beta), float(b_c)
    m.pfs_t, m.pfs_gamma, m.w0, m.p0 = float(pfs_t), float(pfs_gamma), float(w0), float(p0)
    m.J = len(r)
    for j, (rj, pj) in enumerate(zip(list(r)[:32], list(p)[:32])):
        m.r[j], m.p[j] = float(rj), float(pj)
    return m


_lib = None


def lib() -> ctypes.CDLL:
    """Loads the compiled library (fails loudly if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python paper_2101_08734_amd/build.py` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        jp = ctypes.POINTER(_Job)
        sig = {
            "nopfs_stream_shape": [jp, P, P, P],
            "nopfs_access_streams": [jp, P, P],
            "nopfs_access_stats": [jp, P, P, P, P],
            "nopfs_reuse_next": [jp, P, P, P],
            "nopfs_tier_plan": [jp, P, P, P, P, I32, P, P, P],
            "nopfs_plan_job": [jp, P, P, I32, P, P, P, P, P, P, P],
            "nopfs_plan_job_noalloc": [jp, P, P, I32, P, P, P, P, P, P, P],
            "nopfs_prefetch_order": [jp, P, P, I32, P, P, P],
            "nopfs_staging_schedule": [jp, P, P, I64, P, P],
            "nopfs_fetch_model": [jp, P, P, P, ctypes.POINTER(Model), P, P, P],
            "nopfs_buffer_sim": [jp, P, P, P, I64, P, P, P],
            "nopfs_access_streams_range": [jp, ctypes.c_int32, ctypes.c_int32, P, P],
            "nopfs_policy_sim": [jp, P, P, P, P, ctypes.POINTER(Model), ctypes.c_int32, P, P, P, P],
            "nopfs_profile_enable": [ctypes.c_int],
            "nopfs_profile_query": [ctypes.c_int, ctypes.POINTER(ctypes.c_char_p),
                                    ctypes.POINTER(I64), ctypes.POINTER(ctypes.c_double)],
            "nopfs_calibration_copy": [P, P, I64, P],
            "nopfs_scratch_release": [P],
            "nopfs_debug_set": [ctypes.c_int, I64],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.nopfs_strerror.argtypes = [ctypes.c_int]
        L.nopfs_strerror.restype = ctypes.c_char_p
        L.nopfs_last_error.argtypes = []
        L.nopfs_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


EXPORTED = ("nopfs_stream_shape", "nopfs_access_streams", "nopfs_access_streams_range",
            "nopfs_access_stats",
            "nopfs_reuse_next", "nopfs_tier_plan", "nopfs_plan_job", "nopfs_plan_job_noalloc",
            "nopfs_prefetch_order",
            "nopfs_staging_schedule", "nopfs_fetch_model", "nopfs_buffer_sim", "nopfs_policy_sim",
            "nopfs_strerror",
            "nopfs_last_error", "nopfs_profile_enable", "nopfs_profile_query",
            "nopfs_calibration_copy", "nopfs_scratch_release", "nopfs_debug_set")


def _check(rc: int, what: str):
    if rc != NOPFS_OK:
        L = lib()
        detail = L.nopfs_last_error().decode() or L.nopfs_strerror(rc).decode()
        raise NopfsError(rc, what, detail)


def _ptr(t) -> ctypes.c_void_p:
    if t is None:
        return ctypes.c_void_p(0)
    if isinstance(t, int):
        return ctypes.c_void_p(t)
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _device_tensor(t, dtype, shape, name):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)}")
    return t


def stream_shape(job: Job):
    """(T, M_max, [M_i]) on the host; no GPU needed."""
    T = ctypes.c_int64()
    M = ctypes.c_int64()
    Mw = (ctypes.c_int64 * int(job.N))()
    j = job.c()
    _check(lib().nopfs_stream_shape(ctypes.byref(j), ctypes.byref(T), ctypes.byref(M), Mw),
           "nopfs_stream_shape")
    return T.value, M.value, list(Mw)


def access_streams(job: Job, R=None, stream=None):
    _, M, _ = stream_shape(job)
    if R is None:
        R = torch.empty((job.N, M), dtype=torch.int32, device="cuda")
    _device_tensor(R, torch.int32, (job.N, M), "R")
    j = job.c()
    _check(lib().nopfs_access_streams(ctypes.byref(j), _ptr(R), _stream(stream)),
           "nopfs_access_streams")
    return R


def access_stats(job: Job, R, count=None, first=None, stream=None):
    _, M, _ = stream_shape(job)
    _device_tensor(R, torch.int32, (job.N, M), "R")
    if count is None:
        count = torch.empty((job.N, job.F), dtype=torch.uint8, device="cuda")
    if first is None:
        first = torch.empty((job.N, job.F), dtype=torch.int32, device="cuda")
    _device_tensor(count, torch.uint8, (job.N, job.F), "count")
    _device_tensor(first, torch.int32, (job.N, job.F), "first")
    j = job.c()
    _check(lib().nopfs_access_stats(ctypes.byref(j), _ptr(R), _ptr(count), _ptr(first),
                                    _stream(stream)), "nopfs_access_stats")
    return count, first


def access_streams_range(job: Job, e_begin: int, e_end: int, R=None, stream=None):
    """Streams of epochs [e_begin, e_end) (nopfs_access_streams_range), shaped
    as the streams of job.epochs(e_begin, e_end)."""
    sub = job.epochs(e_begin, e_end)
    M = stream_shape(sub)[1] if e_end > e_begin else 0
    if R is None:
        R = torch.empty((job.N, M), dtype=torch.int32, device="cuda")
    _device_tensor(R, torch.int32, (job.N, M), "R")
    j = job.c()
    _check(lib().nopfs_access_streams_range(ctypes.byref(j), int(e_begin), int(e_end), _ptr(R),
                                            _stream(stream)), "nopfs_access_streams_range")
    return R


def reuse_next(job: Job, R, next=None, stream=None):
    _, M, _ = stream_shape(job)
    _device_tensor(R, torch.int32, (job.N, M), "R")
    if next is None:
        next = torch.empty((job.N, M), dtype=torch.int32, device="cuda")
    _device_tensor(next, torch.int32, (job.N, M), "next")
    j = job.c()
    _check(lib().nopfs_reuse_next(ctypes.byref(j), _ptr(R), _ptr(next), _stream(stream)),
           "nopfs_reuse_next")
    return next


def tier_plan(job: Job, count, first, sizes, caps, tier=None, used=None, stream=None):
    """caps: host sequence of per-worker tier capacities (bytes), fastest first."""
    _device_tensor(count, torch.uint8, (job.N, job.F), "count")
    _device_tensor(first, torch.int32, (job.N, job.F), "first")
    _device_tensor(sizes, torch.int64, (job.F,), "sizes")
    caps_list = [int(c) for c in caps]
    J = len(caps_list)
    caps_host = (ctypes.c_int64 * max(J, 1))(*caps_list)
    if tier is None:
        tier = torch.empty((job.N, job.F), dtype=torch.int8, device="cuda")
    if used is None:
        used = torch.empty((job.N, max(J, 1)), dtype=torch.int64, device="cuda")
    _device_tensor(tier, torch.int8, (job.N, job.F), "tier")
    _device_tensor(used, torch.int64, (job.N, max(J, 1)), "used")
    j = job.c()
    _check(lib().nopfs_tier_plan(ctypes.byref(j), _ptr(count), _ptr(first), _ptr(sizes),
                                 ctypes.cast(caps_host, ctypes.c_void_p), J, _ptr(tier),
                                 _ptr(used), _stream(stream)), "nopfs_tier_plan")
    return tier, used


def plan_job(job: Job, sizes, caps, out=None, stream=None):
    """The whole path in one library call (nopfs_plan_job); the same outputs
    as plan(). `out` may hold preallocated R, count, first, next, tier, used."""
    return _plan_job("nopfs_plan_job", job, sizes, caps, out, stream)


def plan_job_noalloc(job: Job, sizes, caps, out, stream=None):
    """nopfs_plan_job_noalloc: plan_job with the library's fixed per-device
    scratch array, no device allocation by the library. `out` must hold all
    six preallocated outputs."""
    for name in ("R", "count", "first", "next", "tier", "used"):
        if out.get(name) is None:
            raise ValueError(f"plan_job_noalloc needs a preallocated {name}")
    return _plan_job("nopfs_plan_job_noalloc", job, sizes, caps, out, stream)


def _plan_job(fn, job: Job, sizes, caps, out, stream):
    _, M, _ = stream_shape(job)
    _device_tensor(sizes, torch.int64, (job.F,), "sizes")
    caps_list = [int(c) for c in caps]
    J = len(caps_list)
    caps_host = (ctypes.c_int64 * max(J, 1))(*caps_list)
    shapes = dict(R=((job.N, M), torch.int32), count=((job.N, job.F), torch.uint8),
                  first=((job.N, job.F), torch.int32), next=((job.N, M), torch.int32),
                  tier=((job.N, job.F), torch.int8), used=((job.N, max(J, 1)), torch.int64))
    o = dict(out or {})
    for name, (shape, dt) in shapes.items():
        if o.get(name) is None:
            o[name] = torch.empty(shape, dtype=dt, device="cuda")
        _device_tensor(o[name], dt, shape, name)
    j = job.c()
    _check(getattr(lib(), fn)(ctypes.byref(j), _ptr(sizes), ctypes.cast(caps_host, ctypes.c_void_p),
                              J, _ptr(o["R"]), _ptr(o["count"]), _ptr(o["first"]), _ptr(o["next"]),
                              _ptr(o["tier"]), _ptr(o["used"]), _stream(stream)), fn)
    return o


def prefetch_order(job: Job, R, tier, J, order=None, qlen=None, stream=None):
    """Per-tier prefetch queues (nopfs_prefetch_order): order [N][M_max] int32
    (tier 0's queue, tier 1's, ..., then -1) and qlen [N][J] int64."""
    _, M, _ = stream_shape(job)
    _device_tensor(R, torch.int32, (job.N, M), "R")
    _device_tensor(tier, torch.int8, (job.N, job.F), "tier")
    J = int(J)
    if order is None:
        order = torch.empty((job.N, M), dtype=torch.int32, device="cuda")
    if qlen is None:
        qlen = torch.empty((job.N, max(J, 1)), dtype=torch.int64, device="cuda")
    _device_tensor(order, torch.int32, (job.N, M), "order")
    _device_tensor(qlen, torch.int64, (job.N, max(J, 1)), "qlen")
    j = job.c()
    _check(lib().nopfs_prefetch_order(ctypes.byref(j), _ptr(R), _ptr(tier), J,
                                      _ptr(order), _ptr(qlen), _stream(stream)),
           "nopfs_prefetch_order")
    return order, qlen


def staging_schedule(job: Job, R, sizes, d0, fill=None, stream=None):
    """Staging-buffer schedule (nopfs_staging_schedule): fill [N][M_max] int32,
    the first stream position from which each read's sample may be staged
    into a buffer of d0 bytes (-1 in padding)."""
    _, M, _ = stream_shape(job)
    _device_tensor(R, torch.int32, (job.N, M), "R")
    _device_tensor(sizes, torch.int64, (job.F,), "sizes")
    if fill is None:
        fill = torch.empty((job.N, M), dtype=torch.int32, device="cuda")
    _device_tensor(fill, torch.int32, (job.N, M), "fill")
    j = job.c()
    _check(lib().nopfs_staging_schedule(ctypes.byref(j), _ptr(R), _ptr(sizes), int(d0), _ptr(fill),
                                        _stream(stream)), "nopfs_staging_schedule")
    return fill


def fetch_model(job: Job, R, tier, sizes, model: Model, src=None, t=None, stream=None):
    """Fetch source and consumption time of every read under the performance
    model (nopfs_fetch_model): src [N][M_max] int16 (0 PFS, 128 + j another
    worker's tier j, 256 + j own tier j, -1 padding), t [N][M_max] float64
    seconds (-1 padding)."""
    _, M, _ = stream_shape(job)
    _device_tensor(R, torch.int32, (job.N, M), "R")
    _device_tensor(tier, torch.int8, (job.N, job.F), "tier")
    _device_tensor(sizes, torch.int64, (job.F,), "sizes")
    if src is None:
        src = torch.empty((job.N, M), dtype=torch.int16, device="cuda")
    if t is None:
        t = torch.empty((job.N, M), dtype=torch.float64, device="cuda")
    _device_tensor(src, torch.int16, (job.N, M), "src")
    _device_tensor(t, torch.float64, (job.N, M), "t")
    j = job.c()
    _check(lib().nopfs_fetch_model(ctypes.byref(j), _ptr(R), _ptr(tier), _ptr(sizes),
                                   ctypes.byref(model), _ptr(src), _ptr(t), _stream(stream)),
           "nopfs_fetch_model")
    return src, t


def buffer_sim(job: Job, R, next, sizes, d0, hit=None, hits=None, stream=None):
    """Clairvoyant buffer of d0 bytes per worker (nopfs_buffer_sim): hit
    [N][M_max] int8 (1 hit, 0 miss, -1 padding), hits [N][2] int64 (hits, hit
    bytes)."""
    _, M, _ = stream_shape(job)
    _device_tensor(R, torch.int32, (job.N, M), "R")
    _device_tensor(next, torch.int32, (job.N, M), "next")
    _device_tensor(sizes, torch.int64, (job.F,), "sizes")
    if hit is None:
        hit = torch.empty((job.N, M), dtype=torch.int8, device="cuda")
    if hits is None:
        hits = torch.empty((job.N, 2), dtype=torch.int64, device="cuda")
    _device_tensor(hit, torch.int8, (job.N, M), "hit")
    _device_tensor(hits, torch.int64, (job.N, 2), "hits")
    j = job.c()
    _check(lib().nopfs_buffer_sim(ctypes.byref(j), _ptr(R), _ptr(next), _ptr(sizes), int(d0),
                                  _ptr(hit), _ptr(hits), _stream(stream)), "nopfs_buffer_sim")
    return hit, hits


POLICY_PERFECT, POLICY_NAIVE, POLICY_STAGING, POLICY_NOPFS = 0, 1, 2, 3


def policy_sim(job: Job, R, sizes, model, policy, src=None, fill=None, t=None, finish=None,
               io=None, stream=None):
    """Simulated training time under a data-loading policy (nopfs_policy_sim):
    t [N][M_max] float64 consumption times (-1 padding), finish [N], io
    [N][1 + 2J] fetch time by source class."""
    _, M, _ = stream_shape(job)
    _device_tensor(R, torch.int32, (job.N, M), "R")
    _device_tensor(sizes, torch.int64, (job.F,), "sizes")
    if src is not None:
        _device_tensor(src, torch.int16, (job.N, M), "src")
    if fill is not None:
        _device_tensor(fill, torch.int32, (job.N, M), "fill")
    K = 1 + 2 * model.J
    if t is None:
        t = torch.empty((job.N, M), dtype=torch.float64, device="cuda")
    if finish is None:
        finish = torch.empty(job.N, dtype=torch.float64, device="cuda")
    if io is None:
        io = torch.empty((job.N, K), dtype=torch.float64, device="cuda")
    _device_tensor(t, torch.float64, (job.N, M), "t")
    _device_tensor(finish, torch.float64, (job.N,), "finish")
    _device_tensor(io, torch.float64, (job.N, K), "io")
    j = job.c()
    _check(lib().nopfs_policy_sim(ctypes.byref(j), _ptr(R), _ptr(sizes),
                                  None if src is None else _ptr(src),
                                  None if fill is None else _ptr(fill), ctypes.byref(model),
                                  int(policy), _ptr(t), _ptr(finish), _ptr(io), _stream(stream)),
           "nopfs_policy_sim")
    return t, finish, io


def plan(job: Job, sizes, caps, stream=None):
    """The whole path: streams, stats, next use, tier plan (all on device)."""
    R = access_streams(job, stream=stream)
    count, first = access_stats(job, R, stream=stream)
    nxt = reuse_next(job, R, stream=stream)
    tier, used = tier_plan(job, count, first, sizes, caps, stream=stream)
    return dict(R=R, count=count, first=first, next=nxt, tier=tier, used=used)


# -- measurement aids -----------------------------------------------------------
def profile_enable(on: bool):
    _check(lib().nopfs_profile_enable(1 if on else 0), "nopfs_profile_enable")


def profile_results():
    """{kernel name: (launches, total ms)} for kernels since profile_enable(True)."""
    out = {}
    idx = 0
    while True:
        name = ctypes.c_char_p()
        n = ctypes.c_int64()
        ms = ctypes.c_double()
        rc = lib().nopfs_profile_query(idx, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms))
        if rc == NOPFS_EINVAL:
            break
        _check(rc, "nopfs_profile_query")
        out[name.value.decode()] = (n.value, ms.value)
        idx += 1
    return out


def scratch_release(stream=None):
    """Frees the scratch block of (current device, stream) after the
    stream's work completes (nopfs_scratch_release)."""
    _check(lib().nopfs_scratch_release(_stream(stream)), "nopfs_scratch_release")


def calibration_copy(src, dst, nbytes: int, stream=None):
    _check(lib().nopfs_calibration_copy(_ptr(src), _ptr(dst), int(nbytes), _stream(stream)),
           "nopfs_calibration_copy")


def debug_set(which: int, value: int):
    _check(lib().nopfs_debug_set(int(which), int(value)), "nopfs_debug_set")
