"""The C ABI on the host (no GPU): the library loads, exports every entry
point that include/nopfs.h declares, and validates arguments before any
device work. Pointers passed here are never dereferenced: every call below
returns an error before it enqueues anything."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nopfs.h")

nopfs = pytest.importorskip("paper_2101_08734_amd.nopfs")

FAKE = ctypes.c_void_p(0x1000)  # never dereferenced by the failing calls below


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nopfs_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(nopfs.LIB_PATH):
        from paper_2101_08734_amd import build
        build.build()
    return nopfs.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) >= 11
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(nopfs.EXPORTED)


@pytest.mark.parametrize("F,E,N,B,d", [
    (10_000, 5, 4, 16, 1), (1_281_167, 90, 16, 32, 1), (1_281_167, 90, 256, 32, 1),
    (14_197_103, 40, 256, 32, 1), (262_144, 40, 1_024, 1, 1), (1_003, 7, 5, 3, 0),
    (5, 2, 2, 2, 0), (10, 2, 4, 3, 1), (1, 1, 3, 1, 0), (64, 3, 100, 1, 0)])
def test_shape_matches_oracle(L, oracle, F, E, N, B, d):
    T, M, Mw = nopfs.stream_shape(nopfs.Job(F, E, N, B, d, 1))
    rT, rM, rMw = oracle.stream_shape(oracle.make_job(F, E, N, B, d, 1))
    assert (T, M) == (rT, rM)
    assert list(Mw) == list(rMw)


def _job(**kw):
    base = dict(F=100, E=3, N=2, B=4, drop_last=1, seed=1)
    base.update(kw)
    return nopfs._Job(base["F"], base["E"], base["N"], base["B"], base["drop_last"], base["seed"])


@pytest.mark.parametrize("kw,code", [
    (dict(F=0), nopfs.NOPFS_EINVAL), (dict(E=0), nopfs.NOPFS_EINVAL),
    (dict(N=0), nopfs.NOPFS_EINVAL), (dict(B=0), nopfs.NOPFS_EINVAL),
    (dict(drop_last=2), nopfs.NOPFS_EINVAL), (dict(F=2**31), nopfs.NOPFS_ERANGE),
    (dict(E=256), nopfs.NOPFS_ERANGE),
    (dict(F=2**31 - 1, E=2, N=1, B=1, drop_last=0), nopfs.NOPFS_ERANGE),  # M_max >= 2^31
])
def test_invalid_jobs(L, kw, code):
    j = _job(**kw)
    T = ctypes.c_int64()
    assert L.nopfs_stream_shape(ctypes.byref(j), ctypes.byref(T), None, None) == code
    assert L.nopfs_access_streams(ctypes.byref(j), FAKE, None) == code
    assert L.nopfs_access_stats(ctypes.byref(j), FAKE, FAKE, FAKE, None) == code
    assert L.nopfs_reuse_next(ctypes.byref(j), FAKE, FAKE, None) == code
    caps = (ctypes.c_int64 * 1)(10)
    assert L.nopfs_tier_plan(ctypes.byref(j), FAKE, FAKE, FAKE, caps, 1, FAKE, FAKE, None) == code
    assert L.nopfs_prefetch_order(ctypes.byref(j), FAKE, FAKE, 1, FAKE, FAKE, None) == code
    assert L.nopfs_staging_schedule(ctypes.byref(j), FAKE, FAKE, 10, FAKE, None) == code
    m = _model()
    assert L.nopfs_fetch_model(ctypes.byref(j), FAKE, FAKE, FAKE, ctypes.byref(m), FAKE, FAKE,
                               None) == code
    assert L.nopfs_last_error()  # a detail string is recorded


def test_null_pointers(L):
    j = _job()
    E = nopfs.NOPFS_EINVAL
    assert L.nopfs_stream_shape(None, None, None, None) == E
    assert L.nopfs_access_streams(ctypes.byref(j), None, None) == E
    assert L.nopfs_access_stats(ctypes.byref(j), None, FAKE, FAKE, None) == E
    assert L.nopfs_access_stats(ctypes.byref(j), FAKE, None, FAKE, None) == E
    assert L.nopfs_reuse_next(ctypes.byref(j), FAKE, None, None) == E
    caps = (ctypes.c_int64 * 2)(10, 20)
    assert L.nopfs_tier_plan(ctypes.byref(j), FAKE, FAKE, None, caps, 2, FAKE, FAKE, None) == E
    assert L.nopfs_tier_plan(ctypes.byref(j), FAKE, FAKE, FAKE, None, 2, FAKE, FAKE, None) == E
    po = L.nopfs_prefetch_order
    assert po(ctypes.byref(j), None, FAKE, 1, FAKE, FAKE, None) == E
    assert po(ctypes.byref(j), FAKE, None, 1, FAKE, FAKE, None) == E
    assert po(ctypes.byref(j), FAKE, FAKE, 1, None, FAKE, None) == E
    assert po(ctypes.byref(j), FAKE, FAKE, 1, FAKE, None, None) == E
    assert po(None, FAKE, FAKE, 1, FAKE, FAKE, None) == E
    ss = L.nopfs_staging_schedule
    assert ss(ctypes.byref(j), None, FAKE, 10, FAKE, None) == E
    assert ss(ctypes.byref(j), FAKE, None, 10, FAKE, None) == E
    assert ss(ctypes.byref(j), FAKE, FAKE, 10, None, None) == E
    assert ss(None, FAKE, FAKE, 10, FAKE, None) == E


def test_plan_argument_checks(L):
    j = _job()
    caps = (ctypes.c_int64 * 128)(*([5] * 128))
    assert L.nopfs_tier_plan(ctypes.byref(j), FAKE, FAKE, FAKE, caps, 0, FAKE, FAKE, None) == nopfs.NOPFS_EINVAL
    assert L.nopfs_tier_plan(ctypes.byref(j), FAKE, FAKE, FAKE, caps, 128, FAKE, FAKE, None) == nopfs.NOPFS_ERANGE
    neg = (ctypes.c_int64 * 2)(5, -1)
    assert L.nopfs_tier_plan(ctypes.byref(j), FAKE, FAKE, FAKE, neg, 2, FAKE, FAKE, None) == nopfs.NOPFS_EINVAL


def test_schedule_argument_checks(L):
    j = _job()
    po = L.nopfs_prefetch_order
    assert po(ctypes.byref(j), FAKE, FAKE, 0, FAKE, FAKE, None) == nopfs.NOPFS_EINVAL
    assert po(ctypes.byref(j), FAKE, FAKE, -3, FAKE, FAKE, None) == nopfs.NOPFS_EINVAL
    assert po(ctypes.byref(j), FAKE, FAKE, 128, FAKE, FAKE, None) == nopfs.NOPFS_ERANGE
    ss = L.nopfs_staging_schedule
    assert ss(ctypes.byref(j), FAKE, FAKE, -1, FAKE, None) == nopfs.NOPFS_EINVAL
    assert b"d0" in L.nopfs_last_error()
    # no stream position at all (zero iterations): R and fill may be NULL
    empty = _job(F=10, N=4, B=3, drop_last=1)
    assert ss(ctypes.byref(empty), None, FAKE, 5, None, None) == 0


def _model(**kw):
    d = dict(c=64e6, beta=200e6, b_c=24e9, pfs_t=2870e6, pfs_gamma=8, w0=111e9, p0=8,
             r=[85e9, 4e9], p=[4, 2])
    d.update(kw)
    return nopfs.make_model(**d)


@pytest.mark.parametrize("kw,code", [
    (dict(c=0.0), nopfs.NOPFS_EINVAL), (dict(beta=-1.0), nopfs.NOPFS_EINVAL),
    (dict(b_c=float("nan")), nopfs.NOPFS_EINVAL), (dict(p0=float("inf")), nopfs.NOPFS_EINVAL),
    (dict(pfs_gamma=0.0), nopfs.NOPFS_EINVAL), (dict(r=[85e9, 0.0]), nopfs.NOPFS_EINVAL),
    (dict(p=[4, -2]), nopfs.NOPFS_EINVAL), (dict(r=[], p=[]), nopfs.NOPFS_EINVAL),
    (dict(r=[1e9] * 33, p=[1] * 33), nopfs.NOPFS_ERANGE),
])
def test_model_argument_checks(L, kw, code):
    j = _job()
    m = _model(**kw)
    if len(kw.get("r", [])) > 32:
        m.J = 33
    assert L.nopfs_fetch_model(ctypes.byref(j), FAKE, FAKE, FAKE, ctypes.byref(m), FAKE, FAKE,
                               None) == code


def test_model_null_pointers(L):
    j = _job()
    m = _model()
    fm = L.nopfs_fetch_model
    E = nopfs.NOPFS_EINVAL
    assert fm(ctypes.byref(j), FAKE, FAKE, FAKE, None, FAKE, FAKE, None) == E
    assert fm(ctypes.byref(j), FAKE, None, FAKE, ctypes.byref(m), FAKE, FAKE, None) == E
    assert fm(ctypes.byref(j), FAKE, FAKE, None, ctypes.byref(m), FAKE, FAKE, None) == E
    assert fm(ctypes.byref(j), None, FAKE, FAKE, ctypes.byref(m), FAKE, FAKE, None) == E
    assert fm(ctypes.byref(j), FAKE, FAKE, FAKE, ctypes.byref(m), None, FAKE, None) == E
    assert fm(ctypes.byref(j), FAKE, FAKE, FAKE, ctypes.byref(m), FAKE, None, None) == E
    assert fm(None, FAKE, FAKE, FAKE, ctypes.byref(m), FAKE, FAKE, None) == E


def test_buffer_argument_checks(L):
    j = _job()
    bs = L.nopfs_buffer_sim
    E = nopfs.NOPFS_EINVAL
    assert bs(ctypes.byref(j), FAKE, FAKE, FAKE, -1, FAKE, FAKE, None) == E
    assert bs(None, FAKE, FAKE, FAKE, 10, FAKE, FAKE, None) == E
    assert bs(ctypes.byref(j), None, FAKE, FAKE, 10, FAKE, FAKE, None) == E
    assert bs(ctypes.byref(j), FAKE, None, FAKE, 10, FAKE, FAKE, None) == E
    assert bs(ctypes.byref(j), FAKE, FAKE, None, 10, FAKE, FAKE, None) == E
    assert bs(ctypes.byref(j), FAKE, FAKE, FAKE, 10, None, FAKE, None) == E
    assert bs(ctypes.byref(j), FAKE, FAKE, FAKE, 10, FAKE, None, None) == E
    bad = _job(B=0)
    assert bs(ctypes.byref(bad), FAKE, FAKE, FAKE, 10, FAKE, FAKE, None) == E
    # a worker's stream of 2^24 reads or more is refused before any device work
    big = _job(F=1 << 24, E=1, N=1, B=1)
    assert bs(ctypes.byref(big), FAKE, FAKE, FAKE, 10, FAKE, FAKE, None) == nopfs.NOPFS_ERANGE
    ok = _job(F=(1 << 24) - 1, E=1, N=1, B=1)
    assert nopfs.stream_shape(nopfs.Job((1 << 24) - 1, 1, 1, 1, 1, 1))[1] == (1 << 24) - 1
    assert L.nopfs_debug_set(3, 1) == 0
    assert bs(ctypes.byref(ok), FAKE, FAKE, FAKE, 10, FAKE, FAKE, None) == nopfs.NOPFS_ENOMEM
    assert L.nopfs_debug_set(3, 0) == 0


def test_policy_argument_checks(L):
    j = _job()
    m = _model()
    ps = L.nopfs_policy_sim
    E = nopfs.NOPFS_EINVAL
    mp = ctypes.byref(m)
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, FAKE, mp, 4, FAKE, FAKE, FAKE, None) == E
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, FAKE, mp, -1, FAKE, FAKE, FAKE, None) == E
    assert ps(None, FAKE, FAKE, FAKE, FAKE, mp, 0, FAKE, FAKE, FAKE, None) == E
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, FAKE, None, 0, FAKE, FAKE, FAKE, None) == E
    assert ps(ctypes.byref(j), None, FAKE, FAKE, FAKE, mp, 0, FAKE, FAKE, FAKE, None) == E
    assert ps(ctypes.byref(j), FAKE, None, FAKE, FAKE, mp, 0, FAKE, FAKE, FAKE, None) == E
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, FAKE, mp, 0, None, FAKE, FAKE, None) == E
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, FAKE, mp, 0, FAKE, None, FAKE, None) == E
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, FAKE, mp, 0, FAKE, FAKE, None, None) == E
    # the staging policies need the schedule, NoPFS the sources
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, None, mp, 2, FAKE, FAKE, FAKE, None) == E
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, None, mp, 3, FAKE, FAKE, FAKE, None) == E
    assert ps(ctypes.byref(j), FAKE, FAKE, None, FAKE, mp, 3, FAKE, FAKE, FAKE, None) == E
    bad = _model(p0=0.0)
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, FAKE, ctypes.byref(bad), 0, FAKE, FAKE, FAKE,
              None) == E
    big = _model(r=[1e9] * 33, p=[1] * 33)
    big.J = 33
    assert ps(ctypes.byref(j), FAKE, FAKE, FAKE, FAKE, ctypes.byref(big), 0, FAKE, FAKE, FAKE,
              None) == nopfs.NOPFS_ERANGE


def test_stream_range_checks(L):
    j = _job(E=5)
    rs = L.nopfs_access_streams_range
    E = nopfs.NOPFS_EINVAL
    assert rs(ctypes.byref(j), -1, 3, FAKE, None) == E
    assert rs(ctypes.byref(j), 3, 2, FAKE, None) == E
    assert rs(ctypes.byref(j), 0, 6, FAKE, None) == E
    assert rs(ctypes.byref(j), 1, 3, None, None) == E
    assert rs(None, 0, 1, FAKE, None) == E
    # an empty range writes nothing and touches no pointer
    assert rs(ctypes.byref(j), 2, 2, None, None) == 0
    assert rs(ctypes.byref(j), 5, 5, None, None) == 0
    assert L.nopfs_debug_set(3, 1) == 0
    assert rs(ctypes.byref(j), 1, 4, FAKE, None) == nopfs.NOPFS_ENOMEM
    assert L.nopfs_debug_set(3, 0) == 0
    sub = nopfs.Job(100, 5, 2, 4, 1, 1).epochs(1, 4)
    assert (sub.E, sub.F, sub.N, sub.B) == (3, 100, 2, 4)


def test_scratch_failure_is_enomem(L):
    """The test hook fails the next internal allocation; the call reports
    NOPFS_ENOMEM before launching anything."""
    j = _job()
    caps = (ctypes.c_int64 * 1)(10)
    calls = [
        lambda: L.nopfs_access_streams(ctypes.byref(j), FAKE, None),
        lambda: L.nopfs_access_stats(ctypes.byref(j), FAKE, FAKE, FAKE, None),
        lambda: L.nopfs_reuse_next(ctypes.byref(j), FAKE, FAKE, None),
        lambda: L.nopfs_tier_plan(ctypes.byref(j), FAKE, FAKE, FAKE, caps, 1, FAKE, FAKE, None),
        lambda: L.nopfs_prefetch_order(ctypes.byref(j), FAKE, FAKE, 1, FAKE, FAKE, None),
        lambda: L.nopfs_staging_schedule(ctypes.byref(j), FAKE, FAKE, 10, FAKE, None),
        lambda: L.nopfs_fetch_model(ctypes.byref(j), FAKE, FAKE, FAKE, ctypes.byref(_model()),
                                    FAKE, FAKE, None),
        lambda: L.nopfs_buffer_sim(ctypes.byref(j), FAKE, FAKE, FAKE, 10, FAKE, FAKE, None),
    ]
    for call in calls:
        assert L.nopfs_debug_set(3, 1) == 0
        assert call() == nopfs.NOPFS_ENOMEM
        assert b"scratch" in L.nopfs_last_error()
    assert L.nopfs_debug_set(3, 0) == 0


def test_strerror(L):
    for c in (0, -1, -2, -3, -4, 7):
        assert L.nopfs_strerror(c)
    assert L.nopfs_debug_set(0, 1) == nopfs.NOPFS_EINVAL
    assert L.nopfs_debug_set(1, -5) == nopfs.NOPFS_EINVAL
    assert L.nopfs_debug_set(6, 1) == nopfs.NOPFS_EINVAL
    assert L.nopfs_debug_set(4, 0) == 0


def test_noalloc_rejects_a_job_beyond_its_scratch_on_the_host():
    """nopfs_plan_job_noalloc sizes a job's scratch on the host before it
    touches the device: a job that needs more than the fixed array is
    rejected with ERANGE (no GPU needed; the pointers are never used)."""
    L = nopfs.lib()
    fake = ctypes.c_void_p(1 << 40)
    caps = (ctypes.c_int64 * 2)(10**9, 10**10)
    j = nopfs.Job(1_000_000, 10, 8, 32).c()
    rc = L.nopfs_plan_job_noalloc(ctypes.byref(j), fake, ctypes.cast(caps, ctypes.c_void_p), 2,
                                  fake, fake, fake, fake, fake, fake, None)
    assert rc == nopfs.NOPFS_ERANGE
    assert "bytes of scratch" in L.nopfs_last_error().decode()
    j = nopfs.Job(1_000_000, 300, 8, 32).c()  # argument errors come first
    rc = L.nopfs_plan_job_noalloc(ctypes.byref(j), fake, ctypes.cast(caps, ctypes.c_void_p), 2,
                                  fake, fake, fake, fake, fake, fake, None)
    assert rc == nopfs.NOPFS_ERANGE and "E must be" in L.nopfs_last_error().decode()


def test_debug_hooks_accept_their_range_only(L):
    """Test hooks 1 to 5 take values >= 0; other hooks and negative values
    are EINVAL (host-only calls, no GPU work)."""
    for which in (1, 2, 3, 4, 5):
        assert L.nopfs_debug_set(which, 0) == 0
    assert L.nopfs_debug_set(0, 1) == nopfs.NOPFS_EINVAL
    assert L.nopfs_debug_set(6, 1) == nopfs.NOPFS_EINVAL
    assert L.nopfs_debug_set(5, -1) == nopfs.NOPFS_EINVAL
