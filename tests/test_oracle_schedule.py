"""Pins for the oracle's prefetch order and staging schedule.

Prefetch order (Design: each storage class is filled in the order its
samples are first needed -- the first rule of optimal prefetching from the
I/O Access Patterns section): re-derived here from the other direction, by
sorting each tier's read samples by their first read, instead of walking R.

Staging schedule (Design: the staging buffer is filled in R order and a
sample is dropped once read; Implementation: the buffer is filled
circularly): re-derived by brute force, the smallest window start whose
window fits, for every position; plus closed forms (unlimited buffer, empty
buffer, equal sizes) that an off-by-one in the fit test would break.
"""
import numpy as np
import pytest

from paper_2101_08734_amd import workloads as wl

JOBS = [
    # F, E, N, B, drop_last, seed, cap fractions
    (60, 4, 3, 2, 1, 1, (0.2, 0.3)),
    (97, 5, 4, 3, 0, 2, (0.1, 0.1, 0.5)),
    (40, 7, 2, 5, 0, 3, (0.05,)),
    (33, 3, 5, 1, 1, 4, (0.0, 1.0)),
    (128, 6, 8, 2, 0, 5, (0.3, 0.3)),
]


def _pipeline(oracle, F, E, N, B, d, seed, fr):
    job = oracle.make_job(F, E, N, B, d, seed)
    sizes = wl.random_sizes(F, seed, 1_000, 200_000)
    caps = np.array([int(f * sizes.sum()) for f in fr], np.int64)
    return job, sizes, caps, oracle.full_pipeline(job, sizes, caps)


@pytest.mark.parametrize("F,E,N,B,d,seed,fr", JOBS)
def test_prefetch_order_by_first_read(oracle, F, E, N, B, d, seed, fr):
    job, sizes, caps, out = _pipeline(oracle, F, E, N, B, d, seed, fr)
    J = len(caps)
    order, qlen = oracle.prefetch_order(job, out["R"], out["first"], out["tier"], J)
    M = out["R"].shape[1]
    for i in range(N):
        want = []
        for j in range(J):
            ks = [k for k in range(F) if out["tier"][i][k] == j and out["first"][i][k] >= 0]
            ks.sort(key=lambda k: out["first"][i][k])
            assert qlen[i][j] == len(ks)
            want += ks
        want += [-1] * (M - len(want))
        np.testing.assert_array_equal(order[i], want)


def _brute_fill(sizes_along, d0):
    out = []
    for h in range(len(sizes_along)):
        f = h
        for g in range(h + 1):
            if sum(sizes_along[g:h + 1]) <= d0:
                f = g
                break
        out.append(f)
    return out


@pytest.mark.parametrize("F,E,N,B,d,seed,fr", JOBS)
def test_staging_schedule_brute_force(oracle, F, E, N, B, d, seed, fr):
    job, sizes, caps, out = _pipeline(oracle, F, E, N, B, d, seed, fr)
    R = out["R"]
    total = int(sizes.sum())
    for d0 in (0, 1, int(sizes.max()) - 1, int(sizes.max()), 300_000, 1_000_000, total * 10):
        fill = oracle.staging_schedule(job, R, sizes, d0)
        for i in range(N):
            row = R[i][R[i] >= 0]
            want = _brute_fill([int(sizes[k]) for k in row], d0)
            want += [-1] * (R.shape[1] - len(want))
            np.testing.assert_array_equal(fill[i], want, err_msg=f"worker {i} d0={d0}")


def test_staging_closed_forms(oracle):
    """Equal sizes s and a buffer of m*s bytes hold exactly m samples:
    fill(h) = max(0, h - m + 1); an unlimited buffer gives 0, an empty one h."""
    F, E, N, B = 5_000, 3, 4, 8
    job = oracle.make_job(F, E, N, B, 0, 9)
    R = oracle.access_streams(job)
    s = 16_777_216
    sizes = np.full(F, s, np.int64)
    Mi = [(E * ((F - i + N - 1) // N)) for i in range(N)]
    for m in (1, 2, 7, 300):
        fill = oracle.staging_schedule(job, R, sizes, m * s)
        for i in range(N):
            h = np.arange(Mi[i])
            np.testing.assert_array_equal(fill[i][:Mi[i]], np.maximum(0, h - m + 1))
            assert (fill[i][Mi[i]:] == -1).all()
    fill = oracle.staging_schedule(job, R, sizes, s * F * E)
    for i in range(N):
        assert (fill[i][:Mi[i]] == 0).all()
    fill = oracle.staging_schedule(job, R, sizes, 0)
    for i in range(N):
        np.testing.assert_array_equal(fill[i][:Mi[i]], np.arange(Mi[i]))


def test_prefetch_order_invariants_medium(oracle):
    """Every read sample of a cache tier is queued once, in increasing first
    read; the queues hold exactly the read samples of tiers >= 0."""
    F, E, N, B, d, seed = 20_000, 6, 5, 16, 0, 12
    job, sizes, caps, out = _pipeline(oracle, F, E, N, B, d, seed, (0.05, 0.2))
    order, qlen = oracle.prefetch_order(job, out["R"], out["first"], out["tier"], 2)
    for i in range(N):
        start = 0
        for j in range(2):
            q = order[i][start:start + qlen[i][j]]
            start += qlen[i][j]
            assert (out["tier"][i][q] == j).all()
            f = out["first"][i][q]
            assert (f >= 0).all() and (np.diff(f) > 0).all()
        read_cached = (out["first"][i] >= 0) & (out["tier"][i] >= 0)
        assert start == int(read_cached.sum())
        assert (order[i][start:] == -1).all()


def test_argument_errors(oracle):
    job = oracle.make_job(10, 2, 2, 1)
    R = oracle.access_streams(job)
    count, first = oracle.access_stats(job, R)
    tier = np.zeros((2, 10), np.int8)
    with pytest.raises(Exception):
        oracle.prefetch_order(job, R, first, tier, 0)
    with pytest.raises(Exception):
        oracle.staging_schedule(job, R, np.ones(10, np.int64), -1)
