"""Pins for the oracle's clairvoyant buffer (I/O Access Patterns section:
Belady's replacement, discard the sample used furthest in the future; do no
harm, never discard a sample used before the one brought in).

 - unit sizes: the buffer is Belady's MIN with bypass, which is optimal; an
   exhaustive search over every admission and discard choice on small
   streams gives the largest possible number of hits, and the oracle must
   reach it exactly;
 - unit sizes: hits never decrease with capacity (MIN keeps the inclusion
   property);
 - a hand-worked case with variable sizes (tests/golden/buffer_sim_example.json);
 - closed forms: a buffer holding everything hits every read but the first
   of each sample; a buffer smaller than every sample never hits;
 - a hit is never a sample's first read, and its bytes add up.
"""
import functools
import json
import os

import numpy as np
import pytest

from paper_2101_08734_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "buffer_sim_example.json")


def _best_hits(stream, C):
    """Largest number of hits any policy gets with C unit slots (brute
    force over held sets; dropping is always free)."""
    M = len(stream)
    future = [set(stream[f + 1:]) for f in range(M)]

    @functools.lru_cache(maxsize=None)
    def go(f, held):
        if f == M:
            return 0
        k = stream[f]
        h = 1 if k in held else 0
        cand = (set(held) | {k}) & future[f]  # only samples used again matter
        cand = sorted(cand)
        best = 0
        # keep any subset of at most C candidates
        n = len(cand)
        for mask in range(1 << n):
            if bin(mask).count("1") > C:
                continue
            keep = frozenset(cand[b] for b in range(n) if mask >> b & 1)
            best = max(best, go(f + 1, keep))
        return h + best
    return go(0, frozenset())


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("C", [1, 2, 3])
def test_unit_sizes_optimal(oracle, seed, C):
    F, E, N, B = 6, 3, 1, 2
    job = oracle.make_job(F, E, N, B, 1, seed)
    R = oracle.access_streams(job)
    nx = oracle.reuse_next(job, R)
    hit, hits = oracle.buffer_sim(job, R, nx, np.ones(F, np.int64), C)
    stream = tuple(int(x) for x in R[0] if x >= 0)
    assert hits[0, 0] == _best_hits(stream, C)
    assert hits[0, 0] == int((hit[0] == 1).sum())


def test_unit_sizes_monotone_in_capacity(oracle):
    job = oracle.make_job(300, 8, 3, 10, 0, 4)
    R = oracle.access_streams(job)
    nx = oracle.reuse_next(job, R)
    ones = np.ones(300, np.int64)
    prev = None
    for C in range(0, 80, 3):
        _, hits = oracle.buffer_sim(job, R, nx, ones, C)
        if prev is not None:
            assert (hits[:, 0] >= prev).all()
        prev = hits[:, 0]


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_hand_worked(oracle, case):
    j = case["job"]
    job = oracle.make_job(j["F"], j["E"], j["N"], j["B"], j["drop_last"], 1)
    R = np.array(case["R"], np.int32)
    nx = oracle.reuse_next(job, R)
    hit, hits = oracle.buffer_sim(job, R, nx, np.array(case["sizes"], np.int64), case["d0"])
    np.testing.assert_array_equal(hit, case["hit"])
    np.testing.assert_array_equal(hits, case["hits"])


def test_closed_forms(oracle):
    F, E, N, B, d = 20_000, 5, 4, 8, 0
    job = oracle.make_job(F, E, N, B, d, 6)
    R = oracle.access_streams(job)
    nx = oracle.reuse_next(job, R)
    count, first = oracle.access_stats(job, R)
    sizes = wl.random_sizes(F, 3, 10, 1_000)
    _, _, Mw = oracle.stream_shape(job)
    # everything fits: every read but each sample's first hits
    hit, hits = oracle.buffer_sim(job, R, nx, sizes, int(sizes.sum()))
    for i in range(N):
        reread = int(Mw[i] - (count[i] > 0).sum())
        assert hits[i, 0] == reread
        k = R[i, :Mw[i]]
        first_read = first[i, k] == np.arange(Mw[i])
        assert (hit[i, :Mw[i]] == (~first_read)).all()
        assert hits[i, 1] == int(sizes[k][~first_read].sum())
    # smaller than every sample: nothing is ever held
    hit, hits = oracle.buffer_sim(job, R, nx, sizes, int(sizes.min()) - 1)
    assert (hits == 0).all() and (hit[hit >= 0] == 0).all()


def test_hits_are_rereads(oracle):
    F, E, N, B, d = 5_000, 6, 3, 8, 1
    job = oracle.make_job(F, E, N, B, d, 8)
    R = oracle.access_streams(job)
    nx = oracle.reuse_next(job, R)
    count, first = oracle.access_stats(job, R)
    sizes = wl.random_sizes(F, 9, 1_000, 2_000_000)
    _, _, Mw = oracle.stream_shape(job)
    for d0 in (3_000_000, 100_000_000, 1_000_000_000):
        hit, hits = oracle.buffer_sim(job, R, nx, sizes, d0)
        for i in range(N):
            k = R[i, :Mw[i]]
            h = hit[i, :Mw[i]] == 1
            assert (first[i, k][h] < np.arange(Mw[i])[h]).all()
            assert hits[i, 0] == h.sum() and hits[i, 1] == int(sizes[k][h].sum())
            assert (hit[i, Mw[i]:] == -1).all()


@pytest.mark.parametrize("d0", [2_000_000, 20_000_000, 200_000_000])
def test_capacity_never_exceeded(oracle, d0):
    """A hit at f means its sample was held from its previous read to f; at
    every moment the samples held that way fit in d0 bytes."""
    F, E, N, B, d = 4_000, 8, 2, 8, 0
    job = oracle.make_job(F, E, N, B, d, 12)
    R = oracle.access_streams(job)
    nx = oracle.reuse_next(job, R)
    sizes = wl.random_sizes(F, 13, 1_000, 2_000_000)
    hit, hits = oracle.buffer_sim(job, R, nx, sizes, d0)
    _, _, Mw = oracle.stream_shape(job)
    for i in range(N):
        m = Mw[i]
        prev = np.full(m, -1, np.int64)
        f = np.arange(m)
        has = nx[i, :m] >= 0
        prev[nx[i, :m][has]] = f[has]
        held = np.zeros(m + 1, np.int64)
        h = np.nonzero(hit[i, :m] == 1)[0]
        assert (prev[h] >= 0).all()
        sz = sizes[R[i, h]]
        np.add.at(held, prev[h], sz)
        np.add.at(held, h, -sz)
        assert np.cumsum(held).max() <= d0
    assert hits[:, 0].sum() > 0


def test_argument_errors(oracle):
    job = oracle.make_job(10, 2, 2, 1)
    R = oracle.access_streams(job)
    nx = oracle.reuse_next(job, R)
    with pytest.raises(Exception):
        oracle.buffer_sim(job, R, nx, np.ones(10, np.int64), -1)


def test_rows_match_full(oracle):
    """Workers are independent: a range of rows gives those rows of the full
    result (the sampled-row check at the largest size relies on this)."""
    F, E, N, B, d = 3_001, 4, 5, 7, 0
    job = oracle.make_job(F, E, N, B, d, 21)
    R = oracle.access_streams(job)
    nx = oracle.reuse_next(job, R)
    sizes = wl.random_sizes(F, 22, 1_000, 2_000_000)
    hit, hits = oracle.buffer_sim(job, R, nx, sizes, 50_000_000)
    for i0, i1 in ((0, 1), (2, 5), (4, 5), (1, 1)):
        h, t = oracle.buffer_sim(job, R[i0:i1], nx[i0:i1], sizes, 50_000_000, rows=(i0, i1))
        assert np.array_equal(h, hit[i0:i1]) and np.array_equal(t, hits[i0:i1])
    with pytest.raises(Exception):
        oracle.buffer_sim(job, R[:2], nx[:2], sizes, 1, rows=(4, 6))
