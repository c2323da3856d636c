"""Brute force on tiny jobs (F <= 8): every stage of the oracle against
enumeration with predicates (tests/brute.py)."""
import itertools

import numpy as np
import pytest

import brute

SHAPES = [
    # F, E, N, B, drop_last
    (1, 1, 1, 1, 1), (1, 3, 2, 1, 0), (2, 2, 1, 1, 1), (3, 2, 2, 1, 0),
    (4, 2, 2, 1, 1), (5, 3, 2, 2, 0), (6, 4, 3, 1, 1), (7, 3, 2, 3, 0),
    (8, 4, 4, 1, 1), (8, 3, 3, 2, 0), (8, 4, 1, 3, 1), (7, 4, 4, 2, 1),
]


@pytest.mark.parametrize("F,E,N,B,d", SHAPES)
@pytest.mark.parametrize("seed", [1, 42])
def test_streams_stats_next_brute(oracle, F, E, N, B, d, seed):
    job = oracle.make_job(F, E, N, B, d, seed)
    perms = []
    for e in range(E):
        keys = [int(x) for x in oracle.epoch_keys(job, e)]
        p = brute.certified_perm(keys)
        np.testing.assert_array_equal(oracle.epoch_perm(job, e), p)
        perms.append(p)
    R = oracle.access_streams(job)
    Rb = brute.streams(F, E, N, B, d, perms)
    if R.shape[1] == 0:
        assert all(len(r) == 0 for r in Rb)
        return
    np.testing.assert_array_equal(R, Rb)
    count, first = oracle.access_stats(job, R)
    cb, fb = brute.stats(F, Rb)
    np.testing.assert_array_equal(count, cb)
    np.testing.assert_array_equal(first, fb)
    np.testing.assert_array_equal(oracle.reuse_next(job, R), brute.next_use(Rb))


def test_equal_keys_go_by_id():
    keys = [5, 3, 5, 3, 1]
    assert brute.certified_perm(keys) == [4, 1, 3, 0, 2]


PLAN_CASES = []
rng = np.random.default_rng(2024)
for F in (1, 2, 3, 5, 6):
    for J in (1, 2, 3):
        PLAN_CASES.append((F, J, int(rng.integers(1 << 30))))
PLAN_CASES += [(7, 2, 11), (7, 3, 12), (8, 1, 13), (8, 2, 14)]


@pytest.mark.parametrize("F,J,s", PLAN_CASES)
def test_plan_brute(oracle, F, J, s):
    r = np.random.default_rng(s)
    E = int(r.integers(1, 5))
    N = int(r.integers(1, 4))
    job = oracle.make_job(F, E, N, 1, int(r.integers(0, 2)), int(s))
    R = oracle.access_streams(job)
    count, first = oracle.access_stats(job, R)
    sizes = r.integers(1, 20, F).astype(np.int64)
    # capacities from "nothing fits" to "everything fits"
    caps = r.integers(0, int(sizes.sum()) + 2, J).astype(np.int64)
    tier, used = oracle.tier_plan(job, count, first, sizes, caps)
    for i in range(count.shape[0]):
        assign, u = brute.plan_row(list(count[i]), list(first[i]),
                                   list(sizes), list(caps))
        np.testing.assert_array_equal(tier[i], assign)
        np.testing.assert_array_equal(used[i], u)


def test_plan_brute_ties_and_oversize(oracle):
    # hand-made rows with equal counts, a sample bigger than every tier,
    # zero capacity and exact fits
    count = np.array([[1, 1, 0, 2, 0, 1]], np.uint8)
    first = np.array([[4, 0, -1, 2, -1, 7]], np.int32)
    sizes = np.array([3, 9, 4, 5, 100, 4], np.int64)
    for caps in ([0, 8], [5, 0, 20], [9, 4], [200], [12, 3, 7]):
        job = oracle.make_job(6, 3, 1, 1, 1, 0)
        tier, used = oracle.tier_plan(job, count, first, sizes, np.array(caps))
        assign, u = brute.plan_row(list(count[0]), list(first[0]), list(sizes),
                                   caps)
        np.testing.assert_array_equal(tier[0], assign)
        np.testing.assert_array_equal(used[0], u)
