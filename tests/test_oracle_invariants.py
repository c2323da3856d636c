"""Invariants of the oracle on the small workload and random small jobs."""
import numpy as np
import pytest

import invariants as inv
from paper_2101_08734_amd import workloads as wl

JOBS = [
    (10_000, 5, 4, 16, 1, 42), (10_000, 5, 4, 16, 1, 7),
    (1_003, 7, 5, 3, 0, 3), (777, 4, 3, 10, 1, 5), (50, 9, 8, 1, 0, 11),
    (64, 3, 100, 1, 0, 12), (10, 2, 4, 3, 1, 13), (4_099, 6, 7, 8, 0, 14),
]


@pytest.mark.parametrize("F,E,N,B,d,seed", JOBS)
def test_invariants(oracle, F, E, N, B, d, seed):
    job = oracle.make_job(F, E, N, B, d, seed)
    _, _, Mw = oracle.stream_shape(job)
    for e in range(min(E, 3)):
        inv.check_perm(oracle.epoch_perm(job, e), oracle.epoch_keys(job, e))
    R = oracle.access_streams(job)
    inv.check_streams(R, F, E, Mw)
    inv.check_issued_once(R, F, E, Mw)
    count, first = oracle.access_stats(job, R)
    inv.check_stats(R, count, first, Mw, E)
    if not d:
        # nothing dropped: every sample read exactly E times over all workers
        assert (count.sum(axis=0) == E).all()
    nxt = oracle.reuse_next(job, R)
    inv.check_next(R, nxt, Mw, E)
    sizes = wl.random_sizes(F, seed, 1, 1000)
    total = int(sizes.sum())
    for caps in ([total // 7, total // 3], [total // 50], [0, total],
                 [total + 1], [0], [1, 2, 3]):
        caps = np.array(caps, np.int64)
        tier, used = oracle.tier_plan(job, count, first, sizes, caps)
        inv.check_plan(count, first, sizes, caps, tier, used)
        if caps[0] >= total:
            assert (tier == 0).all()
        if caps.max() == 0:
            assert (tier == -1).all()


def test_streams_from_perms_matches(oracle):
    job = oracle.make_job(1000, 4, 3, 7, 0, 9)
    perms = np.stack([oracle.epoch_perm(job, e) for e in range(4)])
    np.testing.assert_array_equal(oracle.streams_from_perms(job, perms),
                                  oracle.access_streams(job))


@pytest.mark.parametrize("F,E,N,B,d,seed", JOBS[:6])
def test_sample_columns_agree(oracle, F, E, N, B, d, seed):
    """The per-sample path (rank by counting) against the full path (sort)."""
    job = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(job)
    count, first = oracle.access_stats(job, R)
    nxt = oracle.reuse_next(job, R)
    samples = np.random.default_rng(seed).choice(F, size=min(F, 40), replace=False)
    cols = oracle.sample_columns(job, samples)
    for e in range(E):
        perm = oracle.epoch_perm(job, e)
        np.testing.assert_array_equal(perm[cols["pos"][e]], samples)
    np.testing.assert_array_equal(cols["col_count"], count[:, samples])
    np.testing.assert_array_equal(cols["col_first"], first[:, samples])
    for e in range(E):
        for s_idx, k in enumerate(samples):
            i, f = cols["occ_worker"][e, s_idx], cols["occ_f"][e, s_idx]
            if i < 0:
                continue
            assert R[i, f] == k
            assert nxt[i, f] == cols["occ_next"][e, s_idx]


def test_row_variants_agree(oracle):
    job = oracle.make_job(3_001, 5, 7, 4, 0, 23)
    R = oracle.access_streams(job)
    count, first = oracle.access_stats(job, R)
    nxt = oracle.reuse_next(job, R)
    c2, f2 = oracle.access_stats_rows(job, R[3:6], 3)
    np.testing.assert_array_equal(c2, count[3:6])
    np.testing.assert_array_equal(f2, first[3:6])
    np.testing.assert_array_equal(oracle.reuse_next_rows(job, R[2:7], 2), nxt[2:7])
