"""Shape arithmetic of the oracle against the batch-structure brute force and
the sizes of the five workloads."""
import itertools

import pytest

import brute

WORKLOAD_SHAPES = [
    # F, E, N, B, T, L, M
    (10_000, 5, 4, 16, 156, 2_496, 12_480),
    (1_281_167, 90, 16, 32, 2_502, 80_064, 7_205_760),
    (1_281_167, 90, 256, 32, 156, 4_992, 449_280),
    (14_197_103, 40, 256, 32, 1_733, 55_456, 2_218_240),
    (262_144, 40, 1_024, 1, 256, 256, 10_240),
]


@pytest.mark.parametrize("F,E,N,B,T,L,M", WORKLOAD_SHAPES)
def test_workload_shapes(oracle, F, E, N, B, T, L, M):
    job = oracle.make_job(F, E, N, B, 1, 42)
    t, mmax, mw = oracle.stream_shape(job)
    assert (t, mmax) == (T, M)
    assert (mw == M).all() and L * E == M


def test_shape_vs_batch_structure(oracle):
    for F, E, N, B, d in itertools.product([1, 2, 3, 5, 7, 8, 13, 64], [1, 3],
                                           [1, 2, 3, 4, 9], [1, 2, 5], [0, 1]):
        job = oracle.make_job(F, E, N, B, d, 1)
        T, mmax, mw = oracle.stream_shape(job)
        bT, bL, _ = brute.shape(F, E, N, B, d)
        assert T == bT
        assert list(mw) == [E * x for x in bL]
        assert mmax == E * max(bL)


def test_zero_iterations(oracle):
    # N*B > F with drop_last: no iteration, empty streams
    job = oracle.make_job(10, 2, 4, 3, 1, 1)
    T, mmax, _ = oracle.stream_shape(job)
    assert T == 0 and mmax == 0


def test_invalid_jobs(oracle):
    from oracle.ref import OracleError
    for args in [(0, 1, 1, 1, 1), (5, 0, 1, 1, 1), (5, 1, 0, 1, 1),
                 (5, 1, 1, 0, 1), (5, 1, 1, 1, 2), (5, 256, 1, 1, 1),
                 (2**31, 1, 1, 1, 1)]:
        with pytest.raises(OracleError):
            oracle.stream_shape(oracle.make_job(*args, 1))
