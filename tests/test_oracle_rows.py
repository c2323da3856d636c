"""The oracle's row-range shard (used by the full-size comparisons) against
its whole-job shard and the hand-worked examples.

Worker i's j-th read of epoch e is global position j*N + i (the worker
batches partition each global batch, performance model section); the
row-range function walks that map row by row, the whole-job function walks
the positions of each epoch, and the hand-worked cases fix the streams."""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "structural_example.json")
CASES = json.load(open(GOLDEN))["cases"]


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_rows_of_hand_worked_streams(oracle, case):
    j = case["job"]
    job = oracle.make_job(j["F"], j["E"], j["N"], j["B"], j["drop_last"], j["seed"])
    perms = np.array(case["perms"], np.int32)
    for i0 in range(job.N):
        for i1 in range(i0, job.N + 1):
            np.testing.assert_array_equal(oracle.streams_rows(job, perms, i0, i1),
                                          np.array(case["R"], np.int32)[i0:i1])


@pytest.mark.parametrize("F,E,N,B,drop_last", [
    (37, 3, 4, 2, 1), (37, 3, 4, 2, 0), (5, 2, 8, 1, 0), (5, 2, 8, 1, 1),
    (1000, 4, 7, 3, 0), (1000, 4, 7, 3, 1), (64, 2, 1, 64, 1), (1, 1, 1, 1, 0)])
def test_rows_equal_whole_job_shard(oracle, F, E, N, B, drop_last):
    job = oracle.make_job(F, E, N, B, drop_last, 3)
    rng = np.random.default_rng(F * 31 + N)
    perms = np.stack([rng.permutation(F) for _ in range(E)]).astype(np.int32)
    R = oracle.streams_from_perms(job, perms)
    for i0, i1 in [(0, N), (0, 1), (N - 1, N), (N // 2, N), (0, 0)]:
        np.testing.assert_array_equal(oracle.streams_rows(job, perms, i0, i1), R[i0:i1])
