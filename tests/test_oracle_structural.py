"""Hand-worked structural examples (tests/golden/structural_example.json).

The permutations are given, so these pin the shard, stats, next-use, plan,
prefetch-order and staging-schedule stages of the oracle independently of the
keys."""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "structural_example.json")
CASES = json.load(open(GOLDEN))["cases"]


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_structural_example(oracle, case):
    j = case["job"]
    job = oracle.make_job(j["F"], j["E"], j["N"], j["B"], j["drop_last"], j["seed"])
    R = oracle.streams_from_perms(job, np.array(case["perms"], np.int32))
    np.testing.assert_array_equal(R, case["R"])
    count, first = oracle.access_stats(job, R)
    np.testing.assert_array_equal(count, case["count"])
    np.testing.assert_array_equal(first, case["first"])
    np.testing.assert_array_equal(oracle.reuse_next(job, R), case["next"])
    tier, used = oracle.tier_plan(job, count, first, np.array(case["sizes"]),
                                  np.array(case["caps"]))
    np.testing.assert_array_equal(tier, case["tier"])
    np.testing.assert_array_equal(used, case["used"])
    order, qlen = oracle.prefetch_order(job, R, first, tier, len(case["caps"]))
    np.testing.assert_array_equal(order, case["prefetch_order"])
    np.testing.assert_array_equal(qlen, case["qlen"])
    for st in case["staging"]:
        fill = oracle.staging_schedule(job, R, np.array(case["sizes"]), st["d0"])
        np.testing.assert_array_equal(fill, st["fill"], err_msg=f"d0={st['d0']}")
