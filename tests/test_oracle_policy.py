"""Pins for the oracle's policy simulation (Performance Simulator section:
the Perfect, Naive, StagingBuffer and NoPFS policies on the Performance
Modeling section's model).

 - two cases worked by hand where the buffer limit delays a read
   (tests/golden/policy_sim_example.json), all four policies, exactly;
 - closed forms: Perfect finishes after the summed compute time, Naive after
   the summed read and compute times; with equal sizes both staging
   policies give t(f) = r/p0 + f max(u, r/p0) whatever the buffer size;
 - with a buffer that holds the whole stream, StagingBuffer is the fetch
   model with no caches and NoPFS (with the fetch model's sources) is the
   fetch model itself, bit for bit (the fetch model is pinned on its own);
 - order: Perfect <= NoPFS <= StagingBuffer <= Naive read by read (p0 >= 1);
 - a larger buffer never delays a read.
"""
import json
import math
import os

import numpy as np
import pytest

from paper_2101_08734_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "policy_sim_example.json")
POLICIES = ("perfect", "naive", "staging", "nopfs")


def _model(oracle, **kw):
    d = dict(wl.LASSEN_MODEL)
    d.update(kw)
    return oracle.make_model(**d)


def _job_inputs(oracle, F=6_000, E=4, N=3, B=8, d=0, seed=5, caps=(0.05, 0.2)):
    job = oracle.make_job(F, E, N, B, d, seed)
    sizes = wl.random_sizes(F, seed + 1, 1_000, 2_000_000)
    tot = int(sizes.sum())
    out = oracle.full_pipeline(job, sizes, np.array([int(c * tot) for c in caps], np.int64))
    return job, sizes, out


@pytest.mark.parametrize("case", range(2))
def test_hand_worked(oracle, case):
    g = json.load(open(GOLDEN))["cases"][case]
    j = g["job"]
    job = oracle.make_job(j["F"], j["E"], j["N"], j["B"], j["drop_last"], j["seed"])
    R = np.array([g["R"]], np.int32)
    sizes = np.array(g["sizes"], np.int64)
    fill = oracle.staging_schedule(job, R, sizes, g["d0"])
    assert fill[0].tolist() == g["fill"]
    m = oracle.make_model(**g["model"])
    src = np.array([g["src"]], np.int16) if "src" in g else None
    for pol, name in enumerate(POLICIES):
        if name not in g["expected"]:
            continue
        t, fin, io = oracle.policy_sim(job, R, sizes, m, pol, src=src, fill=fill)
        e = g["expected"][name]
        assert t[0].tolist() == e["t"], name
        assert fin[0] == e["finish"] and io[0].tolist() == e["io"], name


def test_perfect_and_naive_closed_forms(oracle):
    job, sizes, out = _job_inputs(oracle)
    m = _model(oracle)
    R = out["R"]
    _, _, Mw = oracle.stream_shape(job)
    t0, fin0, io0 = oracle.policy_sim(job, R, sizes, m, oracle.PERFECT)
    t1, fin1, io1 = oracle.policy_sim(job, R, sizes, m, oracle.NAIVE)
    pfs = m.pfs_t / m.pfs_gamma
    for i in range(job.N):
        s = sizes[R[i, :Mw[i]]].astype(np.float64)
        u = s / m.c
        fetch = s / pfs
        write = np.maximum(s / m.beta, s / (m.w0 / m.p0))
        assert math.isclose(fin0[i], math.fsum(u), rel_tol=1e-12)
        assert np.allclose(t0[i, :Mw[i]], np.concatenate([[0.0], np.cumsum(u)[:-1]]), rtol=1e-12)
        assert math.isclose(fin1[i], math.fsum(fetch) + math.fsum(write) + math.fsum(u),
                            rel_tol=1e-12)
        assert (io0[i] == 0).all()
        assert math.isclose(io1[i, 0], math.fsum(fetch), rel_tol=1e-12) and (io1[i, 1:] == 0).all()
        assert (t0[i, Mw[i]:] == -1).all() and (t1[i, Mw[i]:] == -1).all()


@pytest.mark.parametrize("compute_bound", [True, False])
def test_equal_sizes_closed_form(oracle, compute_bound):
    F, E, N, B, d = 3_000, 3, 2, 4, 1
    job = oracle.make_job(F, E, N, B, d, 7)
    R = oracle.access_streams(job)
    _, _, Mw = oracle.stream_shape(job)
    S = 100_000
    sizes = np.full(F, S, np.int64)
    m = _model(oracle, c=(64e9 if not compute_bound else 64e6))
    rd = S / (m.pfs_t / m.pfs_gamma) + max(S / m.beta, S / (m.w0 / m.p0))
    u = S / m.c
    assert (u > rd / m.p0) == compute_bound
    for d0 in (0, S - 1, S, 3 * S, 40 * S, 10**15):
        fill = oracle.staging_schedule(job, R, sizes, d0)
        t, fin, _ = oracle.policy_sim(job, R, sizes, m, oracle.STAGING, fill=fill)
        for i in range(N):
            f = np.arange(Mw[i])
            want = rd / m.p0 + f * max(u, rd / m.p0)
            assert np.allclose(t[i, :Mw[i]], want, rtol=1e-12, atol=0), (d0, i)


def test_unlimited_buffer_is_the_fetch_model(oracle):
    job, sizes, out = _job_inputs(oracle)
    m = _model(oracle)
    R = out["R"]
    fill = oracle.staging_schedule(job, R, sizes, int(sizes.sum()) * job.E)
    assert (fill[fill >= 0] == 0).all()
    # no caches anywhere: every read from the PFS
    none = np.full_like(out["tier"], -1)
    src_p, t_p = oracle.fetch_model(job, R, none, sizes, m)
    assert (src_p[src_p >= 0] == 0).all()
    t, _, _ = oracle.policy_sim(job, R, sizes, m, oracle.STAGING, fill=fill)
    assert np.array_equal(t, t_p)
    # the plan's caches, with the fetch model's sources
    src, t_m = oracle.fetch_model(job, R, out["tier"], sizes, m)
    t, _, io = oracle.policy_sim(job, R, sizes, m, oracle.NOPFS, src=src, fill=fill)
    assert np.array_equal(t, t_m)
    assert (io[:, 1:] > 0).any()


def test_policy_order_and_capacity(oracle):
    job, sizes, out = _job_inputs(oracle, F=8_000, E=5, N=2, seed=9)
    m = _model(oracle, c=640e6)
    R = out["R"]
    src, _ = oracle.fetch_model(job, R, out["tier"], sizes, m)
    _, _, Mw = oracle.stream_shape(job)
    prev = None
    for d0 in (0, 500_000, 2_000_000, 20_000_000, 10**13):
        fill = oracle.staging_schedule(job, R, sizes, d0)
        tp, fp, _ = oracle.policy_sim(job, R, sizes, m, oracle.PERFECT)
        tn, fn, _ = oracle.policy_sim(job, R, sizes, m, oracle.NAIVE)
        ts, fs, _ = oracle.policy_sim(job, R, sizes, m, oracle.STAGING, fill=fill)
        tq, fq, io = oracle.policy_sim(job, R, sizes, m, oracle.NOPFS, src=src, fill=fill)
        for i in range(job.N):
            n = Mw[i]
            assert (tp[i, :n] <= tq[i, :n]).all() and (tq[i, :n] <= ts[i, :n]).all()
            assert (ts[i, :n] <= tn[i, :n]).all()
        assert (fp <= fq).all() and (fq <= fs).all() and (fs <= fn).all()
        if prev is not None:
            assert (ts <= prev[0]).all() and (tq <= prev[1]).all()  # a larger buffer never delays
        prev = (ts, tq)
    # the limit binds somewhere at the smallest buffers
    fill0 = oracle.staging_schedule(job, R, sizes, 0)
    fillinf = oracle.staging_schedule(job, R, sizes, 10**13)
    a, _, _ = oracle.policy_sim(job, R, sizes, m, oracle.STAGING, fill=fill0)
    b, _, _ = oracle.policy_sim(job, R, sizes, m, oracle.STAGING, fill=fillinf)
    assert (a > b).any()


def test_rows_match_full(oracle):
    job, sizes, out = _job_inputs(oracle, N=5, seed=11)
    m = _model(oracle)
    R = out["R"]
    src, _ = oracle.fetch_model(job, R, out["tier"], sizes, m)
    fill = oracle.staging_schedule(job, R, sizes, 3_000_000)
    t, fin, io = oracle.policy_sim(job, R, sizes, m, oracle.NOPFS, src=src, fill=fill)
    for i0, i1 in ((0, 1), (2, 5), (4, 5)):
        a, b, c = oracle.policy_sim(job, R[i0:i1], sizes, m, oracle.NOPFS, src=src[i0:i1],
                                    fill=fill[i0:i1], rows=(i0, i1))
        assert np.array_equal(a, t[i0:i1]) and np.array_equal(b, fin[i0:i1])
        assert np.array_equal(c, io[i0:i1])


def test_argument_errors(oracle):
    job = oracle.make_job(10, 2, 2, 1)
    R = oracle.access_streams(job)
    sizes = np.ones(10, np.int64)
    m = _model(oracle)
    with pytest.raises(Exception):
        oracle.policy_sim(job, R, sizes, m, 4)
    with pytest.raises(Exception):
        oracle.policy_sim(job, R, sizes, m, oracle.STAGING)  # no fill
    with pytest.raises(Exception):
        oracle.policy_sim(job, R, sizes, m, oracle.NOPFS, fill=np.zeros_like(R))  # no src
    bad = _model(oracle, p0=0.0)
    with pytest.raises(Exception):
        oracle.policy_sim(job, R, sizes, bad, oracle.PERFECT)
