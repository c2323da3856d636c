"""Pins for the oracle's performance model (Performance Modeling section):
the fetch source of every read and the time the worker consumes it,
t(f) = max(avail(f), t(f-1) + s(R[f-1]) / c).

 - hand-worked cases (tests/golden/fetch_model_example.json): the three
   sources, the preference on equal throughput, both bounds of the max;
 - closed forms for equal sizes from one source: t(f) = a + f*u when the
   staging buffer outruns compute (a = read/p0 <= u = s/c), (f+1)*a when it
   does not;
 - the recurrence unrolled, t(f) = max over g <= f of avail(g) plus the
   compute time of reads g..f-1, evaluated in exact rational arithmetic on
   variable sizes;
 - bounds and monotonicity on planned jobs: the last consumption lies
   between max(total compute, total read/p0) and their sum; faster compute,
   a faster network or more threads never delay any read.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from paper_2101_08734_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fetch_model_example.json")
LASSEN = dict(c=64e6, beta=200e6, b_c=24e9, pfs_t=2870e6, pfs_gamma=8, w0=111e9, p0=8,
              r=[85e9, 4e9], p=[4, 2])


def _model(oracle, **kw):
    d = dict(LASSEN)
    d.update(kw)
    return oracle.make_model(**d)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_hand_worked(oracle, case):
    j = case["job"]
    job = oracle.make_job(j["F"], j["E"], j["N"], j["B"], j["drop_last"], 1)
    m = oracle.make_model(**case["model"])
    src, t = oracle.fetch_model(job, np.array(case["R"], np.int32), np.array(case["tier"], np.int8),
                                np.array(case["sizes"], np.int64), m)
    np.testing.assert_array_equal(src, case["src"])
    np.testing.assert_allclose(t, case["t"], rtol=1e-14, atol=0)


def _stream(oracle, F, E, N, B, d, seed):
    job = oracle.make_job(F, E, N, B, d, seed)
    return job, oracle.access_streams(job)


@pytest.mark.parametrize("slow_compute", [False, True])
@pytest.mark.parametrize("placement", ["none", "own_ram"])
def test_equal_sizes_closed_form(oracle, slow_compute, placement):
    F, E, N, B = 3_000, 4, 3, 5
    job, R = _stream(oracle, F, E, N, B, 0, 4)
    s = 110_000
    sizes = np.full(F, s, np.int64)
    tier = np.full((N, F), -1, np.int8) if placement == "none" else np.zeros((N, F), np.int8)
    c = 1e6 if slow_compute else 64e9
    m = _model(oracle, c=c)
    src, t = oracle.fetch_model(job, R, tier, sizes, m)
    thr = 2870e6 / 8 if placement == "none" else 85e9 / 4
    read = s / thr + max(s / 200e6, s / (111e9 / 8))
    a, u = read / 8, s / c
    _, _, Mw = oracle.stream_shape(job)
    for i in range(N):
        f = np.arange(Mw[i], dtype=np.float64)
        want = a + f * u if a <= u else (f + 1) * a
        np.testing.assert_allclose(t[i, :Mw[i]], want, rtol=1e-9)
        assert (src[i, :Mw[i]] == (0 if placement == "none" else 256)).all()
        assert (src[i, Mw[i]:] == -1).all() and (t[i, Mw[i]:] == -1).all()


def test_unrolled_recurrence_exact(oracle):
    """Nothing cached (the PFS only), so a read's time is s (1/pfs + 1/write)
    with one known source; the oracle's t must equal the unrolled maximum."""
    F, E, N, B = 60, 3, 2, 2
    job, R = _stream(oracle, F, E, N, B, 1, 9)
    sizes = wl.random_sizes(F, 5, 1_000, 3_000_000)
    tier = np.full((N, F), -1, np.int8)
    prm = dict(c=3e6, beta=5e6, pfs_t=12e6, pfs_gamma=3, w0=2e7, p0=3)
    m = _model(oracle, **prm)
    src, t = oracle.fetch_model(job, R, tier, sizes, m)
    assert (src[src >= 0] == 0).all()
    Fr = Fraction
    pfs = Fr(prm["pfs_t"]) / Fr(prm["pfs_gamma"])
    wthr = min(Fr(prm["beta"]), Fr(prm["w0"]) / Fr(prm["p0"]))
    _, _, Mw = oracle.stream_shape(job)
    for i in range(N):
        s = [Fr(int(sizes[k])) for k in R[i, :Mw[i]]]
        read = [x / pfs + x / wthr for x in s]
        avail = [sum(read[:g + 1]) / Fr(prm["p0"]) for g in range(len(s))]
        for f in range(len(s)):
            want = max(avail[g] + sum(s[g:f]) / Fr(prm["c"]) for g in range(f + 1))
            assert abs(Fr(float(t[i, f])) - want) <= want * Fr(1, 10**12), (i, f)


def _planned(oracle, F, E, N, B, d, seed, fr):
    job = oracle.make_job(F, E, N, B, d, seed)
    sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
    caps = np.array([int(x * sizes.sum()) for x in fr], np.int64)
    out = oracle.full_pipeline(job, sizes, caps)
    return job, sizes, out


def test_bounds_on_planned_job(oracle):
    job, sizes, out = _planned(oracle, 20_000, 5, 4, 8, 0, 3, (0.05, 0.3))
    m = _model(oracle)
    src, t = oracle.fetch_model(job, out["R"], out["tier"], sizes, m)
    _, _, Mw = oracle.stream_shape(job)
    thr = {0: 2870e6 / 8, 128: min(24e9, 85e9 / 4), 129: min(24e9, 4e9 / 2), 256: 85e9 / 4,
           257: 4e9 / 2}
    for i in range(job.N):
        k = out["R"][i, :Mw[i]]
        s = sizes[k].astype(np.float64)
        codes = src[i, :Mw[i]]
        read = s / np.array([thr[int(x)] for x in codes]) + np.maximum(s / 200e6, s / (111e9 / 8))
        io = read.sum() / 8
        comp = s[:-1].sum() / 64e6
        last = t[i, Mw[i] - 1]
        assert last >= max(io, comp + read[0] / 8) * (1 - 1e-12)
        assert last <= (io + comp) * (1 + 1e-12)
        # consecutive consumptions are at least one sample's compute apart
        # (up to the rounding of t itself)
        assert (np.diff(t[i, :Mw[i]]) >= s[:-1] / 64e6 - 1e-12 * last).all()
        # a source is only chosen where it exists
        own = out["tier"][i, k]
        loc = codes >= 256
        assert (own[loc] == codes[loc] - 256).all()
        rem = (codes >= 128) & (codes < 256)
        for kk, cc in zip(k[rem], codes[rem]):
            holders = np.nonzero(out["tier"][:, kk] == cc - 128)[0]
            assert len(holders[holders != i]) > 0


@pytest.mark.parametrize("change", [dict(c=128e6), dict(b_c=48e9), dict(p0=16, w0=222e9),
                                    dict(r=[170e9, 8e9]), dict(pfs_t=5740e6)])
def test_faster_resources_never_delay(oracle, change):
    job, sizes, out = _planned(oracle, 8_000, 4, 3, 8, 1, 5, (0.1, 0.2))
    _, t0 = oracle.fetch_model(job, out["R"], out["tier"], sizes, _model(oracle))
    _, t1 = oracle.fetch_model(job, out["R"], out["tier"], sizes, _model(oracle, **change))
    valid = t0 >= 0
    assert (t1[valid] <= t0[valid] * (1 + 1e-12)).all()


def test_caching_never_delays(oracle):
    """Adding cached copies only adds faster sources."""
    job, sizes, out = _planned(oracle, 8_000, 4, 3, 8, 1, 6, (0.1, 0.2))
    none = np.full_like(out["tier"], -1)
    _, t_none = oracle.fetch_model(job, out["R"], none, sizes, _model(oracle))
    _, t_plan = oracle.fetch_model(job, out["R"], out["tier"], sizes, _model(oracle))
    valid = t_none >= 0
    assert (t_plan[valid] <= t_none[valid] * (1 + 1e-12)).all()
    assert t_plan[valid].sum() < t_none[valid].sum()


def test_rows_match_full(oracle):
    job, sizes, out = _planned(oracle, 5_000, 3, 5, 4, 0, 8, (0.1, 0.3))
    m = _model(oracle)
    src, t = oracle.fetch_model(job, out["R"], out["tier"], sizes, m)
    s2, t2 = oracle.fetch_model(job, out["R"][2:4], out["tier"], sizes, m, rows=(2, 4))
    np.testing.assert_array_equal(s2, src[2:4])
    np.testing.assert_array_equal(t2, t[2:4])


@pytest.mark.parametrize("bad", [dict(c=0), dict(beta=-1), dict(p0=float("nan")),
                                 dict(b_c=float("inf")), dict(r=[]), dict(r=[1e9] * 33, p=[1] * 33),
                                 dict(p=[4, 0])])
def test_invalid_model(oracle, bad):
    job, R = _stream(oracle, 20, 2, 2, 2, 1, 1)
    tier = np.full((2, 20), -1, np.int8)
    d = dict(LASSEN)
    d.update(bad)
    m = oracle.RefModel()
    m.c, m.beta, m.b_c, m.pfs_t, m.pfs_gamma, m.w0, m.p0 = (d["c"], d["beta"], d["b_c"], d["pfs_t"],
                                                           d["pfs_gamma"], d["w0"], d["p0"])
    m.J = len(d["r"])
    for j in range(min(m.J, 32)):
        m.r[j], m.p[j] = d["r"][j], d["p"][j]
    with pytest.raises(Exception):
        oracle.fetch_model(job, R, tier, np.ones(20, np.int64), m)
