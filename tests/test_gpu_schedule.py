"""Prefetch queues and staging schedule on the GPU vs the CPU oracle.

Stage isolation: R and tier (and, for the oracle, first) are the oracle's
own (streams, stats and plan on the host), so a mismatch names these two
entry points. Comparisons
are element by element (all integer work). Sizes span many 2048-position
prefetch chunks and 4096-position staging chunks with ragged tails; edge
cases cover empty streams, rows of different lengths (drop_last=0), more
workers than samples, J below and above the placement's tier count,
a tier table at an odd address, buffers from 0
bytes to more than a worker reads, and the staging search's global-memory
path. At ImageNet-1k size the oracle runs in full; at ImageNet-22k size the
outputs are checked on the device by the properties that define them.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2101_08734_amd import nopfs  # noqa: E402
from paper_2101_08734_amd import workloads as wl  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nopfs.lib()
    yield
    nopfs.debug_set(4, 0)
    nopfs.debug_set(5, 0)
    torch.cuda.empty_cache()


JOBS = [
    # name, F, E, N, B, drop_last, seed, caps as fractions of the total size
    ("small", 10_000, 5, 4, 16, 1, 42, (0.004, 0.02)),
    ("ragged", 30_011, 5, 3, 7, 0, 3, (0.05, 0.2)),
    ("medium", 150_000, 7, 8, 16, 1, 9, (0.02, 0.1, 0.3)),
    ("many_epochs", 2_000, 60, 16, 1, 0, 11, (0.1, 0.5)),
    ("e255", 700, 255, 5, 3, 1, 12, (0.05, 0.25)),
    ("wide", 20_000, 3, 300, 2, 1, 13, (0.3,)),
    ("n_gt_f", 50, 4, 64, 1, 0, 14, (0.5, 0.5)),
    ("one_sample", 1, 3, 1, 1, 1, 15, (0.0, 1.0)),
    ("one_worker", 40_000, 4, 1, 64, 1, 16, (0.25, 0.25)),
    ("zero_iters", 10, 2, 4, 3, 1, 17, (0.5,)),
    ("long_rows", 400_000, 2, 2, 1000, 0, 18, (0.01, 0.6)),
]
IDS = [j[0] for j in JOBS]


def _oracle_inputs(oracle, F, E, N, B, d, seed, fr):
    sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
    tot = int(sizes.sum())
    caps = np.array([int(f * tot) for f in fr], np.int64)
    job = oracle.make_job(F, E, N, B, d, seed)
    out = oracle.full_pipeline(job, sizes, caps)
    return job, sizes, caps, out


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _equal(name, got, exp):
    got = got.cpu().numpy() if isinstance(got, torch.Tensor) else got
    assert got.shape == exp.shape, (name, got.shape, exp.shape)
    if not np.array_equal(got, exp):
        bad = np.argwhere(got != exp)
        raise AssertionError(f"{name}: {len(bad)} mismatches, first at {bad[:5].tolist()} "
                             f"got {got[tuple(bad[0])]} expected {exp[tuple(bad[0])]}")


def _d0s(sizes, R, N):
    tot = int(sizes.sum())
    mx = int(sizes.max())
    med = int(np.median(sizes))
    return [0, 1, mx - 1, mx, 3 * med, 40 * med, tot // max(N, 1), 50 * tot]


@pytest.mark.parametrize("name,F,E,N,B,d,seed,fr", JOBS, ids=IDS)
def test_prefetch_order_matches_oracle(oracle, name, F, E, N, B, d, seed, fr):
    rjob, sizes, caps, out = _oracle_inputs(oracle, F, E, N, B, d, seed, fr)
    job = nopfs.Job(F, E, N, B, d, seed)
    R, tier = _dev(out["R"]), _dev(out["tier"])
    for J in sorted({1, len(caps), len(caps) + 2}):
        order, qlen = nopfs.prefetch_order(job, R, tier, J)
        torch.cuda.synchronize()
        eo, eq = oracle.prefetch_order(rjob, out["R"], out["first"], out["tier"], J)
        _equal(f"order J={J}", order, eo)
        _equal(f"qlen J={J}", qlen, eq)


@pytest.mark.parametrize("name,F,E,N,B,d,seed,fr", JOBS, ids=IDS)
def test_staging_schedule_matches_oracle(oracle, name, F, E, N, B, d, seed, fr):
    rjob, sizes, caps, out = _oracle_inputs(oracle, F, E, N, B, d, seed, fr)
    job = nopfs.Job(F, E, N, B, d, seed)
    R, s = _dev(out["R"]), _dev(sizes)
    for d0 in _d0s(sizes, out["R"], N):
        fill = nopfs.staging_schedule(job, R, s, d0)
        torch.cuda.synchronize()
        _equal(f"fill d0={d0}", fill, oracle.staging_schedule(rjob, out["R"], sizes, d0))


@pytest.mark.parametrize("gcap", [1, 16, 700])
@pytest.mark.parametrize("name,F,E,N,B,d,seed,fr", [JOBS[1], JOBS[2], JOBS[10]],
                         ids=[JOBS[1][0], JOBS[2][0], JOBS[10][0]])
def test_staging_global_search_path(oracle, name, F, E, N, B, d, seed, fr, gcap):
    """Chunks whose range of buffer starts exceeds the LDS capacity search the
    row in global memory; a tiny capacity sends most chunks there."""
    rjob, sizes, caps, out = _oracle_inputs(oracle, F, E, N, B, d, seed, fr)
    job = nopfs.Job(F, E, N, B, d, seed)
    R, s = _dev(out["R"]), _dev(sizes)
    nopfs.debug_set(4, gcap)
    try:
        for d0 in _d0s(sizes, out["R"], N):
            fill = nopfs.staging_schedule(job, R, s, d0)
            torch.cuda.synchronize()
            _equal(f"fill d0={d0}", fill, oracle.staging_schedule(rjob, out["R"], sizes, d0))
    finally:
        nopfs.debug_set(4, 0)


@pytest.mark.parametrize("widen", [1, 2, 4])
@pytest.mark.parametrize("name,F,E,N,B,d,seed,fr", [JOBS[1], JOBS[2], JOBS[10]],
                         ids=[JOBS[1][0], JOBS[2][0], JOBS[10][0]])
def test_staging_wide_windows(oracle, name, F, E, N, B, d, seed, fr, widen):
    """Sample windows widened by the test hook (2^15 to 2^18 samples): each
    window tile covers its window in 2 to 16 LDS passes, the path of jobs
    above 2^27 samples."""
    rjob, sizes, caps, out = _oracle_inputs(oracle, F, E, N, B, d, seed, fr)
    job = nopfs.Job(F, E, N, B, d, seed)
    R, s = _dev(out["R"]), _dev(sizes)
    nopfs.debug_set(5, widen)
    try:
        for d0 in _d0s(sizes, out["R"], N):
            fill = nopfs.staging_schedule(job, R, s, d0)
            torch.cuda.synchronize()
            _equal(f"fill d0={d0} widen={widen}", fill,
                   oracle.staging_schedule(rjob, out["R"], sizes, d0))
    finally:
        nopfs.debug_set(5, 0)


def test_staging_heavy_tailed_sizes(oracle):
    """Mostly 1-byte samples and a few of a megabyte: the bytes of one chunk
    can span far more positions elsewhere, so some chunks typically exceed
    the LDS range without any test hook."""
    F, E, N, B, d, seed = 200_000, 4, 2, 50, 0, 21
    rng = np.random.default_rng(5)
    sizes = np.where(rng.random(F) < 0.002, 1_000_000, 1).astype(np.int64)
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(rjob)
    job = nopfs.Job(F, E, N, B, d, seed)
    for d0 in (0, 999_999, 1_000_000, 3_000_000, 20_000, 10_000_000):
        fill = nopfs.staging_schedule(job, _dev(R), _dev(sizes), d0)
        torch.cuda.synchronize()
        _equal(f"fill d0={d0}", fill, oracle.staging_schedule(rjob, R, sizes, d0))


@pytest.mark.parametrize("frac", [0.0005, 1.0])
def test_staging_sizes_beyond_32_bits(oracle, frac):
    """Sizes of 2^32 bytes and more (a share `frac` of the samples, the rest
    as usual) make the staging passes carry 8-byte sizes instead of 4-byte
    ones; the schedule must not depend on which."""
    F, E, N, B, d, seed = 60_000, 4, 3, 16, 0, 23
    rng = np.random.default_rng(7)
    sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
    big = rng.random(F) < frac
    sizes = np.where(big, (1 << 32) + rng.integers(0, 1 << 34, F), sizes).astype(np.int64)
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(rjob)
    job = nopfs.Job(F, E, N, B, d, seed)
    for d0 in _d0s(sizes, R, N) + [(1 << 32) - 1, 1 << 32, 5 << 32]:
        fill = nopfs.staging_schedule(job, _dev(R), _dev(sizes), d0)
        torch.cuda.synchronize()
        _equal(f"fill d0={d0}", fill, oracle.staging_schedule(rjob, R, sizes, d0))


def test_staging_span_sums_of_both_widths(oracle):
    """Sizes around 2^32 / 2^14 bytes: within one row, some spans of 16,384
    positions hold 2^32 bytes or more (their prefix sums are kept as 8-byte
    values) and others less (4-byte values). Buffers larger than a span's
    bytes make windows that reach across spans of both kinds; the staged
    search and the global-memory search must both agree with the oracle."""
    F, E, N, B, d, seed = 30_000, 10, 4, 8, 0, 27
    rng = np.random.default_rng(11)
    sizes = rng.integers(229_500, 294_500, F).astype(np.int64)
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(rjob)
    job = nopfs.Job(F, E, N, B, d, seed)
    _, M, Mw = nopfs.stream_shape(job)
    kinds = set()
    for i in range(N):
        for c in range(Mw[i] // 16384):
            kinds.add(int(sizes[R[i, c * 16384:(c + 1) * 16384]].sum()) >= 1 << 32)
    assert kinds == {False, True}, "the sizes must give spans of both widths"
    try:
        for gcap in (0, 64):
            nopfs.debug_set(4, gcap)
            for d0 in (0, 1_000_000_000, 5_000_000_000, 1 << 32, 12_000_000_000):
                fill = nopfs.staging_schedule(job, _dev(R), _dev(sizes), d0)
                torch.cuda.synchronize()
                _equal(f"fill gcap={gcap} d0={d0}", fill, oracle.staging_schedule(rjob, R, sizes, d0))
    finally:
        nopfs.debug_set(4, 0)


def test_equal_sizes_closed_form(oracle):
    """Equal sizes s and a buffer of m*s bytes: fill(h) = max(0, h - m + 1)."""
    F, E, N, B = 50_000, 3, 4, 8
    rjob = oracle.make_job(F, E, N, B, 0, 9)
    R = oracle.access_streams(rjob)
    job = nopfs.Job(F, E, N, B, 0, 9)
    s = 16_777_216
    sizes = np.full(F, s, np.int64)
    _, M, Mw = nopfs.stream_shape(job)
    for m in (1, 2, 4095, 4097, 9000):
        fill = nopfs.staging_schedule(job, _dev(R), _dev(sizes), m * s).cpu().numpy()
        for i in range(N):
            np.testing.assert_array_equal(fill[i][:Mw[i]], np.maximum(0, np.arange(Mw[i]) - m + 1))
            assert (fill[i][Mw[i]:] == -1).all()


def test_prefetch_arbitrary_placement(oracle):
    """Any placement (tiers outside [0, J) included) over valid first reads."""
    F, E, N, B, d, seed = 60_000, 6, 3, 10, 0, 23
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(rjob)
    count, first = oracle.access_stats(rjob, R)
    rng = np.random.default_rng(3)
    tier = rng.integers(-3, 9, size=(N, F)).astype(np.int8)
    job = nopfs.Job(F, E, N, B, d, seed)
    for J in (1, 4, 6, 127):
        order, qlen = nopfs.prefetch_order(job, _dev(R), _dev(tier), J)
        torch.cuda.synchronize()
        eo, eq = oracle.prefetch_order(rjob, R, first, tier, J)
        _equal(f"order J={J}", order, eo)
        _equal(f"qlen J={J}", qlen, eq)


def test_prefetch_tier_view_with_offset(oracle):
    """A tier table that starts at an odd address (a view into a larger
    buffer) is read like any other."""
    rjob, sizes, caps, out = _oracle_inputs(oracle, *JOBS[1][1:])
    F, N = JOBS[1][1], JOBS[1][3]
    job = nopfs.Job(*JOBS[1][1:7])
    tbuf = torch.empty(N * F + 4, dtype=torch.int8, device="cuda")
    tier = tbuf[3:3 + N * F].view(N, F)
    assert tier.data_ptr() % 4 != 0
    tier.copy_(_dev(out["tier"]))
    order, qlen = nopfs.prefetch_order(job, _dev(out["R"]), tier, len(caps))
    torch.cuda.synchronize()
    eo, eq = oracle.prefetch_order(rjob, out["R"], out["first"], out["tier"], len(caps))
    _equal("order", order, eo)
    _equal("qlen", qlen, eq)


def test_outputs_fully_written():
    """Every element is written (poisoned buffers; a zero-iteration job
    still writes its queue lengths)."""
    job = nopfs.Job(10, 2, 4, 3, 1, 17)  # T = 0, M_max = 0
    R = torch.empty((4, 0), dtype=torch.int32, device="cuda")
    tier = torch.zeros((4, 10), dtype=torch.int8, device="cuda")
    qlen = torch.full((4, 2), 77, dtype=torch.int64, device="cuda")
    order, qlen = nopfs.prefetch_order(job, R, tier, 2, qlen=qlen)
    torch.cuda.synchronize()
    assert order.shape == (4, 0) and int(qlen.abs().sum()) == 0


# ---------------------------------------------------------------- full size --
def test_imagenet1k_full(oracle, imagenet1k_expected):
    w = wl.WORKLOADS["imagenet1k"]
    rjob = oracle.make_job(*w.job_tuple())
    sizes = wl.sizes(w)
    out = imagenet1k_expected
    job = nopfs.Job(*w.job_tuple())
    R, tier = _dev(out["R"]), _dev(out["tier"])
    J = len(w.caps)
    order, qlen = nopfs.prefetch_order(job, R, tier, J)
    fill = nopfs.staging_schedule(job, R, _dev(sizes), int(w.staging))
    torch.cuda.synchronize()
    eo, eq = oracle.prefetch_order(rjob, out["R"], out["first"], out["tier"], J)
    _equal("order", order, eo)
    _equal("qlen", qlen, eq)
    _equal("fill", fill, oracle.staging_schedule(rjob, out["R"], sizes, int(w.staging)))


def check_prefetch_properties(job, R, first, tier, J, order, qlen, rows):
    """Queue j of row i lists exactly the samples with tier j and a first
    read, by strictly increasing first read; -1 after the queues."""
    _, M, Mw = nopfs.stream_shape(job)
    for i in rows:
        read = first[i] >= 0
        start = 0
        for j in range(J):
            n = int(qlen[i, j])
            want = read & (tier[i] == j)
            assert n == int(want.sum()), (i, j)
            q = order[i, start:start + n].to(torch.int64)
            if n == 0:
                continue
            assert int(q.min()) >= 0 and int(q.max()) < job.F
            assert bool((tier[i][q] == j).all())
            fq = first[i][q]
            assert bool((fq >= 0).all()) and bool((fq[1:] > fq[:-1]).all())
            assert bool((R[i][fq.to(torch.int64)] == q.to(torch.int32)).all())
            start += n
        assert bool((order[i, start:] == -1).all())


def check_staging_properties(job, R, sizes, d0, fill, rows):
    """fill[h] = f is the smallest start whose window f..h fits d0 bytes (or h
    when the sample alone does not fit); -1 in padding."""
    _, M, Mw = nopfs.stream_shape(job)
    for i in rows:
        m = Mw[i]
        f = fill[i, :m].to(torch.int64)
        assert bool((fill[i, m:] == -1).all())
        h = torch.arange(m, device=f.device)
        assert bool((f >= 0).all()) and bool((f <= h).all())
        sz = sizes[R[i, :m].to(torch.int64)]
        P = torch.cat([torch.zeros(1, dtype=torch.int64, device=f.device), torch.cumsum(sz, 0)])
        win = P[h + 1] - P[f]                     # bytes of positions f..h
        assert bool(((win <= d0) | (f == h)).all())
        g = (f - 1).clamp(min=0)
        wider = P[h + 1] - P[g]                   # bytes of positions f-1..h
        assert bool(((f == 0) | (wider > d0)).all())
        assert bool((f[1:] >= f[:-1]).all())


def test_imagenet22k_properties():
    w = wl.WORKLOADS["imagenet22k"]
    job = nopfs.Job(*w.job_tuple())
    sizes = torch.from_numpy(wl.sizes(w)).cuda()
    out = nopfs.plan_job(job, sizes, wl.caps(w))
    del out["count"], out["next"]
    torch.cuda.empty_cache()
    J = len(w.caps)
    order, qlen = nopfs.prefetch_order(job, out["R"], out["tier"], J)
    torch.cuda.synchronize()
    rows = [0, 1, 77, 131, 255]
    check_prefetch_properties(job, out["R"], out["first"], out["tier"], J, order, qlen.cpu(), rows)
    del order, qlen
    for d0 in (int(w.staging), 1_000_000, 0):
        fill = nopfs.staging_schedule(job, out["R"], sizes, d0)
        torch.cuda.synchronize()
        check_staging_properties(job, out["R"], sizes, d0, fill, rows)
        del fill
    del out
    torch.cuda.empty_cache()
