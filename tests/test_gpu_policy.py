"""Policy simulation on the GPU vs the CPU oracle.

Stage isolation: R, the fetch sources and the staging schedule are the
oracle's own (streams, plan, fetch model and staging schedule on the host).
Both sides evaluate the same recurrence read by read with the same IEEE
double operations in the same order, so consumption times, finish times and
the fetch time per source class must be identical, bit for bit.

Cases: the four policies on ten job shapes (ragged rows, one worker, more
workers than samples, 255 epochs) at five buffer sizes, from one holding no
sample (every read waits for the previous consumption) to one holding the
stream (no wait), including windows longer than the kernel's 8,192-position
LDS ring; compute- and I/O-bound parameters and non-power-of-two thread
counts; 32 tiers with arbitrary source codes (invalid codes read from the
PFS) and arbitrary windows (out-of-range ones clamped as the oracle does);
an empty job; two calls in a row; ImageNet-1k in full; and at the
ImageNet-22k shape, seeded random epoch permutations and placements, with
sources and windows from the product's own stages for the GPU and from the
oracle (sources) and the schedule's definition (windows) for three sampled
workers, which must match before the oracle replays them.
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
    ("long_rows", 400_000, 2, 2, 1000, 0, 18, (0.01, 0.6)),
]
IDS = [j[0] for j in JOBS]
# buffer as a fraction of the bytes one worker reads in an epoch
D0_FRACTIONS = [0.0, 0.01, 0.2, 0.9, 10.0]
POLICIES = (nopfs.POLICY_PERFECT, nopfs.POLICY_NAIVE, nopfs.POLICY_STAGING, nopfs.POLICY_NOPFS)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _params(J, **kw):
    d = dict(wl.LASSEN_MODEL)
    d["r"] = (list(d["r"]) + [1e9] * J)[:J]
    d["p"] = (list(d["p"]) + [1] * J)[:J]
    d.update(kw)
    return d


def _compare(name, got, want):
    for what, g, w in zip(("t", "finish", "io"), got, want):
        g = g.cpu().numpy()
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)
            raise AssertionError(f"{name} {what}: {len(bad)} mismatches, first {bad[:3].tolist()} "
                                 f"got {g[tuple(bad[0])]!r} expected {w[tuple(bad[0])]!r}")


def _run_all(oracle, name, rjob, job, R, sizes, src, fill, prm):
    m_o, m_g = oracle.make_model(**prm), nopfs.make_model(**prm)
    Rd, sd, srcd, filld = _dev(R), _dev(sizes), _dev(src), _dev(fill)
    for pol in POLICIES:
        want = oracle.policy_sim(rjob, R, sizes, m_o, pol, src=src, fill=fill)
        got = nopfs.policy_sim(job, Rd, sd, m_g, pol, src=srcd, fill=filld)
        torch.cuda.synchronize()
        _compare(f"{name} policy {pol}", got, want)


@pytest.mark.parametrize("name,F,E,N,B,d,seed,fr", JOBS, ids=IDS)
def test_matches_oracle(oracle, name, F, E, N, B, d, seed, fr):
    rjob = oracle.make_job(F, E, N, B, d, seed)
    sizes = wl.random_sizes(F, seed + 1, 1_000, 2_000_000)
    tot = int(sizes.sum())
    out = oracle.full_pipeline(rjob, sizes, np.array([int(f * tot) for f in fr], np.int64))
    prm = _params(len(fr))
    src, _ = oracle.fetch_model(rjob, out["R"], out["tier"], sizes, oracle.make_model(**prm))
    job = nopfs.Job(F, E, N, B, d, seed)
    for f0 in D0_FRACTIONS:
        d0 = int(f0 * tot / N)
        fill = oracle.staging_schedule(rjob, out["R"], sizes, d0)
        _run_all(oracle, f"{name} d0={d0}", rjob, job, out["R"], sizes, src, fill, prm)


REGIMES = {
    "io_bound": dict(c=64e9),
    "compute_bound": dict(c=16e6),
    "p0_3": dict(p0=3, w0=7e9),
    "one_thread": dict(p0=1, w0=1e9),
    "slow_network": dict(b_c=1e6),
}


@pytest.mark.parametrize("regime", list(REGIMES))
def test_parameter_regimes(oracle, regime):
    F, E, N, B, d, seed = 30_011, 5, 3, 7, 0, 3
    rjob = oracle.make_job(F, E, N, B, d, seed)
    sizes = wl.random_sizes(F, 4, 1_000, 2_000_000)
    tot = int(sizes.sum())
    out = oracle.full_pipeline(rjob, sizes, np.array([int(0.05 * tot), int(0.2 * tot)], np.int64))
    prm = _params(2, **REGIMES[regime])
    src, _ = oracle.fetch_model(rjob, out["R"], out["tier"], sizes, oracle.make_model(**prm))
    fill = oracle.staging_schedule(rjob, out["R"], sizes, int(0.3 * tot / N))
    _run_all(oracle, regime, rjob, nopfs.Job(F, E, N, B, d, seed), out["R"], sizes, src, fill, prm)


def test_arbitrary_sources_and_windows(oracle):
    """32 tiers (65 source classes), any source code and any window."""
    F, E, N, B, d, seed = 20_000, 5, 4, 10, 0, 23
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(rjob)
    _, M, _ = oracle.stream_shape(rjob)
    rng = np.random.default_rng(5)
    codes = np.concatenate([[0, -1, 1, 127, 300, 288], 128 + np.arange(32), 256 + np.arange(32)])
    src = rng.choice(codes, size=(N, M)).astype(np.int16)
    fill = rng.integers(-5, M + 5, size=(N, M)).astype(np.int32)
    sizes = wl.random_sizes(F, 7, 1, 5_000_000)
    prm = dict(wl.LASSEN_MODEL)
    prm["r"] = [float(x) for x in rng.uniform(1e9, 1e11, 32)]
    prm["p"] = [float(x) for x in rng.integers(1, 9, 32)]
    _run_all(oracle, "arbitrary", rjob, nopfs.Job(F, E, N, B, d, seed), R, sizes, src, fill, prm)


def test_zero_iterations():
    job = nopfs.Job(10, 2, 4, 3, 1, 17)  # T = 0, M_max = 0
    R = torch.empty((4, 0), dtype=torch.int32, device="cuda")
    sizes = torch.ones(10, dtype=torch.int64, device="cuda")
    fill = torch.empty((4, 0), dtype=torch.int32, device="cuda")
    src = torch.empty((4, 0), dtype=torch.int16, device="cuda")
    m = nopfs.make_model(**wl.LASSEN_MODEL)
    for pol in POLICIES:
        t, fin, io = nopfs.policy_sim(job, R, sizes, m, pol, src=src, fill=fill)
        torch.cuda.synchronize()
        assert t.shape == (4, 0)
        assert (fin.cpu().numpy() == 0).all() and (io.cpu().numpy() == 0).all()


def test_repeat_calls(oracle):
    """Two calls in a row, the second on a smaller job."""
    outs = []
    for F, N in ((50_000, 4), (7_000, 2)):
        rjob = oracle.make_job(F, 6, N, 8, 0, 40)
        sizes = wl.random_sizes(F, 41, 1_000, 2_000_000)
        R = oracle.access_streams(rjob)
        fill = oracle.staging_schedule(rjob, R, sizes, int(0.3 * sizes.sum() / N))
        src = np.zeros_like(R, dtype=np.int16)
        prm = _params(2)
        want = oracle.policy_sim(rjob, R, sizes, oracle.make_model(**prm), nopfs.POLICY_STAGING,
                                 fill=fill)
        got = nopfs.policy_sim(nopfs.Job(F, 6, N, 8, 0, 40), _dev(R), _dev(sizes),
                               nopfs.make_model(**prm), nopfs.POLICY_STAGING, src=_dev(src),
                               fill=_dev(fill))
        torch.cuda.synchronize()
        outs.append((got, want))
    for k, (got, want) in enumerate(outs):
        _compare(f"call {k}", got, want)


def test_imagenet1k_full(oracle, imagenet1k_expected):
    w = wl.WORKLOADS["imagenet1k"]
    rjob = oracle.make_job(*w.job_tuple())
    sizes = wl.sizes(w)
    out = imagenet1k_expected
    prm = dict(wl.LASSEN_MODEL)
    src, _ = oracle.fetch_model(rjob, out["R"], out["tier"], sizes, oracle.make_model(**prm))
    fill = oracle.staging_schedule(rjob, out["R"], sizes, int(w.staging))
    job = nopfs.Job(*w.job_tuple())
    m_o, m_g = oracle.make_model(**prm), nopfs.make_model(**prm)
    Rd, sd, srcd, filld = _dev(out["R"]), _dev(sizes), _dev(src), _dev(fill)
    for pol in (nopfs.POLICY_STAGING, nopfs.POLICY_NOPFS):
        want = oracle.policy_sim(rjob, out["R"], sizes, m_o, pol, src=src, fill=fill)
        got = nopfs.policy_sim(job, Rd, sd, m_g, pol, src=srcd, fill=filld)
        torch.cuda.synchronize()
        _compare(f"imagenet1k policy {pol}", got, want)


def test_imagenet22k_sampled_rows(oracle):
    """The benchmarked shape (14.2M samples, 256 workers, 40 epochs): each
    epoch a seeded random permutation split across the workers as the
    streams are, a seeded random placement; sources and windows from the
    product's own stages, checked against the oracle's on three sampled
    workers, whose policies the oracle then replays."""
    w = wl.WORKLOADS["imagenet22k"]
    job = nopfs.Job(*w.job_tuple())
    _, M, Mw = nopfs.stream_shape(job)
    L = M // w.E
    assert (np.asarray(Mw) == M).all() and L * w.E == M
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2223)
    R = torch.empty((w.N, M), dtype=torch.int32, device="cuda")
    for e in range(w.E):
        perm = torch.randperm(w.F, generator=gen, device="cuda", dtype=torch.int64)
        R[:, e * L:(e + 1) * L] = perm[:w.N * L].view(L, w.N).t().to(torch.int32)
        del perm
    tier = torch.randint(-1, 2, (w.N, w.F), generator=gen, device="cuda", dtype=torch.int8)
    sizes_h = wl.sizes(w)
    sizes = _dev(sizes_h)
    prm = dict(wl.LASSEN_MODEL)
    m_g = nopfs.make_model(**prm)
    src, _ = nopfs.fetch_model(job, R, tier, sizes, m_g)
    fill = torch.empty((w.N, M), dtype=torch.int32, device="cuda")
    nopfs.staging_schedule(job, R, sizes, int(w.staging), fill)
    got = {pol: nopfs.policy_sim(job, R, sizes, m_g, pol, src=src, fill=fill)
           for pol in (nopfs.POLICY_STAGING, nopfs.POLICY_NOPFS)}
    torch.cuda.synchronize()
    rjob = oracle.make_job(*w.job_tuple())
    m_o = oracle.make_model(**prm)
    tier_h = tier.cpu().numpy()
    del tier
    for i in (0, 131, 255):
        Ri = R[i:i + 1].cpu().numpy()
        src_o, _ = oracle.fetch_model(rjob, Ri, tier_h, sizes_h, m_o, rows=(i, i + 1))
        assert np.array_equal(src_o, src[i:i + 1].cpu().numpy()), i
        # the row's staging schedule from its definition (the smallest start
        # whose window of sizes fits d0), on the host; the product's must match
        s = sizes_h[Ri[0]]
        S = np.concatenate([[0], np.cumsum(s)])
        h = np.arange(M)
        lo = np.searchsorted(S, S[h + 1] - int(w.staging), side="left")
        fill_o = np.minimum(lo, h).astype(np.int32)[None]
        assert np.array_equal(fill[i:i + 1].cpu().numpy(), fill_o), i
        for pol in (nopfs.POLICY_STAGING, nopfs.POLICY_NOPFS):
            want = oracle.policy_sim(rjob, Ri, sizes_h, m_o, pol, src=src_o, fill=fill_o,
                                     rows=(i, i + 1))
            g = got[pol]
            _compare(f"imagenet22k row {i} policy {pol}", (g[0][i:i + 1], g[1][i:i + 1],
                                                           g[2][i:i + 1]), want)
    del R, src, fill, got
    torch.cuda.empty_cache()
