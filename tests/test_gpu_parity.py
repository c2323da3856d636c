"""GPU path vs the CPU oracle, element by element (bit-exact: all of this is
integer work). Sizes span several tiles and buckets with ragged tails; edge
cases cover empty streams, one sample, more workers than samples, the
largest epoch count, drop_last=0 padding, zero and unbounded capacities.
Each stage is also fed the oracle's own inputs (stage isolation), so a
failure names the stage that is wrong."""
import numpy as np
import pytest

import invariants as inv

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
    for which in (1, 2, 3):
        nopfs.debug_set(which, 0)


PATHS = ["staged", "fused"]  # four stage calls, or nopfs_plan_job


def gpu_pipeline(job, sizes, caps, path="staged"):
    s = torch.from_numpy(sizes).cuda()
    out = nopfs.plan(job, s, caps) if path == "staged" else nopfs.plan_job(job, s, caps)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def compare(got, exp, names=("R", "count", "first", "next", "tier", "used")):
    for n in names:
        g, e = got[n], exp[n]
        assert g.shape == e.shape, (n, g.shape, e.shape)
        if not np.array_equal(g, e):
            bad = np.argwhere(g != e)
            raise AssertionError(f"{n}: {len(bad)} mismatches, first at {bad[:5].tolist()} "
                                 f"got {g[tuple(bad[0])]} expected {e[tuple(bad[0])]}")


JOBS = [
    # F, E, N, B, drop_last, seed, caps as fractions of the total size
    ("small", 10_000, 5, 4, 16, 1, 42, None),
    ("ragged", 30_011, 5, 3, 7, 0, 3, (0.05, 0.2)),
    ("medium", 150_000, 7, 8, 16, 1, 9, (0.02, 0.1, 0.3)),
    ("many_epochs", 2_000, 60, 16, 1, 0, 11, (0.1, 0.5)),
    ("e255", 700, 255, 5, 3, 1, 12, (0.05, 0.25)),
    ("wide", 20_000, 3, 300, 2, 1, 13, (0.3,)),
    ("n_gt_f", 50, 4, 64, 1, 0, 14, (0.5, 0.5)),
    ("one_sample", 1, 3, 1, 1, 1, 15, (0.0, 1.0)),
    ("one_worker", 40_000, 4, 1, 64, 1, 16, (0.25, 0.25)),
    ("zero_iters", 10, 2, 4, 3, 1, 17, (0.5,)),
    ("big_bucket_count", 400_000, 2, 2, 1000, 0, 18, (0.01, 0.6)),
]


def _caps(sizes, fracs):
    tot = int(sizes.sum())
    return np.array([int(f * tot) for f in fracs], np.int64)


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("name,F,E,N,B,d,seed,fr", JOBS, ids=[j[0] for j in JOBS])
def test_pipeline_matches_oracle(oracle, name, F, E, N, B, d, seed, fr, path):
    if name == "small":
        w = wl.WORKLOADS["small"]
        sizes, caps = wl.sizes(w), wl.caps(w)
    else:
        sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
        caps = _caps(sizes, fr)
    job = nopfs.Job(F, E, N, B, d, seed)
    got = gpu_pipeline(job, sizes, caps, path)
    exp = oracle.full_pipeline(oracle.make_job(F, E, N, B, d, seed), sizes, caps)
    compare(got, exp)


def test_stage_isolation(oracle):
    """Each GPU stage fed with the oracle's inputs."""
    F, E, N, B, d, seed = 60_001, 6, 5, 9, 0, 21
    job = nopfs.Job(F, E, N, B, d, seed)
    rj = oracle.make_job(F, E, N, B, d, seed)
    exp = oracle.full_pipeline(rj, wl.random_sizes(F, 1), np.array([10**8, 10**9], np.int64))
    R = torch.from_numpy(exp["R"]).cuda()
    c, f = nopfs.access_stats(job, R)
    nx = nopfs.reuse_next(job, R)
    sizes = wl.random_sizes(F, 1)
    t, u = nopfs.tier_plan(job, torch.from_numpy(exp["count"]).cuda(),
                           torch.from_numpy(exp["first"]).cuda(),
                           torch.from_numpy(sizes).cuda(), [10**8, 10**9])
    torch.cuda.synchronize()
    compare(dict(count=c.cpu().numpy(), first=f.cpu().numpy(), next=nx.cpu().numpy(),
                 tier=t.cpu().numpy(), used=u.cpu().numpy()), exp,
            ("count", "first", "next", "tier", "used"))


@pytest.mark.parametrize("caps", [[0], [1], [10**15], [0, 0, 10**15], [5_000_000, 0, 7],
                                  [2_000_000] * 7])
@pytest.mark.parametrize("path", PATHS)
def test_plan_capacity_edges(oracle, caps, path):
    F, E, N, B, d, seed = 5_000, 4, 3, 8, 1, 31
    sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
    caps = np.array(caps, np.int64)
    job = nopfs.Job(F, E, N, B, d, seed)
    got = gpu_pipeline(job, sizes, caps, path)
    exp = oracle.full_pipeline(oracle.make_job(F, E, N, B, d, seed), sizes, caps)
    compare(got, exp)
    if caps.max() == 0:
        assert (got["tier"] == -1).all()
    if caps[0] >= sizes.sum():
        assert (got["tier"] == 0).all()


@pytest.mark.parametrize("path", PATHS)
def test_equal_sizes_tie_breaks(oracle, path):
    """All sizes equal (CosmoFlow-like): the cut positions are decided by the
    (count, first, id) tie-breaks alone."""
    F, E, N, B, d, seed = 8_192, 10, 64, 1, 1, 42
    sizes = np.full(F, 16_777_216, np.int64)
    caps = np.array([16_777_216 * 37, 16_777_216 * 500], np.int64)
    job = nopfs.Job(F, E, N, B, d, seed)
    got = gpu_pipeline(job, sizes, caps, path)
    exp = oracle.full_pipeline(oracle.make_job(F, E, N, B, d, seed), sizes, caps)
    compare(got, exp)


@pytest.mark.parametrize("path", PATHS)
def test_slow_paths(oracle, path):
    """Force the oversized-bucket sort, the epoch-serial next-use path and the
    exact plan fallback with the test hooks; results must not change."""
    F, E, N, B, d, seed = 20_000, 6, 4, 8, 0, 41
    sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
    caps = _caps(sizes, (0.03, 0.2))
    job = nopfs.Job(F, E, N, B, d, seed)
    exp = oracle.full_pipeline(oracle.make_job(F, E, N, B, d, seed), sizes, caps)
    try:
        nopfs.debug_set(1, 64)   # tiny LDS bucket capacity: most buckets overflow
        nopfs.debug_set(2, 8)    # tiny candidate / next-use capacities
        got = gpu_pipeline(job, sizes, caps, path)
    finally:
        nopfs.debug_set(1, 0)
        nopfs.debug_set(2, 0)
    compare(got, exp)


@pytest.mark.parametrize("path", PATHS)
def test_deterministic(path):
    F, E, N, B, d, seed = 100_000, 5, 16, 8, 1, 5
    sizes = wl.random_sizes(F, seed)
    job = nopfs.Job(F, E, N, B, d, seed)
    a = gpu_pipeline(job, sizes, [10**9, 10**10], path)
    b = gpu_pipeline(job, sizes, [10**9, 10**10], path)
    compare(a, b)


WIDE = (34_000_000, 1, 1, 4, 0, 51)  # F, E, N, B, drop_last, seed


@pytest.fixture(scope="module")
def wide_case(oracle):
    F, E, N, B, d, seed = WIDE
    sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
    caps = _caps(sizes, (0.1, 0.3))
    return sizes, caps, oracle.full_pipeline(oracle.make_job(*WIDE), sizes, caps)


@pytest.mark.parametrize("path", PATHS)
def test_wide_windows(wide_case, path):
    """F above 4096 * 8192: sample windows wider than the counting pass holds
    in LDS at once (several passes per tile), and more reads per window than
    the next-use fast path takes (the epoch-serial path)."""
    sizes, caps, exp = wide_case
    got = gpu_pipeline(nopfs.Job(*WIDE), sizes, caps, path)
    compare(got, exp)


def _offset_view(shape, dtype):
    """A contiguous tensor one element into its allocation: rows that are
    not 4- or 16-byte aligned (the counting pass's one-cell-at-a-time path)."""
    n = int(np.prod(shape))
    return torch.full((n + 1,), 7, dtype=dtype, device="cuda")[1:].view(shape)


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("name,F,E,N,B,d,seed,fr", [JOBS[1], JOBS[4]], ids=["ragged", "e255"])
def test_unaligned_outputs(oracle, name, F, E, N, B, d, seed, fr, path):
    sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
    caps = _caps(sizes, fr)
    job = nopfs.Job(F, E, N, B, d, seed)
    exp = oracle.full_pipeline(oracle.make_job(F, E, N, B, d, seed), sizes, caps)
    count = _offset_view((N, F), torch.uint8)
    first = _offset_view((N, F), torch.int32)
    tier = _offset_view((N, F), torch.int8)
    assert count.data_ptr() % 4 and first.data_ptr() % 16 and tier.data_ptr() % 4
    s = torch.from_numpy(sizes).cuda()
    if path == "staged":
        R = nopfs.access_streams(job)
        nopfs.access_stats(job, R, count, first)
        _, used = nopfs.tier_plan(job, count, first, s, caps, tier)
        got = dict(count=count, first=first, tier=tier, used=used)
    else:
        got = nopfs.plan_job(job, s, caps, out=dict(count=count, first=first, tier=tier))
        assert got["count"].data_ptr() == count.data_ptr()
        assert got["tier"].data_ptr() == tier.data_ptr()
    torch.cuda.synchronize()
    compare({k: v.cpu().numpy() for k, v in got.items()}, exp,
            names=("count", "first", "tier", "used"))


def test_invariants_medium():
    F, E, N, B, d, seed = 300_000, 9, 12, 16, 0, 77
    sizes = wl.random_sizes(F, seed, 1_000, 2_000_000)
    caps = _caps(sizes, (0.05, 0.3))
    job = nopfs.Job(F, E, N, B, d, seed)
    got = gpu_pipeline(job, sizes, caps)
    _, _, Mw = nopfs.stream_shape(job)
    Mw = np.array(Mw)
    inv.check_streams(got["R"], F, E, Mw)
    inv.check_issued_once(got["R"], F, E, Mw)
    inv.check_stats(got["R"], got["count"], got["first"], Mw, E)
    inv.check_next(got["R"], got["next"], Mw, E)
    inv.check_plan(got["count"], got["first"], sizes, caps, got["tier"], got["used"])


def test_output_tensors_checked():
    job = nopfs.Job(100, 2, 2, 4)
    with pytest.raises(ValueError):
        nopfs.access_streams(job, R=torch.empty((2, 3), dtype=torch.int32, device="cuda"))
    with pytest.raises(TypeError):
        nopfs.access_streams(job, R=torch.empty((2, 48), dtype=torch.int32))
