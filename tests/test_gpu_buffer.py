"""Clairvoyant buffer on the GPU vs the CPU oracle.

Stage isolation: R and next are the oracle's own (streams and next uses on
the host). Hits are integer decisions taken on integer sizes, so the hit
flags and the per-worker hit counts and bytes must be identical.

Cases: capacities from nothing held to everything held, unit sizes (where
the rule is Belady's optimal replacement with bypass), sizes that straddle
the capacity, rows with ragged tails and rows that cross many 32-bit words
of the held-key bitmap, one worker, more workers than samples, 255 epochs,
an empty job; ImageNet-1k against the full oracle with the 5 GB staging
buffer; at ImageNet-22k size (the benchmarked launch), seeded random epoch
permutations split across 256 workers, compared on sampled workers.
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
    # name, F, E, N, B, drop_last, seed
    ("small", 10_000, 5, 4, 16, 1, 42),
    ("ragged", 30_011, 5, 3, 7, 0, 3),
    ("medium", 150_000, 7, 8, 16, 1, 9),
    ("many_epochs", 2_000, 60, 16, 1, 0, 11),
    ("e255", 700, 255, 5, 3, 1, 12),
    ("wide", 20_000, 3, 300, 2, 1, 13),
    ("n_gt_f", 50, 4, 64, 1, 0, 14),
    ("one_sample", 1, 3, 1, 1, 1, 15),
    ("one_worker", 40_000, 4, 1, 64, 1, 16),
    ("long_rows", 400_000, 2, 2, 1000, 0, 18),
]
IDS = [j[0] for j in JOBS]
# capacity as a fraction of the bytes one worker reads in an epoch
D0_FRACTIONS = [0.0, 0.01, 0.2, 0.9, 10.0]


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _compare(name, hit_g, hits_g, hit_o, hits_o):
    hit_g = hit_g.cpu().numpy()
    hits_g = hits_g.cpu().numpy()
    if not np.array_equal(hit_g, hit_o):
        bad = np.argwhere(hit_g != hit_o)
        raise AssertionError(f"{name}: hit {len(bad)} mismatches, first {bad[:5].tolist()}")
    assert np.array_equal(hits_g, hits_o), (name, hits_g[:4], hits_o[:4])


def _epoch_bytes(sizes, N):
    return float(sizes.sum()) / N


@pytest.mark.parametrize("name,F,E,N,B,d,seed", JOBS, ids=IDS)
def test_matches_oracle(oracle, name, F, E, N, B, d, seed):
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(rjob)
    nx = oracle.reuse_next(rjob, R)
    sizes = wl.random_sizes(F, seed + 1, 1_000, 2_000_000)
    job = nopfs.Job(F, E, N, B, d, seed)
    Rd, nd, sd = _dev(R), _dev(nx), _dev(sizes)
    for fr in D0_FRACTIONS:
        d0 = int(fr * _epoch_bytes(sizes, N))
        hit_o, hits_o = oracle.buffer_sim(rjob, R, nx, sizes, d0)
        hit_g, hits_g = nopfs.buffer_sim(job, Rd, nd, sd, d0)
        torch.cuda.synchronize()
        _compare(f"{name} d0={d0}", hit_g, hits_g, hit_o, hits_o)


@pytest.mark.parametrize("C", [0, 1, 2, 31, 32, 33, 1000, 5000])
def test_unit_sizes(oracle, C):
    F, E, N, B, d, seed = 8_000, 6, 3, 5, 0, 31
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(rjob)
    nx = oracle.reuse_next(rjob, R)
    sizes = np.ones(F, np.int64)
    hit_o, hits_o = oracle.buffer_sim(rjob, R, nx, sizes, C)
    hit_g, hits_g = nopfs.buffer_sim(nopfs.Job(F, E, N, B, d, seed), _dev(R), _dev(nx),
                                     _dev(sizes), C)
    torch.cuda.synchronize()
    _compare(f"unit C={C}", hit_g, hits_g, hit_o, hits_o)


def test_sizes_around_capacity(oracle):
    """Samples larger than d0 are never admitted; samples exactly d0 are."""
    F, E, N, B, d, seed = 5_000, 5, 2, 4, 1, 32
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R = oracle.access_streams(rjob)
    nx = oracle.reuse_next(rjob, R)
    d0 = 1_000_000
    rng = np.random.default_rng(5)
    sizes = rng.choice(np.array([d0 - 1, d0, d0 + 1, d0 // 2, d0 // 3], np.int64), F)
    hit_o, hits_o = oracle.buffer_sim(rjob, R, nx, sizes, d0)
    hit_g, hits_g = nopfs.buffer_sim(nopfs.Job(F, E, N, B, d, seed), _dev(R), _dev(nx),
                                     _dev(sizes), d0)
    torch.cuda.synchronize()
    _compare("around d0", hit_g, hits_g, hit_o, hits_o)
    assert hits_o[:, 0].sum() > 0


def test_zero_iterations():
    job = nopfs.Job(10, 2, 4, 3, 1, 17)  # T = 0, M_max = 0
    R = torch.empty((4, 0), dtype=torch.int32, device="cuda")
    sizes = torch.ones(10, dtype=torch.int64, device="cuda")
    hit, hits = nopfs.buffer_sim(job, R, R.clone(), sizes, 5)
    torch.cuda.synchronize()
    assert hit.shape == (4, 0)
    assert (hits.cpu().numpy() == 0).all()


def test_repeat_calls_reuse_nothing(oracle):
    """Two calls in a row, the second on a smaller job: nothing of the first
    call's state leaks into the second."""
    outs = []
    for F, N in ((50_000, 4), (7_000, 2)):
        rjob = oracle.make_job(F, 6, N, 8, 0, 40)
        R = oracle.access_streams(rjob)
        nx = oracle.reuse_next(rjob, R)
        sizes = wl.random_sizes(F, 41, 1_000, 2_000_000)
        d0 = int(0.3 * _epoch_bytes(sizes, N))
        hit_o, hits_o = oracle.buffer_sim(rjob, R, nx, sizes, d0)
        hit_g, hits_g = nopfs.buffer_sim(nopfs.Job(F, 6, N, 8, 0, 40), _dev(R), _dev(nx),
                                         _dev(sizes), d0)
        torch.cuda.synchronize()
        outs.append((hit_g, hits_g, hit_o, hits_o))
    for k, o in enumerate(outs):
        _compare(f"call {k}", *o)


def test_imagenet1k_full(oracle, imagenet1k_expected):
    w = wl.WORKLOADS["imagenet1k"]
    rjob = oracle.make_job(*w.job_tuple())
    sizes = wl.sizes(w)
    out = imagenet1k_expected
    d0 = int(w.staging)
    hit_o, hits_o = oracle.buffer_sim(rjob, out["R"], out["next"], sizes, d0)
    job = nopfs.Job(*w.job_tuple())
    hit_g, hits_g = nopfs.buffer_sim(job, _dev(out["R"]), _dev(out["next"]), _dev(sizes), d0)
    torch.cuda.synchronize()
    _compare("imagenet1k", hit_g, hits_g, hit_o, hits_o)
    assert hits_o[:, 0].min() > 0


def test_imagenet22k_sampled_rows(oracle):
    """The benchmarked shape (14.2M samples, 256 workers, 40 epochs): each
    epoch a seeded random permutation of the samples, split across the
    workers as the access streams are; next uses from the product's own
    stage, checked against the oracle's on the sampled workers; the oracle
    replays three sampled workers with the 5 GB staging buffer."""
    w = wl.WORKLOADS["imagenet22k"]
    job = nopfs.Job(*w.job_tuple())
    _, M, Mw = nopfs.stream_shape(job)
    L = M // w.E
    assert (np.asarray(Mw) == M).all() and L * w.E == M
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2222)
    R = torch.empty((w.N, M), dtype=torch.int32, device="cuda")
    for e in range(w.E):
        perm = torch.randperm(w.F, generator=gen, device="cuda", dtype=torch.int64)
        R[:, e * L:(e + 1) * L] = perm[:w.N * L].view(L, w.N).t().to(torch.int32)
        del perm
    nx = nopfs.reuse_next(job, R)
    sizes_h = wl.sizes(w)
    d0 = int(w.staging)
    hit_g, hits_g = nopfs.buffer_sim(job, R, nx, _dev(sizes_h), d0)
    torch.cuda.synchronize()
    rjob = oracle.make_job(*w.job_tuple())
    for i in (0, 131, 255):
        Ri = R[i:i + 1].cpu().numpy()
        nxi = oracle.reuse_next_rows(rjob, Ri, i)
        assert np.array_equal(nxi, nx[i:i + 1].cpu().numpy()), i
        hit_o, hits_o = oracle.buffer_sim(rjob, Ri, nxi, sizes_h, d0, rows=(i, i + 1))
        _compare(f"imagenet22k row {i}", hit_g[i:i + 1], hits_g[i:i + 1], hit_o, hits_o)
        assert hits_o[0, 0] > 0
    del R, nx, hit_g, hits_g
    torch.cuda.empty_cache()
