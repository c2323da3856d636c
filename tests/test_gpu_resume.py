"""Epoch-range streams (a job resumed at epoch e0) on the GPU vs the oracle.

Every epoch's shuffle depends only on the seed and the epoch, so the streams
of epochs [e0, e1) are the columns [e0 * L_i, e1 * L_i) of each worker's full
stream. Expected values are the oracle's full streams, sliced per row (no
arithmetic in the slice); the product's range output must equal them and its
own full run's slice, element by element. The remaining epochs' counts, first
reads, next uses and plan are then computed on the range's shape (a job of
e1 - e0 epochs) and compared with the oracle's on the sliced streams.
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
    ("small", 10_000, 6, 4, 16, 1, 42),
    ("ragged", 30_011, 7, 3, 7, 0, 3),
    ("n_gt_f", 50, 5, 64, 1, 0, 14),
    ("one_worker", 40_000, 4, 1, 64, 1, 16),
    ("multi_bucket", 300_000, 5, 8, 32, 0, 21),
]
IDS = [j[0] for j in JOBS]


def _slice(oracle, job, R, e0, e1):
    """Rows of epochs [e0, e1) of the oracle's full streams, -1 padded."""
    _, _, Mw = oracle.stream_shape(job)
    L = [m // job.E for m in Mw]
    M = (e1 - e0) * max(L)
    out = np.full((job.N, M), -1, np.int32)
    for i in range(job.N):
        seg = R[i, e0 * L[i]:e1 * L[i]]
        out[i, :len(seg)] = seg
    return out


@pytest.mark.parametrize("name,F,E,N,B,d,seed", JOBS, ids=IDS)
def test_ranges_match_full_run(oracle, name, F, E, N, B, d, seed):
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R_o = oracle.access_streams(rjob)
    job = nopfs.Job(F, E, N, B, d, seed)
    R_full = nopfs.access_streams(job).cpu().numpy()
    assert np.array_equal(R_full, R_o)
    for e0, e1 in ((0, E), (1, E), (E - 1, E), (0, 1), (2, E - 1), (E // 2, E // 2 + 1)):
        if not 0 <= e0 < e1 <= E:
            continue
        got = nopfs.access_streams_range(job, e0, e1).cpu().numpy()
        want = _slice(oracle, rjob, R_o, e0, e1)
        assert got.shape == want.shape, (e0, e1)
        assert np.array_equal(got, want), (name, e0, e1)


@pytest.mark.parametrize("name,F,E,N,B,d,seed", JOBS[:3] + JOBS[4:], ids=IDS[:3] + IDS[4:])
def test_resumed_plan(oracle, name, F, E, N, B, d, seed):
    """Counts, first reads, next uses and the plan of the remaining epochs."""
    rjob = oracle.make_job(F, E, N, B, d, seed)
    R_o = oracle.access_streams(rjob)
    job = nopfs.Job(F, E, N, B, d, seed)
    sizes = wl.random_sizes(F, seed + 1, 1_000, 2_000_000)
    tot = int(sizes.sum())
    caps = np.array([int(0.01 * tot), int(0.1 * tot)], np.int64)
    e0 = E // 2
    sub = job.epochs(e0, E)
    rsub = oracle.make_job(F, E - e0, N, B, d, seed)
    R_rest = _slice(oracle, rjob, R_o, e0, E)
    count_o, first_o = oracle.access_stats(rsub, R_rest)
    next_o = oracle.reuse_next(rsub, R_rest)
    tier_o, used_o = oracle.tier_plan(rsub, count_o, first_o, sizes, caps)
    R_g = nopfs.access_streams_range(job, e0, E)
    count_g, first_g = nopfs.access_stats(sub, R_g)
    next_g = nopfs.reuse_next(sub, R_g)
    tier_g, used_g = nopfs.tier_plan(sub, count_g, first_g, torch.from_numpy(sizes).cuda(),
                                     [int(c) for c in caps])
    torch.cuda.synchronize()
    for what, g, o in (("R", R_g, R_rest), ("count", count_g, count_o), ("first", first_g, first_o),
                       ("next", next_g, next_o), ("tier", tier_g, tier_o), ("used", used_g, used_o)):
        assert np.array_equal(g.cpu().numpy(), o), (name, what)


def test_empty_range():
    job = nopfs.Job(1_000, 4, 3, 8, 1, 5)
    R = nopfs.access_streams_range(job, 2, 2)
    torch.cuda.synchronize()
    assert R.shape == (3, 0)
