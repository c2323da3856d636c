"""The five workloads at full size on the GPU, in the launch configuration the
benchmark times.

 - imagenet1k (N=16, 1.28M samples, 90 epochs): the oracle runs in full and
   every output is compared element by element.
 - imagenet1k_256 and cosmoflow: streams, counts, first reads and next uses
   compared in full; the tier plan in full for a subset of workers (the
   oracle's per-worker sort of all samples is the slow part) and by its
   defining properties for the others.
 - imagenet22k (14.2M samples, N=256, 26.5 GB of outputs): sampled samples,
   whose positions in every epoch the oracle computes one by one from the
   definition of the shuffle; every output touching them is compared, plus
   the properties that hold at any size, checked on the device.
"""
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
    torch.cuda.empty_cache()


PATHS = ["staged", "fused"]  # four stage calls, or nopfs_plan_job (the benchmarked call)


def run(w, path="fused"):
    job = nopfs.Job(*w.job_tuple())
    sizes = wl.sizes(w)
    s = torch.from_numpy(sizes).cuda()
    out = nopfs.plan(job, s, wl.caps(w)) if path == "staged" else nopfs.plan_job(job, s, wl.caps(w))
    torch.cuda.synchronize()
    return job, sizes, out


def check_sampled(oracle, w, job, out, n_samples=24, seed=0):
    rng = np.random.default_rng(seed)
    samples = np.unique(np.concatenate([rng.choice(w.F, n_samples, replace=False),
                                        [0, w.F - 1]])).astype(np.int32)
    cols = oracle.sample_columns(oracle.make_job(*w.job_tuple()), samples)
    ks = torch.from_numpy(samples.astype(np.int64)).cuda()
    np.testing.assert_array_equal(out["count"][:, ks].cpu().numpy(), cols["col_count"])
    np.testing.assert_array_equal(out["first"][:, ks].cpu().numpy(), cols["col_first"])
    occ_i = cols["occ_worker"].ravel()
    occ_f = cols["occ_f"].ravel()
    keep = occ_i >= 0
    ii = torch.from_numpy(occ_i[keep].astype(np.int64)).cuda()
    ff = torch.from_numpy(occ_f[keep].astype(np.int64)).cuda()
    np.testing.assert_array_equal(out["R"][ii, ff].cpu().numpy(),
                                  np.broadcast_to(samples, cols["occ_f"].shape).ravel()[keep])
    np.testing.assert_array_equal(out["next"][ii, ff].cpu().numpy(),
                                  cols["occ_next"].ravel()[keep])


def check_device_properties(job, out):
    """Properties at any size, evaluated with torch on the device."""
    _, M, Mw = nopfs.stream_shape(job)
    count, first, R = out["count"], out["first"], out["R"]
    assert torch.equal(count.sum(dim=1, dtype=torch.int64).cpu(),
                       torch.tensor(Mw, dtype=torch.int64))
    assert int(count.sum(dim=0, dtype=torch.int64).max()) <= job.E
    assert torch.equal(first == -1, count == 0)
    # each epoch segment of a row holds distinct samples
    L = M // job.E
    for i in range(0, job.N, max(1, job.N // 8)):
        seg = R[i].view(job.E, L).to(torch.int64).sort(dim=1).values
        assert bool((seg[:, 1:] > seg[:, :-1]).all())
        assert int(seg.min()) >= 0 and int(seg.max()) < job.F


def check_plan_rows(job, sizes, caps, out, rows):
    c = out["count"][rows].cpu().numpy()
    f = out["first"][rows].cpu().numpy()
    t = out["tier"][rows].cpu().numpy()
    u = out["used"][rows].cpu().numpy()
    inv.check_plan(c, f, sizes, caps, t, u)


@pytest.mark.parametrize("path", PATHS)
def test_imagenet1k_full(imagenet1k_expected, path):
    w = wl.WORKLOADS["imagenet1k"]
    job, sizes, out = run(w, path)
    for n in ("R", "count", "first", "next", "tier", "used"):
        np.testing.assert_array_equal(out[n].cpu().numpy(), imagenet1k_expected[n], err_msg=n)


@pytest.mark.parametrize("name", ["imagenet1k_256", "cosmoflow"])
def test_full_streams_stats_next_and_plan_rows(oracle, name):
    w = wl.WORKLOADS[name]
    job, sizes, out = run(w)
    rj = oracle.make_job(*w.job_tuple())
    R = oracle.access_streams(rj)
    np.testing.assert_array_equal(out["R"].cpu().numpy(), R)
    count, first = oracle.access_stats(rj, R)
    np.testing.assert_array_equal(out["count"].cpu().numpy(), count)
    np.testing.assert_array_equal(out["first"].cpu().numpy(), first)
    np.testing.assert_array_equal(out["next"].cpu().numpy(), oracle.reuse_next(rj, R))
    rows = np.arange(0, w.N, w.N // 8)
    tier, used = oracle.tier_plan(rj, count[rows], first[rows], sizes, wl.caps(w))
    np.testing.assert_array_equal(out["tier"][torch.from_numpy(rows).cuda()].cpu().numpy(), tier)
    np.testing.assert_array_equal(out["used"][torch.from_numpy(rows).cuda()].cpu().numpy(), used)
    check_plan_rows(job, sizes, wl.caps(w), out, np.arange(1, w.N, w.N // 4))


@pytest.mark.parametrize("path", PATHS)
def test_imagenet22k_sampled(oracle, path):
    w = wl.WORKLOADS["imagenet22k"]
    job, sizes, out = run(w, path)
    check_sampled(oracle, w, job, out, n_samples=16)
    check_device_properties(job, out)
    check_plan_rows(job, sizes, wl.caps(w), out, [0, 131, 255])
    # the first tier boundary sits among samples read once (RAM 64 GB < the
    # ~237 GB a worker reads), the second among unread samples: no -1 left
    # unless the worker's whole row exceeds both tiers
    del out
    torch.cuda.empty_cache()
