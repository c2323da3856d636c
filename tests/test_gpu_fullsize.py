"""The five workloads at full size on the GPU, in the launch configuration the
benchmark times, compared element by element with the oracle.

 - imagenet1k (N=16, 1.28M samples, 90 epochs): the oracle's whole pipeline.
 - imagenet1k_256, cosmoflow and imagenet22k (14.2M samples, N=256, 26.5 GB
   of outputs per path): every element of R, count, first, next, tier and
   used, for every worker, on both paths (the four stage calls and the fused
   nopfs_plan_job). The oracle runs in a host thread pool: one task per
   epoch permutation, then one per chunk of worker rows (its per-worker
   counting, next-use and plan functions on its own rows of R); each chunk
   of device rows is copied back and compared as it is reached.
 - imagenet22k also checks the properties that hold at any size on the
   device (row sums of count, column sums at most E, first = -1 exactly
   where count = 0, distinct samples in each epoch segment of every row).
"""
import sys
import time

import numpy as np
import pytest

import oracle_pool

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


def log(msg):
    print(f"[fullsize {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def run(w, path="fused"):
    job = nopfs.Job(*w.job_tuple())
    sizes = wl.sizes(w)
    s = torch.from_numpy(sizes).cuda()
    out = nopfs.plan(job, s, wl.caps(w)) if path == "staged" else nopfs.plan_job(job, s, wl.caps(w))
    torch.cuda.synchronize()
    return job, sizes, out


def check_device_properties(job, out):
    """Properties at any size, evaluated with torch on the device."""
    _, M, Mw = nopfs.stream_shape(job)
    count, first, R = out["count"], out["first"], out["R"]
    assert torch.equal(count.sum(dim=1, dtype=torch.int64).cpu(),
                       torch.tensor(Mw, dtype=torch.int64))
    assert int(count.sum(dim=0, dtype=torch.int64).max()) <= job.E
    assert torch.equal(first == -1, count == 0)
    L = M // job.E
    for i in range(0, job.N, 16):
        seg = R[i:i + 16].view(-1, job.E, L).to(torch.int64).sort(dim=2).values
        assert bool((seg[..., 1:] > seg[..., :-1]).all())
        assert int(seg.min()) >= 0 and int(seg.max()) < job.F


@pytest.mark.parametrize("path", PATHS)
def test_imagenet1k_full(imagenet1k_expected, path):
    w = wl.WORKLOADS["imagenet1k"]
    job, sizes, out = run(w, path)
    for n in ("R", "count", "first", "next", "tier", "used"):
        np.testing.assert_array_equal(out[n].cpu().numpy(), imagenet1k_expected[n], err_msg=n)


def run_both(name):
    w = wl.WORKLOADS[name]
    t0 = time.perf_counter()
    outs = {}
    for path in PATHS:
        job, sizes, outs[path] = run(w, path)
    log(f"{name}: both paths on the device ({time.perf_counter() - t0:.1f}s)")
    return w, job, sizes, outs


@pytest.mark.parametrize("name", ["imagenet1k_256", "cosmoflow"])
def test_full_size_every_element(oracle, name):
    w, job, sizes, outs = run_both(name)
    rj = oracle.make_job(*w.job_tuple())
    perms = oracle_pool.oracle_perms(oracle, rj)
    mism = oracle_pool.compare_all_rows(oracle, rj, sizes, wl.caps(w), outs, perms=perms,
                                        chunk=8, log=log)
    assert not mism, "\n".join(mism[:20])
    del outs, perms
    torch.cuda.empty_cache()


# ImageNet-22k: both paths run once (53 GB of outputs stay on the device),
# the oracle's 40 permutations are computed once, and the 256 workers are
# compared in 8 parts of 32 (each part a test of its own, ~20 s of oracle work
# on 16 host threads).
I22K_PARTS = 8


@pytest.fixture(scope="module")
def i22k_device():
    w, job, sizes, outs = run_both("imagenet22k")
    yield w, job, sizes, outs
    del outs
    torch.cuda.empty_cache()


@pytest.fixture(scope="module")
def i22k_perms(oracle):
    w = wl.WORKLOADS["imagenet22k"]
    rj = oracle.make_job(*w.job_tuple())
    t0 = time.perf_counter()
    perms = oracle_pool.oracle_perms(oracle, rj)
    log(f"imagenet22k: oracle permutations ({time.perf_counter() - t0:.1f}s, "
        f"{oracle_pool.pool_threads()} threads)")
    return rj, perms


def test_imagenet22k_device_properties(i22k_device):
    _, job, _, outs = i22k_device
    for path in PATHS:
        check_device_properties(job, outs[path])


@pytest.mark.parametrize("part", range(I22K_PARTS))
def test_imagenet22k_every_element(oracle, i22k_device, i22k_perms, part):
    w, job, sizes, outs = i22k_device
    rj, perms = i22k_perms
    per = job.N // I22K_PARTS
    i0, i1 = part * per, (part + 1) * per
    t0 = time.perf_counter()
    mism = oracle_pool.compare_all_rows(oracle, rj, sizes, wl.caps(w), outs, perms=perms,
                                        chunk=2, rows=(i0, i1))
    log(f"imagenet22k: workers {i0}..{i1 - 1} compared ({time.perf_counter() - t0:.1f}s)")
    assert not mism, "\n".join(mism[:20])
