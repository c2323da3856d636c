"""Seeded synthetic workloads shaped like the paper's datasets.

This module only generates inputs (job shapes, per-sample byte sizes and
per-tier capacities). It holds none of the planning arithmetic and is shared
by the tests, the benchmark and the oracle-side checks.

Sizes are int64 bytes drawn as ``rint(clip(lognormal(mu, sigma)))`` from
``numpy.random.default_rng(42 + index)``; capacities are decimal (1 GB =
1e9 bytes). The shuffle seed is 42 for every workload.

Stand-ins (the datasets themselves are not used):
  small       -- a 10k-sample sanity case
  imagenet1k  -- ImageNet-1k, 1,281,167 samples, N=16 (access-frequency example)
  imagenet1k_256 -- the same dataset over 256 workers
  imagenet22k -- ImageNet-22k, 14,197,103 samples, N=256 (largest)
  cosmoflow   -- CosmoFlow, 262,144 samples of 16 MiB, N=1024

Staging-buffer capacities (d0, the input of the staging schedule): 5 GB for
the ImageNet stand-ins (the simulated ImageNet-22k configuration fixes the
staging buffer at 5 GB), 5 GiB for CosmoFlow (the per-rank staging buffer of
the evaluation runs), 20 MB for the sanity case.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

SHUFFLE_SEED = 42


@dataclass(frozen=True)
class Workload:
    name: str
    index: int          # 1-based; the sizes generator is seeded with 42 + index
    F: int
    E: int
    N: int
    B: int              # per-worker batch
    drop_last: int
    caps: tuple         # per-worker tier capacities, fastest first (bytes)
    size_mu: float = 0.0
    size_sigma: float = 0.0
    size_lo: int = 0
    size_hi: int = 0
    fixed_size: int = 0  # > 0: every sample has this size
    staging: int = 0     # staging-buffer capacity, recorded but not a plan tier
    seed: int = SHUFFLE_SEED
    extra: dict = field(default_factory=dict)

    def job_tuple(self):
        return (self.F, self.E, self.N, self.B, self.drop_last, self.seed)


WORKLOADS = {
    "small": Workload("small", 1, 10_000, 5, 4, 16, 1, (100e6, 500e6),
                      size_mu=math.log(110e3), size_sigma=0.5,
                      size_lo=1_000, size_hi=2_000_000, staging=20e6),
    "imagenet1k": Workload("imagenet1k", 2, 1_281_167, 90, 16, 32, 1,
                           (64e9, 800e9), size_mu=math.log(110e3),
                           size_sigma=0.6, size_lo=1_000, size_hi=15_000_000,
                           staging=5e9),
    "imagenet1k_256": Workload("imagenet1k_256", 3, 1_281_167, 90, 256, 32, 1,
                               (16e9, 200e9), size_mu=math.log(110e3),
                               size_sigma=0.6, size_lo=1_000,
                               size_hi=15_000_000, staging=5e9),
    "imagenet22k": Workload("imagenet22k", 4, 14_197_103, 40, 256, 32, 1,
                            (64e9, 400e9), size_mu=math.log(90e3),
                            size_sigma=0.7, size_lo=1_000, size_hi=20_000_000,
                            staging=5e9),
    "cosmoflow": Workload("cosmoflow", 5, 262_144, 40, 1_024, 1, 1,
                          (32e9, 256e9), fixed_size=16_777_216, staging=5 * 2**30),
}

ORDER = ["small", "imagenet1k", "imagenet1k_256", "imagenet22k", "cosmoflow"]

# Performance-model parameters of the simulated small cluster (Lassen-like
# benchmarks of the Performance Simulator section), in bytes and bytes/s:
# compute 64 MB/s, preprocessing 200 MB/s, network 24,000 MB/s; staging
# buffer with 8 threads at 111 GB/s (its write rate taken equal to its read
# rate, the only one given); RAM with 4 threads at 85 GB/s, SSD with 2
# threads at 4 GB/s (the cache tiers, fastest first); PFS 2,870 MB/s at 8
# readers (per reader t(8)/8; larger reader counts are taken at that rate).
LASSEN_MODEL = dict(c=64e6, beta=200e6, b_c=24e9, pfs_t=2870e6, pfs_gamma=8, w0=111e9, p0=8,
                    r=(85e9, 4e9), p=(4, 2))


def sizes(w: Workload) -> np.ndarray:
    """Per-sample byte sizes, int64, length F."""
    if w.fixed_size:
        return np.full(w.F, w.fixed_size, dtype=np.int64)
    rng = np.random.default_rng(42 + w.index)
    s = rng.lognormal(w.size_mu, w.size_sigma, w.F)
    return np.rint(np.clip(s, w.size_lo, w.size_hi)).astype(np.int64)


def caps(w: Workload) -> np.ndarray:
    return np.array([int(c) for c in w.caps], dtype=np.int64)


def random_sizes(F: int, seed: int, lo: int = 1, hi: int = 1 << 20) -> np.ndarray:
    """Uniform integer sizes for ad-hoc test jobs."""
    return np.random.default_rng(seed).integers(lo, hi, F).astype(np.int64)
