import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU; parity vs the CPU oracle")
    config.addinivalue_line(
        "markers", "slow: CPU test that takes tens of seconds")


@pytest.fixture(scope="session")
def oracle():
    from oracle import ref
    ref.build()
    return ref


@pytest.fixture(scope="session")
def imagenet1k_expected(oracle):
    """The oracle's whole pipeline at ImageNet-1k size (N=16), shared by the
    full-size GPU tests."""
    from paper_2101_08734_amd import workloads as wl
    w = wl.WORKLOADS["imagenet1k"]
    return oracle.full_pipeline(oracle.make_job(*w.job_tuple()), wl.sizes(w), wl.caps(w))
