"""Pins for the oracle's Philox-4x32-10 keys.

Two implementations written independently of the oracle and already present
in this image are compiled here, test-only, and must agree word for word:
PyTorch's ATen engine header and rocRAND's engine header. Neither header is
copied into the repository.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
TORCH_INC = None
try:
    import torch.utils.cpp_extension as _ce  # noqa: F401
    import torch
    TORCH_INC = os.path.join(os.path.dirname(torch.__file__), "include")
except Exception:  # pragma: no cover
    pass

ROCRAND_HDR = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"


def _build(tmp_path, src, cmd):
    exe = str(tmp_path / os.path.splitext(os.path.basename(src))[0])
    subprocess.run(cmd + [os.path.join(HERE, "crosscheck", src), "-o", exe],
                   check=True, capture_output=True)
    return exe


def _blocks(exe, seed, e, n):
    out = subprocess.run([exe, str(seed), str(e), str(n)], check=True,
                         capture_output=True, text=True).stdout
    return np.array([[int(w) for w in line.split()] for line in out.splitlines()],
                    dtype=np.uint32)


CASES = [(42, 0, 64), (42, 3, 64), (7, 89, 16), (0, 0, 8),
         (0xFFFFFFFFFFFFFFFF, 254, 8), (123456789012345, 17, 8)]


def _oracle_blocks(oracle, seed, e, n):
    job = oracle.make_job(4 * n, e + 1, 1, 1, 1, seed)
    return oracle.epoch_keys(job, e).reshape(n, 4)


@pytest.mark.skipif(TORCH_INC is None or shutil.which("g++") is None,
                    reason="needs torch headers and g++")
def test_philox_matches_aten(oracle, tmp_path):
    exe = _build(tmp_path, "philox_aten.cpp",
                 ["g++", "-std=c++17", "-O1", f"-I{TORCH_INC}"])
    for seed, e, n in CASES:
        np.testing.assert_array_equal(_oracle_blocks(oracle, seed, e, n),
                                      _blocks(exe, seed, e, n))


@pytest.mark.skipif(not os.path.exists(ROCRAND_HDR) or shutil.which("hipcc") is None,
                    reason="needs rocRAND headers and hipcc")
def test_philox_matches_rocrand(oracle, tmp_path):
    exe = _build(tmp_path, "philox_rocrand.cpp",
                 ["hipcc", "-std=c++17", "-O1", "-x", "hip", "--offload-arch=gfx950"])
    for seed, e, n in CASES:
        np.testing.assert_array_equal(_oracle_blocks(oracle, seed, e, n),
                                      _blocks(exe, seed, e, n))


def test_block_function_direct(oracle):
    # the single-block entry point agrees with the keys of the epoch
    job = oracle.make_job(32, 6, 1, 1, 1, 99)
    keys = oracle.epoch_keys(job, 5)
    for b in range(8):
        out = oracle.philox4x32_10([b, 5, 0, 0], [99, 0])
        np.testing.assert_array_equal(out, keys[4 * b:4 * b + 4])


def test_keys_depend_on_epoch_and_seed(oracle):
    j1 = oracle.make_job(1000, 3, 1, 1, 1, 42)
    j2 = oracle.make_job(1000, 3, 1, 1, 1, 43)
    k0, k1 = oracle.epoch_keys(j1, 0), oracle.epoch_keys(j1, 1)
    assert (k0 != k1).mean() > 0.99
    assert (k0 != oracle.epoch_keys(j2, 0)).mean() > 0.99
    # keys of an epoch do not depend on F beyond the prefix
    j3 = oracle.make_job(1003, 3, 1, 1, 1, 42)
    np.testing.assert_array_equal(oracle.epoch_keys(j3, 1)[:1000], k1)
