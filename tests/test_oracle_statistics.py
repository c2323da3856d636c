"""Distributional pins of the oracle (Distribution of Accesses, section 3.1).

The paper states that one worker's access frequency of a sample is
Binomial(E, 1/N) and gives a worked example for ImageNet-1k (N=16, E=90):
about 31,635 samples expected to be read more than 10 times by one worker
(31,863 in its Monte Carlo run). With drop_last the per-epoch inclusion
probability of a sample on worker i is exactly L/F rather than 1/N, so the
exact expectation is F * P(Binomial(E, L/F) > 10)."""
import json
import os

import numpy as np
import pytest
from scipy import stats as st

import invariants as inv

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "paper_access_frequency.json")))


def test_paper_closed_form_reading():
    """The printed sum has upper limit K and exponent K-k (garbled); read as E.
    With that reading the closed form reproduces the paper's 31,635."""
    F, N, E, d = GOLDEN["F"], GOLDEN["N"], GOLDEN["E"], GOLDEN["delta"]
    mu = E / N
    kmin = int(np.ceil((1 + d) * mu))
    assert kmin == GOLDEN["threshold_more_than"] + 1
    est = F * st.binom.sf(kmin - 1, E, 1 / N)
    assert abs(est - GOLDEN["paper_estimate"]) < 1.0
    # the paper's Monte Carlo value lies within 2 standard deviations
    sd = np.sqrt(F * st.binom.sf(kmin - 1, E, 1 / N) * (1 - st.binom.sf(kmin - 1, E, 1 / N)))
    assert abs(GOLDEN["paper_monte_carlo"] - est) < 2 * sd


@pytest.mark.slow
def test_paper_worked_example(oracle):
    """ImageNet-1k, N=16, E=90, B=32/worker, drop_last=1: per-worker number
    of samples read more than 10 times, from the oracle's full streams."""
    F, N, E = GOLDEN["F"], GOLDEN["N"], GOLDEN["E"]
    job = oracle.make_job(F, E, N, 32, 1, 42)
    _, _, Mw = oracle.stream_shape(job)
    R = oracle.access_streams(job)
    count, first = oracle.access_stats(job, R)
    L = int(Mw[0]) // E
    p = L / F
    q = st.binom.sf(GOLDEN["threshold_more_than"], E, p)
    exp, sd = F * q, np.sqrt(F * q * (1 - q))
    over = (count > GOLDEN["threshold_more_than"]).sum(axis=1)
    assert (np.abs(over - exp) < 5 * sd).all(), (over, exp, sd)
    assert abs(over.mean() - exp) < 4 * sd / np.sqrt(N)
    # against the paper's own numbers (p = 1/16, no tail dropped): within 1%
    assert abs(over.mean() - GOLDEN["paper_estimate"]) / GOLDEN["paper_estimate"] < 0.01
    assert abs(over.mean() - GOLDEN["paper_monte_carlo"]) / GOLDEN["paper_monte_carlo"] < 0.02
    # whole histogram against Binomial(E, L/F), pooled over workers
    _chi2_counts(count, E, p)
    # Lemma 1: counts over workers sum to at most E per sample; a worker
    # reading a sample (1+delta)E/N times forces another below the bound
    tot = count.sum(axis=0, dtype=np.int64)
    assert tot.max() <= E
    _lemma1(count, E, N, GOLDEN["delta"])


def _chi2_counts(count, E, p):
    obs = np.bincount(count.ravel(), minlength=E + 1).astype(np.float64)
    pmf = st.binom.pmf(np.arange(E + 1), E, p) * count.size
    keep = pmf > 20
    o = np.append(obs[keep], obs[~keep].sum())
    x = np.append(pmf[keep], pmf[~keep].sum())
    if x[-1] < 5:
        o, x = o[:-1], x[:-1]
        x = x * o.sum() / x.sum()
    chi2 = ((o - x) ** 2 / x).sum()
    pval = st.chi2.sf(chi2, len(o) - 1)
    assert pval > 1e-4, (chi2, pval)


def _lemma1(count, E, N, delta):
    hi = int(np.ceil((1 + delta) * E / N))
    bound = int(np.ceil((N - 1 - delta) / (N - 1) * E / N))
    cols = np.nonzero((count >= hi).any(axis=0))[0]
    for k in cols[:2000]:
        c = count[:, k].astype(np.int64)
        w = int(np.argmax(c))
        others = np.delete(c, w)
        assert others.min() <= bound


def test_small_counts_binomial(oracle):
    """10k samples, E=5, N=4: per-worker histogram ~ Binomial(E, L/F)."""
    job = oracle.make_job(10_000, 5, 4, 16, 1, 42)
    _, _, Mw = oracle.stream_shape(job)
    R = oracle.access_streams(job)
    count, _ = oracle.access_stats(job, R)
    p = (int(Mw[0]) // 5) / 10_000
    _chi2_counts(count, 5, p)
    distinct = (count > 0).sum(axis=1)
    exp = 10_000 * (1 - (1 - p) ** 5)
    assert (np.abs(distinct - exp) < 5 * np.sqrt(exp * (1 - p) ** 5)).all()


@pytest.mark.parametrize("F,trials", [(4, 48_000), (5, 60_000)])
def test_permutation_uniform(oracle, F, trials):
    """Each of the F! orders is equally likely over seeds (chi-square)."""
    import itertools
    idx = {p: n for n, p in enumerate(itertools.permutations(range(F)))}
    hist = np.zeros(len(idx))
    for s in range(trials):
        job = oracle.make_job(F, 1, 1, 1, 1, s * 0x9E3779B97F4A7C15 % (1 << 64))
        hist[idx[tuple(oracle.epoch_perm(job, 0))]] += 1
    x = trials / len(idx)
    chi2 = ((hist - x) ** 2 / x).sum()
    assert st.chi2.sf(chi2, len(idx) - 1) > 1e-4


def test_epochs_independent(oracle):
    """Counter-based keys: epoch e's order does not depend on the others, and
    different epochs are (nearly) uncorrelated."""
    job = oracle.make_job(20_000, 4, 1, 1, 1, 42)
    p0 = oracle.epoch_perm(job, 0)
    p3 = oracle.epoch_perm(job, 3)
    job_big = oracle.make_job(20_000, 200, 1, 1, 1, 42)
    np.testing.assert_array_equal(oracle.epoch_perm(job_big, 3), p3)
    inv0 = np.argsort(p0)
    inv3 = np.argsort(p3)
    r = np.corrcoef(inv0, inv3)[0, 1]
    assert abs(r) < 5 / np.sqrt(20_000)
