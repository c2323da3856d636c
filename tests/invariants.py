"""Property checks shared by the oracle tests and the GPU parity tests.

Each check follows a statement of the paper (cited per function) and holds at
any size, so it also serves where the oracle is too slow to run in full."""
from __future__ import annotations

import numpy as np


def check_perm(perm, keys):
    """Background: every sample exactly once per epoch; the order is the
    unique ascending (key, id) order (certificate checkable in O(F))."""
    F = len(keys)
    assert perm.shape == (F,)
    seen = np.zeros(F, bool)
    seen[perm] = True
    assert seen.all(), "not a permutation"
    k = keys[perm].astype(np.int64)
    dk = np.diff(k)
    assert (dk >= 0).all(), "keys not ascending"
    ties = dk == 0
    assert (np.diff(perm.astype(np.int64))[ties] > 0).all(), "equal keys not by id"


def check_streams(R, F, E, M_w):
    """Performance Modeling: within one epoch a worker's local batches are
    disjoint, so each epoch segment of a row holds distinct samples."""
    N, M_max = R.shape
    for i in range(N):
        M = int(M_w[i])
        row = R[i]
        assert (row[M:] == -1).all()
        if M == 0:
            continue
        L = M // E
        seg = row[:M].reshape(E, L)
        assert ((seg >= 0) & (seg < F)).all()
        s = np.sort(seg, axis=1)
        assert (np.diff(s, axis=1) > 0).all(), "repeat within an epoch"


def check_issued_once(R, F, E, M_w):
    """Across workers, each sample is read at most once per epoch (exactly
    once when no tail is dropped)."""
    N = R.shape[0]
    for e in range(E):
        seen = np.zeros(F, np.int64)
        for i in range(N):
            L = int(M_w[i]) // E
            np.add.at(seen, R[i, e * L:(e + 1) * L], 1)
        assert seen.max() <= 1


def check_stats(R, count, first, M_w, E):
    """Distribution of Accesses: counts sum to the reads issued; per sample
    the workers' counts sum to at most E (Lemma 1's premise); first = -1
    exactly when count = 0, and first points at the earliest read."""
    N, F = count.shape
    assert (count.sum(axis=1, dtype=np.int64) == M_w).all()
    assert (count.sum(axis=0, dtype=np.int64) <= E).all()
    assert ((first == -1) == (count == 0)).all()
    for i in range(N):
        M = int(M_w[i])
        acc = np.nonzero(count[i])[0]
        if len(acc) == 0:
            continue
        f = first[i, acc]
        assert (R[i, f] == acc).all()
        # no earlier read: the first occurrence index via a reversed scatter
        earliest = np.full(F, -1, np.int64)
        earliest[R[i, :M][::-1]] = np.arange(M - 1, -1, -1)
        assert (earliest[acc] == f).all()


def check_next(R, nxt, M_w, E):
    """I/O Access Patterns: next use = the following read of the same sample
    by the same worker; it always lies in a later epoch (a sample is read
    once per epoch); the number of reads with no next use = distinct samples."""
    N = R.shape[0]
    for i in range(N):
        M = int(M_w[i])
        assert (nxt[i, M:] == -1).all()
        if M == 0:
            continue
        L = M // E
        row, nx = R[i, :M], nxt[i, :M]
        has = nx >= 0
        f = np.nonzero(has)[0]
        assert (row[nx[has]] == row[has]).all()
        assert (nx[has] // L > f // L).all()
        assert (~has).sum() == len(np.unique(row))
        # nothing of the same sample strictly between f and next[f]: walking
        # the chain from each first read must visit every read exactly once
        visits = np.zeros(M, np.int64)
        starts = np.setdiff1d(np.arange(M), nx[has])
        for s in starts:
            g = s
            while g >= 0:
                visits[g] += 1
                g = nx[g]
        assert (visits == 1).all()


def check_plan(count, first, sizes, caps, tier, used):
    """Design: frequency-ordered fill, fastest class first, until the data is
    cached or storage is full. Checked as: tiers are non-decreasing along the
    ranking (uncached = last), each tier within capacity, each tier stopped
    only by a sample that would overflow it, used = bytes placed."""
    N, F = count.shape
    J = len(caps)
    sizes = sizes.astype(np.int64)
    for i in range(N):
        fr = np.where(first[i] >= 0, first[i].astype(np.int64), np.int64(2**62))
        order = np.lexsort((np.arange(F), fr, -count[i].astype(np.int64)))
        t = tier[i, order].astype(np.int64)
        t = np.where(t < 0, J, t)
        assert (np.diff(t) >= 0).all(), "tiers not monotone along the ranking"
        for j in range(J):
            u = int(sizes[tier[i] == j].sum())
            assert u == int(used[i, j])
            assert u <= int(caps[j])
            after = np.nonzero(t > j)[0]
            if len(after):
                assert u + int(sizes[order[after[0]]]) > int(caps[j]), "tier not maximal"
