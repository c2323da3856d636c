"""Brute-force checkers for tiny jobs (F <= 8).

Independent of the oracle: nothing here imports it. Each function enumerates
candidates and keeps the ones that satisfy a predicate taken from the paper's
definitions, so that a mistake in the oracle's construction (a wrong index, a
transposed operand, a dropped tie-break) shows up as a disagreement.
"""
from __future__ import annotations

import itertools


def shape(F, E, N, B, drop_last):
    """T, per-worker epoch lengths L_i and issued positions per epoch.

    Built from the batch structure (Performance Modeling): iteration h reads
    the global batch of N*B consecutive positions; worker i's local batch is
    the batch's offsets o with o % N == i."""
    G = N * B
    T = F // G if drop_last else -(-F // G)
    L = [0] * N
    for h in range(T):
        batch = range(h * G, min((h + 1) * G, F))
        for o, _p in enumerate(batch):
            L[o % N] += 1
    issued = sum(L)
    return T, L, issued


def certified_perm(keys):
    """The unique order of range(F) whose keys are ascending, equal keys by id.

    Enumerates all F! orders and keeps those that pass the certificate."""
    F = len(keys)
    good = []
    for perm in itertools.permutations(range(F)):
        ok = True
        for a, b in zip(perm, perm[1:]):
            if keys[a] > keys[b] or (keys[a] == keys[b] and a > b):
                ok = False
                break
        if ok:
            good.append(list(perm))
    assert len(good) == 1, f"{len(good)} orders pass the certificate"
    return good[0]


def streams(F, E, N, B, drop_last, perms):
    """R[i] = concatenation of worker i's local batches, iteration by iteration."""
    T, L, _ = shape(F, E, N, B, drop_last)
    G = N * B
    R = [[] for _ in range(N)]
    for e in range(E):
        for h in range(T):
            batch = perms[e][h * G:min((h + 1) * G, F)]
            for o, k in enumerate(batch):
                R[o % N].append(k)
    M_max = max(len(r) for r in R)
    return [r + [-1] * (M_max - len(r)) for r in R]


def stats(F, R_rows):
    count, first = [], []
    for row in R_rows:
        c = [0] * F
        fi = [-1] * F
        for f, k in enumerate(row):
            if k < 0:
                continue
            c[k] += 1
            if fi[k] < 0:
                fi[k] = f
        count.append(c)
        first.append(fi)
    return count, first


def next_use(R_rows):
    out = []
    for row in R_rows:
        nx = []
        for f, k in enumerate(row):
            found = -1
            if k >= 0:
                for g in range(f + 1, len(row)):
                    if row[g] == k:
                        found = g
                        break
            nx.append(found)
        out.append(nx)
    return out


def ranking(count_row, first_row):
    F = len(count_row)
    c = [int(x) for x in count_row]
    fr = [int(x) for x in first_row]
    inf = float("inf")
    return sorted(range(F), key=lambda k: (-c[k], fr[k] if fr[k] >= 0 else inf, k))


def plan_row(count_row, first_row, sizes, caps):
    """All (J+1)^F tier assignments; keep those that are capacity-feasible,
    contiguous and monotone along the ranking, and maximal (each tier stops at
    a sample that would overflow it). Exactly one must survive."""
    F, J = len(count_row), len(caps)
    sizes = [int(x) for x in sizes]
    caps = [int(x) for x in caps]
    order = ranking(count_row, first_row)
    survivors = []
    for assign in itertools.product(range(-1, J), repeat=F):
        along = [assign[k] if assign[k] >= 0 else J for k in order]
        if any(a > b for a, b in zip(along, along[1:])):
            continue
        used = [0] * J
        for k in range(F):
            if assign[k] >= 0:
                used[assign[k]] += sizes[k]
        if any(used[j] > caps[j] for j in range(J)):
            continue
        maximal = True
        for j in range(J):
            # first sample along the ranking placed after tier j
            after = [order[r] for r in range(F) if along[r] > j]
            if after and used[j] + sizes[after[0]] <= caps[j]:
                maximal = False
                break
        if not maximal:
            continue
        survivors.append((list(assign), used))
    assert len(survivors) == 1, f"{len(survivors)} assignments satisfy the plan predicate"
    return survivors[0]
