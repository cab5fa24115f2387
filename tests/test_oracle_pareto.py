"""Pins for the oracle's GetFrontier (Algorithm 1's return, Algorithm 2's last step).

Checked against the definition by brute force: a point is dropped iff another point
is no worse in time and energy and better in one, or is an exact duplicate with a
smaller index.  Inputs include injected duplicates and equal-time / equal-energy ties.
"""

import numpy as np
import pytest


def brute_force_frontier(T, E):
    keep = []
    n = len(T)
    for a in range(n):
        dominated = False
        for b in range(n):
            if b == a:
                continue
            if T[b] <= T[a] and E[b] <= E[a] and (T[b] < T[a] or E[b] < E[a]):
                dominated = True
                break
            if T[b] == T[a] and E[b] == E[a] and b < a:
                dominated = True
                break
        if not dominated:
            keep.append(a)
    return sorted(keep, key=lambda i: (T[i], E[i], i))


def _tied_set(rng, n):
    T = rng.integers(0, 12, size=n).astype(np.float64) * 0.25 + 1.0
    E = rng.integers(0, 12, size=n).astype(np.float64) * 0.5 + 2.0
    dup = rng.integers(0, n, size=n // 4)
    T[dup[1:]] = T[dup[0]]
    E[dup[1:]] = E[dup[0]]
    return T, E


@pytest.mark.parametrize("seed", range(20))
def test_matches_brute_force_with_ties(oracle_lib, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 120))
    T, E = _tied_set(rng, n)
    got = oracle_lib.pareto(T, E)
    assert list(got) == brute_force_frontier(T, E)


@pytest.mark.parametrize("seed", range(5))
def test_matches_brute_force_continuous(oracle_lib, seed):
    rng = np.random.default_rng(100 + seed)
    n = 400
    T = rng.lognormal(size=n)
    E = 1.0 / T + rng.random(n)
    assert list(oracle_lib.pareto(T, E)) == brute_force_frontier(T, E)


def test_strict_staircase_and_domination_witness(oracle_lib):
    rng = np.random.default_rng(7)
    T, E = _tied_set(rng, 3000)
    idx = oracle_lib.pareto(T, E)
    assert np.all(np.diff(T[idx]) > 0) and np.all(np.diff(E[idx]) < 0)
    kept = set(idx.tolist())
    for a in range(len(T)):
        if a in kept:
            continue
        # every dropped point has a kept witness no worse in both objectives
        w = (T[idx] <= T[a]) & (E[idx] <= E[a])
        assert w.any()


def test_decomposable(oracle_lib):
    """Pareto(A u B) = Pareto(Pareto(A) u Pareto(B)): the identity that lets the GPU
    filter tiles independently and merge their staircases."""
    rng = np.random.default_rng(3)
    T, E = _tied_set(rng, 2000)
    full = oracle_lib.pareto(T, E)
    parts = np.array_split(np.arange(len(T)), 7)
    survivors = np.concatenate([p[oracle_lib.pareto(T[p], E[p])] for p in parts])
    survivors.sort()
    merged = survivors[oracle_lib.pareto(T[survivors], E[survivors])]
    assert list(merged) == list(full)


def test_empty_and_single(oracle_lib):
    assert len(oracle_lib.pareto(np.zeros(0), np.zeros(0))) == 0
    assert list(oracle_lib.pareto(np.array([3.0]), np.array([1.0]))) == [0]
    assert list(oracle_lib.pareto(np.array([1.0, 1.0]), np.array([2.0, 2.0]))) == [0]
