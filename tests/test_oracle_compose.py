"""Pins for the oracle's frontier composition (Section 4.4, Algorithm 2).

Algorithm 2 sums time and energy over the Cartesian product of per-partition choices
and keeps the frontier.  The oracle instead runs a min-plus recurrence over a
discretised time axis.  Checked here against:
  * brute-force enumeration of the Cartesian product for 2-3 partitions (same bins):
    the composed array is bit-identical, because fp64 rounding is monotone;
  * the exact un-binned frontier of the Cartesian product: every exact frontier point
    is matched or beaten by a staircase point, and every staircase point's true time
    lies within P bin widths of its bin edge;
  * Pareto(A (+) B) = Pareto(Pareto(A) (+) Pareto(B)): composing raw candidate sets or
    their frontiers gives the same staircase;
  * one partition: the composed array is the binned input itself;
  * back-pointers: every reachable bin extracts to a schedule whose offsets add up to
    the bin and whose energies add up to the composed value bit-exactly.
"""

import itertools
import math
from fractions import Fraction as Fr

import numpy as np
import pytest


def _random_parts(rng, P, nmax):
    sizes = rng.integers(1, nmax + 1, size=P)
    off = np.zeros(P + 1, dtype=np.int64)
    off[1:] = np.cumsum(sizes)
    T = rng.uniform(1e-4, 5e-3, size=off[-1])
    E = rng.uniform(0.2, 1.0, size=off[-1])
    # inject exact ties in energy and time
    if off[-1] > 3:
        E[1] = E[0]
        T[2] = T[0]
    return off, T, E


def _tied_parts(rng, P, nmax):
    """Times on a coarse grid and energies on a dyadic grid: exact ties everywhere,
    both inside a bin and among min-plus sums."""
    sizes = rng.integers(2, nmax + 1, size=P)
    off = np.zeros(P + 1, dtype=np.int64)
    off[1:] = np.cumsum(sizes)
    T = rng.integers(0, 8, size=off[-1]) * 0.5e-3 + 1e-3
    E = rng.integers(1, 6, size=off[-1]) * 0.125
    return off, T, E


def _enumerate(off, T, E, pt_bin, upto):
    """Brute force over partitions 0..upto-1: F[b] = least left-to-right fp64 energy
    sum among combinations whose offsets add up to b."""
    P = upto
    ranges = [range(int(off[k]), int(off[k + 1])) for k in range(P)]
    F = {}
    for combo in itertools.product(*ranges):
        b = sum(int(pt_bin[j]) for j in combo)
        e = 0.0
        for j in combo:
            e = e + E[j]
        if b not in F or e < F[b]:
            F[b] = e
    return F


@pytest.mark.parametrize("tied", [False, True])
@pytest.mark.parametrize("seed", range(12))
def test_min_plus_equals_cartesian_enumeration(oracle_lib, seed, tied):
    rng = np.random.default_rng(seed)
    P = int(rng.integers(2, 4))
    off, T, E = (_tied_parts if tied else _random_parts)(rng, P, 7)
    B = int(rng.integers(8, 60))
    c = oracle_lib.compose(off, T, E, B)
    # bin rule written out: width = total range / (B - 1), nudged up until it fits
    tmin = [T[off[k]:off[k + 1]].min() for k in range(P)]
    rng_k = [T[off[k]:off[k + 1]].max() - tmin[k] for k in range(P)]
    R = 0.0
    for r in rng_k:
        R = R + r
    delta = R / (B - 1) if R > 0 else 1.0
    while 1 + sum(math.floor(r / delta) for r in rng_k) > B:
        delta = np.nextafter(delta, np.inf)
    assert c.delta == delta
    for k in range(P):
        for j in range(off[k], off[k + 1]):
            assert c.pt_bin[j] == min(math.floor((T[j] - tmin[k]) / delta),
                                      math.floor(rng_k[k] / delta))
    Fk = [_enumerate(off, T, E, c.pt_bin, k + 1) for k in range(P)]
    for b in range(B):
        if b in Fk[-1]:
            assert c.F[b] == Fk[-1][b]
        else:
            assert c.F[b] == np.inf and np.all(c.bp[:, b][P - 1:] == -1)
    # back-pointer tie rule: smallest offset b2 among the minimisers of stage k
    for k in range(1, P):
        lo, hi = int(off[k]), int(off[k + 1])
        e = {}
        for j in range(lo, hi):
            b2 = int(c.pt_bin[j])
            if b2 not in e or E[j] < e[b2][0]:
                e[b2] = (E[j], j - lo)
        for b in range(B):
            if b not in Fk[k]:
                assert c.bp[k, b] == -1
                continue
            best = None
            for b2 in sorted(e):
                a = b - b2
                if a in Fk[k - 1]:
                    v = Fk[k - 1][a] + e[b2][0]
                    if best is None or v < best[0]:
                        best = (v, e[b2][1])
            assert best[0] == Fk[k][b]
            assert c.bp[k, b] == best[1]


@pytest.mark.parametrize("seed", range(8))
def test_extracted_schedules_and_error_bound(oracle_lib, seed):
    rng = np.random.default_rng(50 + seed)
    P = int(rng.integers(2, 4))
    off, T, E = _random_parts(rng, P, 6)
    B = 64
    c = oracle_lib.compose(off, T, E, B)
    bins, tlo, e = oracle_lib.staircase(c.F, c.delta, c.tmin_sum)
    assert np.all(np.diff(bins) > 0) and np.all(np.diff(e) < 0)
    # every reachable bin extracts consistently
    for b in range(c.L):
        if not np.isfinite(c.F[b]):
            continue
        choice, ts, es = oracle_lib.extract(off, T, E, c, b)
        assert es == c.F[b]
        assert sum(int(c.pt_bin[off[k] + choice[k]]) for k in range(P)) == b
    # exact un-binned frontier of the Cartesian product
    combos = []
    for combo in itertools.product(*[range(int(off[k]), int(off[k + 1])) for k in range(P)]):
        combos.append((sum(Fr(T[j]) for j in combo), sum(Fr(E[j]) for j in combo)))
    combos.sort()
    exact = []
    for t_, e_ in combos:
        if not exact or e_ < exact[-1][1]:
            exact.append((t_, e_))
    tol = 1e-12
    for t_, e_ in exact:
        ok = (tlo <= float(t_) * (1 + tol)) & (e <= float(e_) * (1 + tol))
        assert ok.any()
    for b, t_lo in zip(bins, tlo):
        choice, ts, es = oracle_lib.extract(off, T, E, c, int(b))
        assert t_lo * (1 - tol) <= ts < t_lo + P * c.delta * (1 + tol)


@pytest.mark.parametrize("seed", range(6))
def test_compose_raw_equals_compose_frontiers(oracle_lib, seed):
    rng = np.random.default_rng(200 + seed)
    P = 3
    off, T, E = _random_parts(rng, P, 40)
    kept = [np.arange(off[k], off[k + 1])[oracle_lib.pareto(T[off[k]:off[k + 1]],
                                                            E[off[k]:off[k + 1]])]
            for k in range(P)]
    off2 = np.zeros(P + 1, dtype=np.int64)
    off2[1:] = np.cumsum([len(x) for x in kept])
    sel = np.concatenate(kept)
    raw = oracle_lib.compose(off, T, E, 200)
    fr = oracle_lib.compose(off2, T[sel], E[sel], 200, delta=raw.delta)
    a = oracle_lib.staircase(raw.F, raw.delta, raw.tmin_sum)
    b = oracle_lib.staircase(fr.F, fr.delta, fr.tmin_sum)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_single_partition_is_binned_input(oracle_lib):
    rng = np.random.default_rng(9)
    off, T, E = _random_parts(rng, 1, 50)
    c = oracle_lib.compose(off, T, E, 16)
    for b in range(16):
        members = [j for j in range(off[1]) if c.pt_bin[j] == b]
        if members:
            best = min(members, key=lambda j: (E[j], j))
            assert c.F[b] == E[best] and c.bp[0, b] == best
        else:
            assert c.F[b] == np.inf and c.bp[0, b] == -1


def test_degenerate_inputs(oracle_lib):
    # every partition a single point: range 0, width 1.0, one bin
    off = np.array([0, 1, 2, 3], dtype=np.int64)
    T = np.array([1e-3, 2e-3, 3e-3])
    E = np.array([1.0, 2.0, 3.0])
    c = oracle_lib.compose(off, T, E, 4)
    assert c.delta == 1.0 and c.L == 1 and c.F[0] == 6.0 and np.all(c.F[1:] == np.inf)
    assert c.tmin_sum == 1e-3 + 2e-3 + 3e-3
    # a caller-given width that needs more bins than allowed is refused
    off = np.array([0, 3], dtype=np.int64)
    with pytest.raises(oracle_lib.OracleError):
        oracle_lib.compose(off, np.array([0.0, 1.0, 2.0]), np.array([3.0, 2.0, 1.0]), 2,
                           delta=0.5)
    # empty partitions are rejected
    with pytest.raises(oracle_lib.OracleError):
        oracle_lib.compose(np.array([0, 0], dtype=np.int64), np.zeros(0), np.zeros(0), 4)
