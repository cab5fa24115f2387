"""Pins for the oracle's microbatch frontier (Section 4.4, Algorithm 2 with its two rules:
one GPU frequency per microbatch, one SM allocation and launch timing per partition
type, plus the non-partition components).

Checked here against the plain definition, computed by brute force in this file:
  * every configuration of every frequency (Cartesian product of one point per used
    type), its time and energy summed in execution order with the components last,
    and the non-dominated set of all of them;
  * every reported point is such a configuration, summed bit for bit the same way;
  * every exact frontier point is matched or beaten by a reported point up to the bin
    width of its frequency times the number of used types, and no reported point is
    beaten by an exact point by more than that;
  * with one type, one partition and bins finer than every time gap, the result is
    exactly the non-dominated set of all points of all frequencies (also with repeated
    partitions of one type, and with components);
  * a frequency at which a used type has no point contributes nothing; an unused type
    reports no choice.
"""

import itertools

import numpy as np
import pytest

import oracle


def _case(rng, K, F, nmax, empty=None):
    segs, T, E = [], [], []
    for t in range(K):
        for f in range(F):
            n = 0 if empty == (t, f) else int(rng.integers(1, nmax + 1))
            T.extend(rng.uniform(1e-3, 5e-3, n) * (1.0 + 0.1 * f))
            E.extend(rng.uniform(0.5, 2.0, n) / (1.0 + 0.05 * f))
            segs.append(n)
    seg_off = np.zeros(K * F + 1, dtype=np.int64)
    seg_off[1:] = np.cumsum(segs)
    return seg_off, np.array(T), np.array(E)


def _config_sums(seg_off, T, E, F, f, seq, choice, cT, cE):
    """Time and energy of one configuration: execution order, components last."""
    Tm, Em = 0.0, 0.0
    for t in seq:
        x = seg_off[t * F + f] + choice[t]
        Tm = Tm + T[x]
        Em = Em + E[x]
    for c in range(len(cT)):
        Tm = Tm + cT[c][f]
        Em = Em + cE[c][f]
    return Tm, Em


def _exact(seg_off, T, E, K, F, seq, cT, cE):
    used = sorted(set(seq))
    pts = []
    for f in range(F):
        ranges = [range(int(seg_off[t * F + f + 1] - seg_off[t * F + f])) for t in used]
        if any(len(r) == 0 for r in ranges):
            continue
        for combo in itertools.product(*ranges):
            choice = dict(zip(used, combo))
            pts.append(_config_sums(seg_off, T, E, F, f, seq, choice, cT, cE) + (f,))
    return pts


def _nondominated(pts):
    keep = []
    for i, (t, e, *_) in enumerate(pts):
        if not any((t2 <= t and e2 <= e) and (t2 < t or e2 < e) for (t2, e2, *_) in pts):
            keep.append(pts[i])
    return keep


def _delta(seg_off, T, F, f, seq, B):
    """Automatic bin width of frequency f's composition (before its ulp nudges)."""
    cnt = {t: seq.count(t) for t in set(seq)}
    R = 0.0
    for t in sorted(cnt):
        x = T[seg_off[t * F + f]: seg_off[t * F + f + 1]] * cnt[t]
        R = R + (x.max() - x.min())
    return R / (B - 1) if R > 0 else 1.0


@pytest.mark.parametrize("seed", range(12))
def test_against_enumeration(seed):
    rng = np.random.default_rng(seed)
    K, F = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    seg_off, T, E = _case(rng, K, F, 4)
    seq = [int(x) for x in rng.integers(0, K, int(rng.integers(1, 5)))]
    nc = int(rng.integers(0, 3))
    cT = rng.uniform(1e-4, 1e-3, (nc, F))
    cE = rng.uniform(0.01, 0.1, (nc, F))
    B = int(rng.choice([16, 64, 1024]))
    oT, oE, of, och = oracle.microbatch(seg_off, T, E, K, F, seq, cT if nc else None,
                                        cE if nc else None, n_bins=B)
    # a frontier, in ascending time
    assert len(oT) > 0
    assert np.all(np.diff(oT) > 0) and np.all(np.diff(oE) < 0)
    used = sorted(set(seq))
    for r in range(len(oT)):
        choice = {t: int(och[r][t]) for t in range(K)}
        for t in range(K):
            assert (choice[t] >= 0) == (t in used)
        Tm, Em = _config_sums(seg_off, T, E, F, int(of[r]), seq, choice, cT, cE)
        assert Tm == oT[r] and Em == oE[r]
    exact = _nondominated(_exact(seg_off, T, E, K, F, seq, cT, cE))
    Ku = len(used)
    eps = 1e-12
    for (Ts, Es, f) in exact:
        tol = Ku * _delta(seg_off, T, F, f, seq, B) * (1 + 1e-9) + eps * Ts
        assert np.any((oT <= Ts + tol) & (oE <= Es * (1 + eps))), (Ts, Es, f)
    for r in range(len(oT)):
        for (Ts, Es, f) in exact:
            tol = Ku * _delta(seg_off, T, F, f, seq, B) * (1 + 1e-9) + eps * Ts
            assert not (Ts + tol < oT[r] and Es * (1 + eps) < oE[r])


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("reps,nc", [(1, 0), (3, 0), (1, 2)])
def test_one_type_fine_bins_is_exact(seed, reps, nc):
    rng = np.random.default_rng(100 + seed)
    F = 3
    seg_off, T, E = _case(rng, 1, F, 6)
    cT = rng.uniform(1e-4, 1e-3, (nc, F))
    cE = rng.uniform(0.01, 0.1, (nc, F))
    seq = [0] * reps
    oT, oE, of, och = oracle.microbatch(seg_off, T, E, 1, F, seq, cT if nc else None,
                                        cE if nc else None, n_bins=1 << 20)
    pts = []
    for f in range(F):
        for j in range(int(seg_off[f + 1] - seg_off[f])):
            pts.append(_config_sums(seg_off, T, E, F, f, seq, {0: j}, cT, cE) + (f, j))
    want = sorted(_nondominated(pts))
    assert len(want) == len(oT)
    for r, (t, e, f, j) in enumerate(want):
        assert (oT[r], oE[r], of[r], och[r][0]) == (t, e, f, j)


def test_missing_points_and_unused_types():
    rng = np.random.default_rng(7)
    K, F = 3, 3
    seg_off, T, E = _case(rng, K, F, 3, empty=(1, 2))
    # type 1 has no point at frequency 2: that frequency contributes nothing
    oT, oE, of, och = oracle.microbatch(seg_off, T, E, K, F, [0, 1, 0], n_bins=256)
    assert 2 not in set(of.tolist())
    assert np.all(och[:, 2] == -1) and np.all(och[:, 0] >= 0) and np.all(och[:, 1] >= 0)
    # without type 1 in the sequence, frequency 2 is back
    oT, oE, of, och = oracle.microbatch(seg_off, T, E, K, F, [2, 0], n_bins=256)
    assert np.all(och[:, 1] == -1)
    exact = _nondominated(_exact(seg_off, T, E, K, F, [2, 0], np.zeros((0, F)),
                                 np.zeros((0, F))))
    assert 2 in {f for (_, _, f) in exact} or len(exact) > 0


def test_rejects_bad_sequence():
    rng = np.random.default_rng(8)
    seg_off, T, E = _case(rng, 2, 2, 3)
    with pytest.raises(oracle.OracleError):
        oracle.microbatch(seg_off, T, E, 2, 2, [0, 2], n_bins=64)


@pytest.mark.parametrize("seed", range(6))
def test_repeated_types_fine_bins_is_exact(seed):
    """Types repeated different numbers of times, with times on grids that keep every
    configuration's time apart by more than the types' bin widths: the result is
    exactly the non-dominated set of the Cartesian enumeration (so each type's weight in
    the composition is its repeat count)."""
    rng = np.random.default_rng(200 + seed)
    K, F = 2 + seed % 2, 2
    segs, T, E = [], [], []
    for t in range(K):
        for f in range(F):
            n = int(rng.integers(2, 5))  # at most 4 points: j * repeats < 16
            T.extend((1.0 + np.arange(n) * 16.0 ** t) * 1e-3 * (1.0 + 0.1 * f))
            E.extend(rng.uniform(0.5, 2.0, n))
            segs.append(n)
    seg_off = np.zeros(K * F + 1, dtype=np.int64)
    seg_off[1:] = np.cumsum(segs)
    T, E = np.array(T), np.array(E)
    seq = [0, 1, 0, 0] + ([2] if K == 3 else [])
    nc = seed % 2
    cT = rng.uniform(1e-4, 1e-3, (nc, F))
    cE = rng.uniform(0.01, 0.1, (nc, F))
    oT, oE, of, och = oracle.microbatch(seg_off, T, E, K, F, seq, cT if nc else None,
                                        cE if nc else None, n_bins=1 << 14)
    want = sorted(_nondominated(_exact(seg_off, T, E, K, F, seq, cT, cE)))
    assert [(t, e, f) for (t, e, f) in want] == list(zip(oT.tolist(), oE.tolist(),
                                                         of.tolist()))


def test_repeat_count_weights_the_choice():
    """Type 0 three times, type 1 once.  Choosing (type 0: point 0, type 1: point 1)
    is on the frontier only when type 0 counts three times: with weight one it is beaten
    by (point 1, point 0)."""
    T = np.array([1.0, 2.0, 1.0, 2.5]) * 1e-3  # type 0: points 0, 1; type 1: points 0, 1
    E = np.array([3.0, 0.0, 2.0, 1.0])
    seg_off = np.array([0, 2, 4], dtype=np.int64)  # one frequency
    oT, oE, of, och = oracle.microbatch(seg_off, T, E, 2, 1, [0, 0, 0, 1], n_bins=64)
    want = sorted(_nondominated(_exact(seg_off, T, E, 2, 1, [0, 0, 0, 1], np.zeros((0, 1)),
                                       np.zeros((0, 1)))))
    assert len(want) == 4
    assert [(t, e) for (t, e, _) in want] == list(zip(oT.tolist(), oE.tolist()))
    assert [tuple(c) for c in och.tolist()] == [(0, 0), (0, 1), (1, 0), (1, 1)]


# ---- the enumerating oracle -------------------------------------------------------


@pytest.mark.parametrize("seed", range(10))
def test_exact_against_brute_force(seed):
    """Enumeration against the brute-force non-dominated set (pairwise dominance, not
    sort-and-scan), with every reported choice re-summed."""
    rng = np.random.default_rng(400 + seed)
    K, F = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    seg_off, T, E = _case(rng, K, F, 4, empty=(0, 0) if seed == 3 else None)
    seq = [int(x) for x in rng.integers(0, K, int(rng.integers(1, 6)))]
    nc = int(rng.integers(0, 3))
    cT = rng.uniform(1e-4, 1e-3, (nc, F))
    cE = rng.uniform(0.01, 0.1, (nc, F))
    oT, oE, of, och = oracle.microbatch_exact(seg_off, T, E, K, F, seq, cT if nc else None,
                                              cE if nc else None)
    want = sorted(_nondominated(_exact(seg_off, T, E, K, F, seq, cT, cE)))
    assert [(t, e, f) for (t, e, f) in want] == list(zip(oT.tolist(), oE.tolist(), of.tolist()))
    for r in range(len(oT)):
        choice = {t: int(och[r][t]) for t in range(K)}
        assert _config_sums(seg_off, T, E, F, int(of[r]), seq, choice, cT, cE) == (oT[r], oE[r])


@pytest.mark.parametrize("seed", range(4))
def test_exact_equals_grid_with_fine_bins(seed):
    """The enumeration and the grid composition (pinned above) agree once the bins are
    finer than every gap between configuration times."""
    rng = np.random.default_rng(500 + seed)
    K, F = 2, 2
    segs, T, E = [], [], []
    for t in range(K):
        for f in range(F):
            n = int(rng.integers(2, 5))
            T.extend((1.0 + np.arange(n) * 16.0 ** t) * 1e-3 * (1.0 + 0.1 * f))
            E.extend(rng.uniform(0.5, 2.0, n))
            segs.append(n)
    seg_off = np.zeros(K * F + 1, dtype=np.int64)
    seg_off[1:] = np.cumsum(segs)
    T, E = np.array(T), np.array(E)
    seq = [0, 1, 0, 0]
    a = oracle.microbatch_exact(seg_off, T, E, K, F, seq)
    b = oracle.microbatch(seg_off, T, E, K, F, seq, n_bins=1 << 14)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_exact_dominated_points_change_nothing():
    """Adding dominated points to a type's set leaves the frontier unchanged (fp64
    rounding is monotone, so a dominated choice never helps a sum)."""
    rng = np.random.default_rng(9)
    K, F = 2, 2
    seg_off, T, E = _case(rng, K, F, 4)
    seq = [0, 1, 1]
    a = oracle.microbatch_exact(seg_off, T, E, K, F, seq)
    # each segment gets a copy of its points, 1% slower and 1% more energy, appended
    segs, T2, E2 = [], [], []
    for g in range(K * F):
        x, y = T[seg_off[g]:seg_off[g + 1]], E[seg_off[g]:seg_off[g + 1]]
        T2.extend(list(x) + list(x * 1.01))
        E2.extend(list(y) + list(y * 1.01))
        segs.append(2 * len(x))
    seg2 = np.zeros(K * F + 1, dtype=np.int64)
    seg2[1:] = np.cumsum(segs)
    b = oracle.microbatch_exact(seg2, np.array(T2), np.array(E2), K, F, seq)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    np.testing.assert_array_equal(a[2], b[2])
