"""Pins for the oracle's Bayesian-optimisation scores (Section 4.3, Algorithm 1;
reference point and stopping rule from Appendix C).

Checked here against what the definitions fix, by means independent of the oracle's
strip sweep:
  * HV and HVI equal the area counted cell by cell on the grid of all point coordinates
    (coordinate compression): exactly for integer points, to rounding otherwise, for
    all three energy variants (dynamic = total - static power x time, static = static
    power x time);
  * a hand-worked staircase; a single point's rectangle; points outside the box add
    nothing; dominated, duplicate and outside-box candidates score exactly 0;
  * the static variant's closed form (its frontier is the fastest measured point);
  * with zero static power the dynamic variant equals the total one and the static
    box is empty;
  * scaling time and energy by powers of two scales every score exactly;
  * the reference point is 1.1 x the worst measured value;
  * uncertainty against numpy's population standard deviation and closed forms;
  * selection: one pass equals numpy's lexsort order, hand-built overlaps between
    passes, exclusion of measured candidates, ties to the smaller index, NaN rejected;
  * the stopping rule on hand-computed histories.
"""

import numpy as np
import pytest

import oracle


def _area_cells(pts, rT, rE, extra=None):
    """Area dominated by `pts` (or, with `extra`, dominated by `extra` and by none of
    `pts`) inside the box below (rT, rE), summed over the cells of the grid spanned by
    every coordinate."""
    allp = list(pts) + ([extra] if extra is not None else [])
    xs = sorted({p[0] for p in allp if p[0] < rT} | {rT})
    ys = sorted({p[1] for p in allp if p[1] < rE} | {rE})
    area = 0.0
    for i in range(len(xs) - 1):
        for j in range(len(ys) - 1):
            x, y = xs[i], ys[j]
            by_pts = any(p[0] <= x and p[1] <= y and p[0] < rT and p[1] < rE for p in pts)
            if extra is None:
                hit = by_pts
            else:
                hit = (extra[0] <= x and extra[1] <= y and extra[0] < rT and extra[1] < rE
                       and not by_pts)
            if hit:
                area += (xs[i + 1] - x) * (ys[j + 1] - y)
    return area


def test_hv_hand_staircase():
    # strips [1,2) x (4-3), [2,3) x (4-2), [3,4) x (4-1): 1 + 2 + 3
    assert oracle.hypervolume([1, 2, 3], [3, 2, 1], 4, 4) == 6.0
    # order of the input and a dominated point change nothing
    assert oracle.hypervolume([3, 2.5, 1, 2], [1, 2.5, 3, 2], 4, 4) == 6.0


def test_hv_single_point_and_box():
    assert oracle.hypervolume([1.5], [0.25], 4.0, 2.0) == (4.0 - 1.5) * (2.0 - 0.25)
    # on or beyond the box edge: nothing
    assert oracle.hypervolume([4.0, 5.0, 1.0], [1.0, 0.0, 2.0], 4.0, 2.0) == 0.0
    assert oracle.hypervolume([], [], 4.0, 2.0) == 0.0


@pytest.mark.parametrize("seed", range(8))
def test_hv_integer_grid_exact(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 14))
    T = rng.integers(0, 12, n).astype(float)
    E = rng.integers(0, 12, n).astype(float)
    rT, rE = float(rng.integers(5, 14)), float(rng.integers(5, 14))
    assert oracle.hypervolume(T, E, rT, rE) == _area_cells(list(zip(T, E)), rT, rE)


def _obs_case(rng, n_seg, n_obs, n_cand, integer=False):
    cand_off = np.zeros(n_seg + 1, dtype=np.int64)
    cand_off[1:] = np.cumsum(n_cand)
    obs_off = np.zeros(n_seg + 1, dtype=np.int64)
    obs_off[1:] = np.cumsum(n_obs)
    if integer:
        T_obs = rng.integers(1, 20, obs_off[-1]).astype(float)
        E_obs = rng.integers(1, 20, obs_off[-1]).astype(float)
        T_hat = rng.integers(0, 24, cand_off[-1]).astype(float)
        E_hat = rng.integers(0, 24, cand_off[-1]).astype(float)
    else:
        T_obs = rng.uniform(1e-3, 4e-3, obs_off[-1])
        E_obs = rng.uniform(0.8, 2.0, obs_off[-1])
        T_hat = rng.uniform(0.5e-3, 5e-3, cand_off[-1])
        E_hat = rng.uniform(0.5, 2.4, cand_off[-1])
    return cand_off, T_hat, E_hat, obs_off, T_obs, E_obs


def _variant(v, t, e, ps):
    return e if v == 0 else (e - ps * t if v == 1 else ps * t)


@pytest.mark.parametrize("seed", range(4))
def test_hvi_integer_grid_exact_total(seed):
    rng = np.random.default_rng(100 + seed)
    # reference point 1.1 * max is not an integer, so use zero static power and check
    # the total and dynamic variants cell by cell (rectangle areas stay exact in
    # binary only up to rounding of rT, rE: compare to a few ulps of the box area)
    cand_off, Th, Eh, obs_off, To, Eo = _obs_case(rng, 2, [5, 9], [40, 30], integer=True)
    hvi, hv, ref = oracle.hvi(cand_off, Th, Eh, obs_off, To, Eo, 0.0)
    for g in range(2):
        o = slice(obs_off[g], obs_off[g + 1])
        pts = list(zip(To[o], Eo[o]))
        rT, rE = ref[g, 0], ref[g, 1]
        assert rT == 1.1 * To[o].max() and rE == 1.1 * Eo[o].max()
        box = rT * rE
        assert abs(hv[g, 0] - _area_cells(pts, rT, rE)) <= 1e-14 * box
        for x in range(cand_off[g], cand_off[g + 1]):
            want = _area_cells(pts, rT, rE, extra=(Th[x], Eh[x]))
            assert abs(hvi[0, x] - want) <= 1e-14 * box, (g, x)
            assert hvi[1, x] == hvi[0, x]
            assert hvi[2, x] == 0.0
    assert np.all(hv[:, 2] == 0.0)


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("v", [0, 1, 2])
def test_hvi_cells_all_variants(seed, v):
    rng = np.random.default_rng(200 + seed)
    ps = 90.0
    cand_off, Th, Eh, obs_off, To, Eo = _obs_case(rng, 1, [12], [60])
    hvi, hv, ref = oracle.hvi(cand_off, Th, Eh, obs_off, To, Eo, ps)
    pts = [(t, _variant(v, t, e, ps)) for t, e in zip(To, Eo)]
    rT = 1.1 * max(p[0] for p in pts)
    rE = 1.1 * max(p[1] for p in pts)
    assert ref[0, 0] == rT and ref[0, 1 + v] == rE
    base = _area_cells(pts, rT, rE)
    assert abs(hv[0, v] - base) <= 1e-12 * base
    for x in range(60):
        y = (Th[x], _variant(v, Th[x], Eh[x], ps))
        want = _area_cells(pts, rT, rE, extra=y)
        assert abs(hvi[v, x] - want) <= 1e-12 * (base + want), (x, hvi[v, x], want)


def test_hvi_zero_cases():
    To = np.array([1.0, 2.0, 3.0])
    Eo = np.array([3.0, 2.0, 1.0])
    # dominated, equal to an observation, on the box edge, beyond it, weakly dominated
    Th = np.array([2.5, 2.0, 3.3, 9.0, 2.0, 1.0, 0.5])
    Eh = np.array([2.5, 2.0, 0.1, 0.1, 2.0, 3.2, 3.3])
    cand_off = np.array([0, 7])
    obs_off = np.array([0, 3])
    hvi, hv, ref = oracle.hvi(cand_off, Th, Eh, obs_off, To, Eo, 0.0)
    assert hvi[0, 0] == 0.0 and hvi[0, 1] == 0.0 and hvi[0, 3] == 0.0 and hvi[0, 4] == 0.0
    assert hvi[0, 5] == 0.0  # (1, 3.2) is dominated by (1, 3)
    # (3.3, 0.1) sits a rounding step inside the box (1.1 * 3 rounds up): its exact gain
    # is a sliver far below the HV's rounding, so the difference is 0 up to that
    sliver = max(ref[0, 0] - 3.3, 0.0) * (ref[0, 1] - 0.1)
    assert abs(hvi[0, 2] - sliver) <= 4 * 2.0 ** -52 * hv[0, 0]
    # (0.5, 3.3): new strip [0.5, 1) x (rE - 3.3) with rE = 1.1 * 3
    assert abs(hvi[0, 6] - 0.5 * (ref[0, 1] - 3.3)) <= 1e-15 * 10


def test_hvi_static_closed_form():
    rng = np.random.default_rng(7)
    ps = 90.0
    cand_off, Th, Eh, obs_off, To, Eo = _obs_case(rng, 1, [20], [200])
    hvi, hv, ref = oracle.hvi(cand_off, Th, Eh, obs_off, To, Eo, ps)
    t0 = To.min()
    rT, rE = ref[0, 0], ref[0, 3]
    assert rE == 1.1 * (ps * To.max())
    base = (rT - t0) * (rE - ps * t0)
    assert abs(hv[0, 2] - base) <= 1e-15 * base
    for x in range(200):
        if Th[x] >= t0:
            assert hvi[2, x] == 0.0
        else:
            want = (rT - Th[x]) * (rE - ps * Th[x]) - base
            assert abs(hvi[2, x] - want) <= 1e-13 * base


def test_hvi_power_of_two_scaling_exact():
    rng = np.random.default_rng(11)
    cand_off, Th, Eh, obs_off, To, Eo = _obs_case(rng, 3, [7, 15, 1], [50, 10, 20])
    a, b = 2.0 ** 5, 2.0 ** -3
    h1, hv1, r1 = oracle.hvi(cand_off, Th, Eh, obs_off, To, Eo, 90.0)
    h2, hv2, r2 = oracle.hvi(cand_off, Th * a, Eh * b, obs_off, To * a, Eo * b, 90.0 * b / a)
    assert np.array_equal(h2, h1 * (a * b))
    assert np.array_equal(hv2, hv1 * (a * b))


def test_hvi_single_observation_and_order():
    rng = np.random.default_rng(12)
    cand_off, Th, Eh, obs_off, To, Eo = _obs_case(rng, 2, [1, 9], [30, 30])
    h1, hv1, _ = oracle.hvi(cand_off, Th, Eh, obs_off, To, Eo, 90.0)
    perm = np.concatenate([[0], 1 + rng.permutation(9)])
    h2, hv2, _ = oracle.hvi(cand_off, Th, Eh, obs_off, To[perm], Eo[perm], 90.0)
    assert np.array_equal(h1, h2) and np.array_equal(hv1, hv2)
    # one observation: HV is its rectangle to 1.1x itself
    t, e = To[0], Eo[0]
    assert hv1[0, 0] == (1.1 * t - t) * (1.1 * e - e)


def test_hvi_more_observations_never_raise_scores():
    rng = np.random.default_rng(13)
    cand_off, Th, Eh, obs_off, To, Eo = _obs_case(rng, 1, [10], [300])
    # keep the reference point fixed: the added points are not the worst ones
    To2 = np.concatenate([To, [To.min() * 1.01, To.mean()]])
    Eo2 = np.concatenate([Eo, [Eo.mean(), Eo.min() * 1.01]])
    h1, hv1, r1 = oracle.hvi(cand_off, Th, Eh, obs_off, To, Eo, 90.0)
    h2, hv2, r2 = oracle.hvi(cand_off, Th, Eh, np.array([0, 12]), To2, Eo2, 90.0)
    assert np.array_equal(r1[:, :2], r2[:, :2])
    assert np.all(h2[0] <= h1[0] + 1e-12 * hv1[0, 0])
    assert hv2[0, 0] >= hv1[0, 0]
    assert np.all(h1 >= -1e-12 * hv1.max())


def test_hvi_rejects_empty_observations():
    with pytest.raises(oracle.OracleError):
        oracle.hvi([0, 3], np.ones(3), np.ones(3), [0, 0], np.ones(0), np.ones(0), 90.0)


# --- uncertainty ---------------------------------------------------------------------

def test_uncertainty_numpy_std():
    rng = np.random.default_rng(21)
    Tm = rng.uniform(1e-3, 2e-3, (5, 400))
    Em = rng.uniform(0.5, 1.5, (5, 400))
    u = oracle.uncertainty(Tm, Em)
    want = np.std(Tm, axis=0) + np.std(Em, axis=0)
    assert np.allclose(u, want, rtol=1e-14, atol=0)


def test_uncertainty_closed_forms():
    Tm = np.array([[1.0, 5.0, 2.0], [3.0, 5.0, 2.0]])
    Em = np.array([[10.0, 1.0, 7.0], [10.0, 4.0, 7.0]])
    # two members a, b: std = |a - b| / 2
    assert np.array_equal(oracle.uncertainty(Tm, Em), [1.0, 1.5, 0.0])
    assert np.array_equal(oracle.uncertainty(Tm[:1], Em[:1]), [0.0, 0.0, 0.0])


# --- selection -----------------------------------------------------------------------

def _topk_lex(s, excl, m):
    idx = np.arange(s.shape[0])
    keep = ~np.isin(idx, excl)
    order = np.lexsort((idx[keep], -s[keep]))
    return idx[keep][order][:m]


@pytest.mark.parametrize("seed", range(4))
def test_select_single_pass_is_lexsort(seed):
    rng = np.random.default_rng(300 + seed)
    n = [500, 37, 3]
    off = np.concatenate([[0], np.cumsum(n)])
    s = np.round(rng.uniform(0, 4, (3, off[-1])), 1)  # many ties
    obs_n = [20, 5, 1]
    obs_off = np.concatenate([[0], np.cumsum(obs_n)])
    obs = np.concatenate([rng.choice(n[g], obs_n[g], replace=False) for g in range(3)])
    for p, (k1, k2, k3) in enumerate([(16, 0, 0), (0, 16, 0), (0, 0, 16)]):
        sel = oracle.select(off, s, None, obs_off, obs, k1, k2, k3, 16)
        for g in range(3):
            want = _topk_lex(s[p, off[g]:off[g + 1]], obs[obs_off[g]:obs_off[g + 1]], 16)
            assert np.array_equal(sel[g], want), (p, g)


def test_select_hand_overlap_and_fill():
    # 8 candidates; D = {0}
    s0 = np.array([9, 8, 7, 6, 5, 4, 3, 2], float)
    s1 = np.array([0, 7, 9, 1, 2, 3, 4, 5], float)  # top-2 over X\D: 2, 1 (1 already in)
    s2 = np.array([5, 5, 5, 5, 5, 5, 5, 5], float)  # all tied: smallest indices 1, 2
    unc = np.array([9, 0, 0, 8, 1, 7, 6, 7], float)
    sel = oracle.select([0, 8], np.stack([s0, s1, s2]), unc, [0, 1], [0], 2, 2, 2, 6)
    # pass 0: {1, 2}; pass 1: 2, 1 already in; pass 2: 1, 2 already in;
    # unc over X \ D \ C: 3 (8), then 5 and 7 tie at 7 -> 5, 7; need 6 - 2 = 4: 3, 5, 7, 6
    assert sel[0].tolist() == [1, 2, 3, 5, 7, 6]


def test_select_small_partition_and_no_unc():
    s = np.zeros((3, 4))
    sel = oracle.select([0, 4], s, np.zeros(4), [0, 2], [3, 1], 2, 1, 1, 8)
    assert sel[0].tolist() == [0, 2]
    sel = oracle.select([0, 4], s, None, [0, 0], np.zeros(0, np.int64), 1, 1, 1, 8)
    assert sel[0].tolist() == [0]


def test_select_negative_zero_ties_and_out_of_range_obs():
    s = np.array([[0.0, -0.0, 0.0, -0.0]] * 3)
    sel = oracle.select([0, 4], s, None, [0, 2], [-1, 7], 3, 0, 0, 3)
    assert sel[0].tolist() == [0, 1, 2]


@pytest.mark.parametrize("seed", range(3))
def test_select_invariants(seed):
    rng = np.random.default_rng(400 + seed)
    n = [300, 64, 20]
    off = np.concatenate([[0], np.cumsum(n)])
    s = rng.uniform(0, 1, (3, off[-1]))
    s[:, rng.random(off[-1]) < 0.5] = 0.0
    unc = rng.uniform(0, 1, off[-1])
    obs_n = [30, 8, 15]
    obs_off = np.concatenate([[0], np.cumsum(obs_n)])
    obs = np.concatenate([rng.choice(n[g], obs_n[g], replace=False) for g in range(3)])
    k, k1, k2, k3 = 32, 13, 6, 6
    sel = oracle.select(off, s, unc, obs_off, obs, k1, k2, k3, k)
    for g in range(3):
        D = set(obs[obs_off[g]:obs_off[g + 1]].tolist())
        C = sel[g].tolist()
        assert len(C) == len(set(C)) == min(k, n[g] - len(D))
        assert not (set(C) & D)
        for p, m in enumerate((k1, k2, k3)):
            top = _topk_lex(s[p, off[g]:off[g + 1]], list(D), m)
            assert set(top.tolist()) <= set(C)


def test_select_rejects_nan_and_bad_counts():
    s = np.zeros((3, 4))
    s[1, 2] = np.nan
    with pytest.raises(oracle.OracleError):
        oracle.select([0, 4], s, None, [0, 0], np.zeros(0, np.int64), 1, 1, 1, 3)
    with pytest.raises(oracle.OracleError):
        oracle.select([0, 4], np.zeros((3, 4)), None, [0, 0], np.zeros(0, np.int64), 2, 1, 1, 3)


# --- stopping rule -------------------------------------------------------------------

def test_hv_converged_hand():
    # improvements 5e-4 and ~1e-4: mean 3e-4 < 1e-3
    assert oracle.hv_converged([1.0, 1.0005, 1.0006], 2, 1e-3)
    # improvements 0.1, ~9e-5: mean ~0.05
    assert not oracle.hv_converged([1.0, 1.1, 1.1001], 2, 1e-3)
    # fewer batches than the window
    assert not oracle.hv_converged([1.0, 1.0], 2, 1e-3)
    assert oracle.hv_converged([1.0, 1.0, 1.0], 2, 1e-3)
    # a zero HV before the window's batches never converges
    assert not oracle.hv_converged([0.0, 0.0, 1.0, 1.0], 2, 1e-3)
    assert oracle.hv_converged([0.0, 1.0, 1.0, 1.0], 2, 1e-3)
