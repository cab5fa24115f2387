"""Pins for the oracle's frontier comparison metrics (Section 6.1, "Metrics"):
max-throughput (leftmost point) time and energy reductions, iso-time energy reduction at
the baseline's least time, iso-energy time reduction at the baseline's least energy.

Checked against hand-worked cases and closed forms, and against what the definitions
fix: comparing a set with itself gives zeros, point order and dominated points change
nothing, a method with no point inside the deadline or budget gives NaN, and improving
the method never lowers a reduction.
"""

import numpy as np
import pytest

import oracle


def test_hand_case():
    # A: (1, 10), (2, 5), (4, 2);  B: (0.8, 9), (1.5, 4), (3, 1)
    r = oracle.compare([1, 2, 4], [10, 5, 2], [0.8, 1.5, 3], [9, 4, 1])
    # leftmost: (1, 10) vs (0.8, 9) -> 20 % time, 10 % energy
    # deadline 1: A 10, B 9 (only (0.8, 9) is in time) -> 10 %
    # budget 2: A 4, B 3 ((3, 1) is the fastest within 2) -> 25 %
    np.testing.assert_allclose(r[:4], [20, 10, 10, 25], rtol=1e-13)
    np.testing.assert_array_equal(r[4:], [1, 10, 9, 2, 4, 3])


def test_self_comparison_is_zero():
    rng = np.random.default_rng(1)
    T = rng.uniform(1, 2, 50)
    E = rng.uniform(1, 2, 50)
    r = oracle.compare(T, E, T, E)
    assert np.all(r[:4] == 0.0)


@pytest.mark.parametrize("n", [1, 2, 5, 8, 33])
def test_scaled_staircase_closed_form(n):
    i = np.arange(1, n + 1, dtype=float)
    TA, EA = i, 1.0 / i
    r = oracle.compare(TA, EA, 0.5 * TA, 0.5 * EA)
    np.testing.assert_allclose(r[:2], [50, 50], rtol=1e-14)
    # deadline 1: B's points with i/2 <= 1 are i <= 2, least energy 0.5 / min(n, 2)
    np.testing.assert_allclose(r[2], (1 - 0.5 / min(n, 2)) * 100, rtol=1e-14)
    # budget 1/n: B's points with 0.5/i <= 1/n are i >= n/2, least time ceil(n/2)/2
    np.testing.assert_allclose(r[3], (n - 0.5 * np.ceil(n / 2)) / n * 100, rtol=1e-14)


def test_order_and_dominated_points_change_nothing():
    rng = np.random.default_rng(2)
    TA, EA = rng.uniform(1, 3, 40), rng.uniform(1, 3, 40)
    TB, EB = rng.uniform(0.8, 3, 30), rng.uniform(0.8, 3, 30)
    r = oracle.compare(TA, EA, TB, EB)
    pa, pb = rng.permutation(40), rng.permutation(30)
    np.testing.assert_array_equal(oracle.compare(TA[pa], EA[pa], TB[pb], EB[pb]), r)
    # a point dominated by some point of its own set, and a leftmost tie with more energy
    TA2 = np.concatenate([TA, [TA[0] + 0.1, TA.min()]])
    EA2 = np.concatenate([EA, [EA[0] + 0.1, EA[np.argmin(TA)] + 1.0]])
    TB2 = np.concatenate([TB, [TB[3] + 0.5]])
    EB2 = np.concatenate([EB, [EB[3] + 0.5]])
    np.testing.assert_array_equal(oracle.compare(TA2, EA2, TB2, EB2), r)


def test_unreachable_deadline_and_budget_are_nan():
    r = oracle.compare([1.0, 2.0], [2.0, 1.0], [1.5, 3.0], [1.8, 1.2])
    assert np.isnan(r[2]) and np.isnan(r[6])   # no B point within time 1
    assert np.isnan(r[3]) and np.isnan(r[9])   # no B point within energy 1
    assert r[0] == pytest.approx(-50.0) and r[1] == pytest.approx(10.0)


def test_improving_the_method_never_lowers_a_reduction():
    rng = np.random.default_rng(3)
    TA, EA = rng.uniform(1, 3, 30), rng.uniform(1, 3, 30)
    TB, EB = rng.uniform(0.9, 3, 30), rng.uniform(0.9, 3, 30)
    r = oracle.compare(TA, EA, TB, EB)
    TB2, EB2 = TB * 0.97, EB * 0.95
    r2 = oracle.compare(TA, EA, TB2, EB2)
    for k in range(4):
        if not np.isnan(r[k]):
            assert r2[k] >= r[k]


def test_empty_sets_are_rejected():
    with pytest.raises(oracle.OracleError):
        oracle.compare([], [], [1.0], [1.0])
