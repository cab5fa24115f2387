"""Pins for the oracle's launch-timing dynamic program (Appendix B).

Checked against:
  * brute force: every schedule of tiny instances (every sequence of groups: a lone op
    of either sequence, or a communication overlapped with a run of 1 .. Kmax
    computations of the other sequence), each costed exactly in rationals by a
    discrete-event walk written in this file, and the exact non-dominated set of all of
    them.  The DP frontier matches it point for point to rounding;
  * every schedule the DP reports, re-costed exactly, gives the point it is reported at;
  * the partition cost model (pinned on its own): with S1 = a partition's computations
    and S2 = its communication, every candidate of the cost model at that frequency and
    SM choice is matched or beaten by the DP frontier;
  * a hand-worked pair, the closed form without communication, no overlap when Kmax = 0,
    and the symmetry of swapping the two sequences.
"""

from fractions import Fraction as Fr

import numpy as np
import pytest

import oracle
from paper_2601_17654_amd import inputs as I


def _exact_group(ops, comm, run, ps):
    """Exact (T, E) of a communication overlapped with computations `run`: both start
    together; computations run in order in the shared state until the communication
    ends and alone after it; the group ends when both are done."""
    tc, pc = Fr(ops[comm][0]), Fr(ops[comm][1])
    now, e = Fr(0), Fr(0)
    for o in run:
        t0, p0, t1, p1 = (Fr(x) for x in ops[o])
        work = Fr(1)
        if now < tc:
            # shared state until tc or the end of the op
            can = (tc - now) / t1
            done = min(work, can)
            now += done * t1
            e += done * t1 * p1
            work -= done
        if work > 0:
            now += work * t0
            e += work * t0 * p0
    T = max(now, tc)
    return T, e + tc * pc + Fr(ps) * T


def _exact_alone(ops, o, ps):
    t, p = Fr(ops[o][0]), Fr(ops[o][1])
    return t, t * p + Fr(ps) * t


def _all_schedules(kind1, kind2, ops, ps, kmax):
    I_, J_ = len(kind1), len(kind2)
    out = []

    def rec(i, j, T, E, codes):
        if i == I_ and j == J_:
            out.append((T, E, tuple(codes)))
            return
        if i < I_:
            t, e = _exact_alone(ops, i, ps)
            rec(i + 1, j, T + t, E + e, codes + [0])
        if j < J_:
            t, e = _exact_alone(ops, I_ + j, ps)
            rec(i, j + 1, T + t, E + e, codes + [32])
        if i < I_ and kind1[i] == 1:
            for k in range(1, kmax + 1):
                if j + k > J_ or kind2[j + k - 1] != 0:
                    break
                t, e = _exact_group(ops, i, [I_ + j + r for r in range(k)], ps)
                rec(i + 1, j + k, T + t, E + e, codes + [64 + k])
        if j < J_ and kind2[j] == 1:
            for k in range(1, kmax + 1):
                if i + k > I_ or kind1[i + k - 1] != 0:
                    break
                t, e = _exact_group(ops, I_ + j, [i + r for r in range(k)], ps)
                rec(i + k, j + 1, T + t, E + e, codes + [96 + k])

    rec(0, 0, Fr(0), Fr(0), [])
    return out


def _exact_frontier(pts):
    pts = sorted(pts, key=lambda p: (p[0], p[1]))
    best, out = None, []
    for p in pts:
        if best is None or p[1] < best:
            out.append(p)
            best = p[1]
    return out


def _recost(codes, kind1, kind2, ops, ps):
    I_, J_ = len(kind1), len(kind2)
    i = j = 0
    T = E = Fr(0)
    for c in codes:
        if c < 0:
            break
        case, k = divmod(int(c), 32)
        if case == 0:
            t, e = _exact_alone(ops, i, ps)
            i += 1
        elif case == 1:
            t, e = _exact_alone(ops, I_ + j, ps)
            j += 1
        elif case == 2:
            assert kind1[i] == 1 and all(kind2[j + r] == 0 for r in range(k))
            t, e = _exact_group(ops, i, [I_ + j + r for r in range(k)], ps)
            i, j = i + 1, j + k
        else:
            assert kind2[j] == 1 and all(kind1[i + r] == 0 for r in range(k))
            t, e = _exact_group(ops, I_ + j, [i + r for r in range(k)], ps)
            i, j = i + k, j + 1
        T, E = T + t, E + e
    assert (i, j) == (I_, J_)
    return T, E


def _random_instance(rng, n1, n2, n_comm1, n_comm2):
    kind1 = [0] * n1
    kind2 = [0] * n2
    for p in rng.choice(n1, n_comm1, replace=False):
        kind1[p] = 1
    for p in rng.choice(n2, n_comm2, replace=False):
        kind2[p] = 1
    ops = []
    for k in kind1 + kind2:
        if k == 0:
            t0 = rng.uniform(1e-4, 2e-3)
            p0 = rng.uniform(300, 700)
            ops.append([t0, p0, t0 * rng.uniform(1.05, 1.6), p0 * rng.uniform(0.6, 0.95)])
        else:
            ops.append([rng.uniform(2e-4, 4e-3), rng.uniform(80, 200), 0.0, 0.0])
    return kind1, kind2, np.array(ops)


def test_hand_pair():
    ops = np.array([[2.0, 100.0, 4.0, 60.0], [1.0, 50.0, 0.0, 0.0]])
    T, E, sched, mc = oracle.launch_dp([0], [1], ops, 0.0, 1)
    # overlapped: 1 s shared (a quarter of the op), the rest alone: 1 + 0.75 * 2 = 2.5 s,
    # 1 * 60 + 1.5 * 100 + 1 * 50 = 260 J;  one after the other: 3 s, 200 + 50 = 250 J
    assert T.tolist() == [2.5, 3.0] and E.tolist() == [260.0, 250.0]
    assert sched[0].tolist() == [97, -1] and sched[1].tolist() == [0, 32]


@pytest.mark.parametrize("seed,n1,n2,c1,c2,kmax", [
    (0, 3, 3, 1, 1, 3), (1, 4, 3, 1, 1, 2), (2, 4, 4, 2, 1, 4), (3, 2, 4, 1, 2, 2),
    (4, 4, 4, 1, 1, 1), (5, 5, 1, 0, 1, 5), (6, 3, 3, 0, 0, 3), (7, 4, 4, 2, 2, 4)])
def test_brute_force(seed, n1, n2, c1, c2, kmax):
    rng = np.random.default_rng(seed)
    kind1, kind2, ops = _random_instance(rng, n1, n2, c1, c2)
    ps = 90.0
    T, E, sched, mc = oracle.launch_dp(kind1, kind2, ops, ps, kmax)
    want = _exact_frontier(_all_schedules(kind1, kind2, ops, ps, kmax))
    wt = np.array([float(x[0]) for x in want])
    we = np.array([float(x[1]) for x in want])
    tol = 1e-12
    # every exact frontier point is met by the DP to rounding ...
    for a, b in zip(wt, we):
        assert np.any((np.abs(T - a) <= tol * a) & (np.abs(E - b) <= tol * b)), (a, b)
    # ... and every DP point is an exact frontier point to rounding (schedules summed in
    # different orders can leave rounding-distinct copies of one exact point)
    for q in range(len(T)):
        assert np.any((np.abs(wt - T[q]) <= tol * T[q]) & (np.abs(we - E[q]) <= tol * E[q]))
        rt, re_ = _recost(sched[q], kind1, kind2, ops, ps)
        assert abs(float(rt) - T[q]) <= tol * T[q] and abs(float(re_) - E[q]) <= tol * E[q]
    assert np.all(np.diff(T) > 0) and np.all(np.diff(E) < 0)


def test_no_communication_closed_form():
    rng = np.random.default_rng(9)
    kind1, kind2, ops = _random_instance(rng, 3, 2, 0, 0)
    T, E, sched, mc = oracle.launch_dp(kind1, kind2, ops, 90.0, 3)
    tot_t = float(sum(Fr(o[0]) for o in ops))
    tot_e = float(sum(Fr(o[0]) * Fr(o[1]) + 90 * Fr(o[0]) for o in ops))
    # every interleaving is the same schedule up to the order of the sums
    assert np.all(np.abs(T - tot_t) <= 1e-14 * tot_t) and np.all(np.abs(E - tot_e) <= 1e-13 * tot_e)
    assert np.all((sched[:, :5] == 0) | (sched[:, :5] == 32))


def test_no_overlap_when_kmax_is_zero():
    rng = np.random.default_rng(10)
    kind1, kind2, ops = _random_instance(rng, 4, 4, 1, 1)
    T, E, sched, mc = oracle.launch_dp(kind1, kind2, ops, 90.0, 0)
    assert np.all((sched == 0) | (sched == 32))
    assert np.ptp(T) <= 1e-14 * T[0] and np.ptp(E) <= 1e-13 * E[0]


def test_swapping_the_sequences():
    rng = np.random.default_rng(11)
    kind1, kind2, ops = _random_instance(rng, 5, 4, 1, 2)
    a = oracle.launch_dp(kind1, kind2, ops, 90.0, 3)
    ops2 = np.concatenate([ops[5:], ops[:5]])
    b = oracle.launch_dp(kind2, kind1, ops2, 90.0, 3)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


@pytest.mark.parametrize("case", range(3))
def test_partition_cost_model_is_matched_or_beaten(case):
    """S1 = a partition's computations, S2 = its communication: launching the
    communication with computation p is the schedule 'p lone ops, the communication
    overlapped with the ops until it ends, the rest alone', so the DP frontier must
    match or beat every candidate of the partition cost model at that (f, SM choice)."""
    sp = I.SPACES[0]["space"]
    w = I.config_workload(0)
    p = case
    T_c, E_c = oracle.evaluate_partition(sp, w.t, w.pw, w.tc, w.pc, p)
    N, S = sp.n_kernels, sp.n_sm
    rng = np.random.default_rng(case)
    for f in rng.choice(sp.n_freq, 4, replace=False):
        for s in rng.choice(S, 3, replace=False):
            ops = [[w.t[p, f, o, 0], w.pw[p, f, o, 0], w.t[p, f, o, s + 1], w.pw[p, f, o, s + 1]]
                   for o in range(N)]
            ops.append([w.tc[p, f, 0, s], w.pc[p, f, 0, s], 0.0, 0.0])
            T, E, sched, mc = oracle.launch_dp([0] * N, [1], np.array(ops), sp.p_static, N)
            for pos in range(sp.n_pos):
                x = (f * sp.n_pos + pos) * S + s
                hit = (T <= T_c[x] * (1 + 1e-12)) & (E <= E_c[x] * (1 + 1e-12))
                assert hit.any(), (f, s, pos)
            xs = [(f * sp.n_pos + pos) * S + s for pos in range(sp.n_pos)]
            assert T[0] <= min(T_c[xs]) * (1 + 1e-12)
