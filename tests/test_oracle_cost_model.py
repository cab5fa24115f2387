"""Pins for the oracle's partition cost model (Sections 2.1, 2.3, 3.2, 4.2).

The oracle evaluates a candidate with a prefix-sum walk.  Here it is checked against
things that do not share that formulation:
  * an exact-rational discrete-event simulation of the same fluid model, written from
    the model's description (kernels progress at 1/t in the current SM state; comm
    kernels launch at kernel boundaries and run FIFO on one stream);
  * closed forms for degenerate schedules (fully exposed comm, zero-length comm, one
    kernel, no SM loss);
  * bounds that hold for any schedule;
  * the paper's energy decomposition (static power x time + dynamic energy), checked
    against the printed energy-breakdown table.
"""

import os
from fractions import Fraction as Fr

import numpy as np
import pytest

from paper_2601_17654_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def simulate(t, pw, tcm, pcm, sigma, pos, p_static):
    """Event-driven simulation in exact rationals.

    t[i][s], pw[i][s]: kernel time / dynamic power in SM state s (one frequency).
    Comm m is launched once compute has finished kernels 0..pos[m]-1, starts when the
    comm stream is free (FIFO), runs tcm[m] seconds drawing pcm[m] W, and while it runs
    compute is in state sigma[m].  Returns (T, E) as Fractions.
    """
    N, M = len(t), len(tcm)
    now = Fr(0)
    k = 0  # kernel in progress
    frac = Fr(0)  # finished fraction of kernel k
    energy = Fr(0)
    nxt_comm = 0
    active = None
    comm_end = None
    while True:
        if active is None and nxt_comm < M and k >= pos[nxt_comm]:
            active = nxt_comm
            comm_end = now + tcm[active]
            energy += pcm[active] * tcm[active]
            nxt_comm += 1
            continue
        state = sigma[active] if active is not None else 0
        events = []
        if k < N:
            events.append(now + (1 - frac) * t[k][state])
        if active is not None:
            events.append(comm_end)
        if not events:
            break
        t_next = min(events)
        dt = t_next - now
        if k < N:
            energy += pw[k][state] * dt
            frac += dt / t[k][state]
            if frac == 1:
                k += 1
                frac = Fr(0)
        if active is not None and t_next == comm_end:
            active = None
        now = t_next
    return now, p_static * now + energy


def _fr(a):
    return [[Fr(float(x)) for x in row] for row in a]


def exact_all(space, tab, part):
    """(T, E) float64 arrays of every candidate, enumerated in the documented order:
    frequency slowest, then launch position (pair), then SM choice(s)."""
    S = space.n_sm
    Ts, Es = [], []
    for f in range(space.n_freq):
        t = _fr(tab["t"][part, f])
        pw = _fr(tab["pw"][part, f])
        tc = tab["tc"][part, f]
        pc = tab["pc"][part, f]
        if space.n_comm == 1:
            combos = [((p,), (s,)) for p in range(space.n_pos) for s in range(S)]
        else:
            combos = [((p1, p2), (s1, s2)) for p1 in range(space.n_pos)
                      for p2 in range(p1, space.n_pos) for s1 in range(S) for s2 in range(S)]
        for pos, sms in combos:
            tcm = [Fr(float(tc[m, s])) for m, s in enumerate(sms)]
            pcm = [Fr(float(pc[m, s])) for m, s in enumerate(sms)]
            T, E = simulate(t, pw, tcm, pcm, [s + 1 for s in sms], pos, Fr(space.p_static))
            Ts.append(float(T))
            Es.append(float(E))
    return np.array(Ts), np.array(Es)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("n_comm", [1, 2])
def test_walk_matches_exact_event_simulation(oracle_lib, seed, n_comm):
    rng = np.random.default_rng(1000 + seed)
    space = I.random_space(rng, n_comm=n_comm, max_kernels=5, max_sm=3 if n_comm == 2 else 4,
                           max_freq=2, n_parts=2)
    tab = I.make_tables(space, seed=seed, comm_bytes=(4e6, 64e6))
    for part in range(space.n_parts):
        T, E = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], part)
        Tx, Ex = exact_all(space, tab, part)
        assert T.shape == Tx.shape == (space.n_cand,)
        np.testing.assert_allclose(T, Tx, rtol=1e-12, atol=0)
        np.testing.assert_allclose(E, Ex, rtol=1e-12, atol=0)


def test_walk_matches_simulation_long_comm(oracle_lib):
    """Comm longer than all compute, and comm shorter than one kernel: both regimes."""
    space = I.Space(1, 4, 2, 5, (1, 16, 32), (1005.0, 1980.0))
    for scale in (1e-3, 1e3):
        tab = I.make_tables(space, seed=7, comm_bytes=(4e6, 64e6))
        tab["tc"] = tab["tc"] * scale
        T, E = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], 0)
        Tx, Ex = exact_all(space, tab, 0)
        np.testing.assert_allclose(T, Tx, rtol=1e-12)
        np.testing.assert_allclose(E, Ex, rtol=1e-12)


def _single(space, tab, f, p, s):
    return (f * space.n_pos + p) * space.n_sm + s


def test_exposed_comm_closed_form(oracle_lib):
    """Launching after the last kernel: T = sum of state-0 times + Tc (Section 3.2.1:
    exposed communication), E = P_static*T + sum pw*t + pc*Tc."""
    space = I.Space(1, 7, 1, 8, (2, 8, 24), (1005.0, 1500.0, 1980.0))
    tab = I.make_tables(space, seed=3, comm_bytes=(16e6, 256e6))
    T, E = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], 0)
    for f in range(space.n_freq):
        t0 = tab["t"][0, f, :, 0]
        p0 = tab["pw"][0, f, :, 0]
        for s in range(space.n_sm):
            tc, pc = tab["tc"][0, f, 0, s], tab["pc"][0, f, 0, s]
            c = _single(space, tab, f, space.n_kernels, s)
            Tref = float(sum(Fr(x) for x in t0) + Fr(tc))
            Eref = float(Fr(space.p_static) * Fr(Tref) + sum(Fr(a) * Fr(b) for a, b in zip(p0, t0))
                         + Fr(pc) * Fr(tc))
            assert T[c] == pytest.approx(Tref, rel=1e-14)
            assert E[c] == pytest.approx(Eref, rel=1e-14)


def test_zero_length_comm_and_no_sm_loss(oracle_lib):
    """Tc = 0: the schedule is plain sequential compute.  Giving comm zero SMs' worth
    of slowdown (state tables equal to state 0): T = max(sum t, L + Tc)."""
    space = I.Space(1, 5, 1, 6, (4, 12), (1200.0, 1980.0))
    tab = I.make_tables(space, seed=11, comm_bytes=(4e6, 64e6))
    tab["t"] = np.repeat(tab["t"][..., :1], 3, axis=-1)
    tab["pw"] = np.repeat(tab["pw"][..., :1], 3, axis=-1)
    T, E = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], 0)
    for f in range(space.n_freq):
        t0 = tab["t"][0, f, :, 0]
        for p in range(space.n_pos):
            for s in range(space.n_sm):
                L = float(sum(Fr(x) for x in t0[:p]))
                ref = max(float(sum(Fr(x) for x in t0)), L + tab["tc"][0, f, 0, s])
                assert T[_single(space, tab, f, p, s)] == pytest.approx(ref, rel=1e-14)
    tab["tc"] = np.zeros_like(tab["tc"])
    T, E = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], 0)
    for f in range(space.n_freq):
        total = float(sum(Fr(x) for x in tab["t"][0, f, :, 0]))
        np.testing.assert_allclose(T[f * 12:(f + 1) * 12], total, rtol=1e-14)


def test_single_kernel_closed_form(oracle_lib):
    """N = 1, launch with the kernel: if Tc >= t_sigma the kernel finishes under comm
    and T = Tc; otherwise the unfinished fraction 1 - Tc/t_sigma runs in state 0:
    T = Tc + (1 - Tc/t_sigma) * t_0."""
    space = I.Space(1, 1, 1, 1, (1, 4, 16, 32), (1005.0, 1980.0))
    for scale in (0.05, 1.0, 20.0):
        tab = I.make_tables(space, seed=5, comm_bytes=(4e6, 64e6))
        tab["tc"] = tab["tc"] * scale
        T, E = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], 0)
        for f in range(2):
            for s in range(4):
                ts, t0 = Fr(tab["t"][0, f, 0, s + 1]), Fr(tab["t"][0, f, 0, 0])
                ps, p0 = Fr(tab["pw"][0, f, 0, s + 1]), Fr(tab["pw"][0, f, 0, 0])
                tc, pc = Fr(tab["tc"][0, f, 0, s]), Fr(tab["pc"][0, f, 0, s])
                if tc >= ts:
                    Tr, Ed = tc, ps * ts
                else:
                    rest = (1 - tc / ts) * t0
                    Tr, Ed = tc + rest, ps * tc + p0 * rest
                Er = Fr(space.p_static) * Tr + Ed + pc * tc
                c = f * 4 + s
                assert T[c] == pytest.approx(float(Tr), rel=1e-14)
                assert E[c] == pytest.approx(float(Er), rel=1e-14)


def test_time_bounds(oracle_lib):
    """For one comm kernel launched at p: T >= max(sum t_0, L + Tc) (nothing can beat
    all-SM compute, comm cannot start before p) and T <= L + max(Tc, A_sigma[N] -
    A_sigma[p]) (running everything after p in the slowed state is never faster)."""
    w = I.config_workload(0)
    sp = w.space
    T, E = oracle_lib.evaluate_partition(sp, w.t, w.pw, w.tc, w.pc, 1)
    for f in range(sp.n_freq):
        t = w.t[1, f]
        for p in range(sp.n_pos):
            for s in range(sp.n_sm):
                c = _single(sp, w, f, p, s)
                L = t[:p, 0].sum()
                tc = w.tc[1, f, 0, s]
                lo = max(t[:, 0].sum(), L + tc)
                hi = L + max(tc, t[p:, s + 1].sum())
                assert lo * (1 - 1e-12) <= T[c] <= hi * (1 + 1e-12)


def test_energy_is_static_times_time_plus_dynamic(oracle_lib):
    """Section 2.3: total = static power x time + dynamic.  The oracle's energy is
    affine in static power with slope T, and linear in the dynamic power tables."""
    w = I.config_workload(0)
    sp = w.space
    import dataclasses

    z = dataclasses.replace(sp, p_static=0.0)
    T1, E1 = oracle_lib.evaluate_partition(sp, w.t, w.pw, w.tc, w.pc, 2)
    T0, E0 = oracle_lib.evaluate_partition(z, w.t, w.pw, w.tc, w.pc, 2)
    np.testing.assert_array_equal(T1, T0)
    np.testing.assert_allclose(E1 - E0, sp.p_static * T1, rtol=1e-9)
    T2, E2 = oracle_lib.evaluate_partition(z, w.t, 2.0 * w.pw, w.tc, 2.0 * w.pc, 2)
    np.testing.assert_allclose(E2, 2.0 * E0, rtol=1e-12)
    Tn, En = oracle_lib.evaluate_partition(z, w.t, 0.0 * w.pw, w.tc, 0.0 * w.pc, 2)
    np.testing.assert_array_equal(En, 0.0)


def test_paper_energy_breakdown_table():
    """The printed table satisfies the same decomposition: one static power (about
    60 W per GPU on 16 GPUs) explains every row's static energy within print rounding,
    and static + dynamic = total within 1 J."""
    rows = []
    with open(os.path.join(GOLDEN, "energy_breakdown_table.txt")) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            name, t, st, dy, tot = line.split()
            rows.append((float(t), float(st), float(dy), float(tot)))
    lo, hi = 0.0, np.inf
    for t, st, dy, tot in rows:
        assert abs(st + dy - tot) <= 1.0
        # static in [st-0.5, st+0.5], time in [t-0.005, t+0.005]
        lo = max(lo, (st - 0.5) / (t + 0.005))
        hi = min(hi, (st + 0.5) / (t - 0.005))
    assert lo <= hi, "no single static power explains the table"
    per_gpu = 0.5 * (lo + hi) / 16
    assert 59.0 < per_gpu < 61.0
