"""GPU parity: the HIP library (through its C ABI) against the CPU oracle, element by
element, on the same seeded inputs.

Bars: frontier index sets, chosen candidates, offsets and back-pointers bit-exact;
T and E within 1e-9 relative (fp64); composed energies within 1e-6 relative.  With
identical fp64 operation orders on both sides the values are expected to agree bit
for bit, and the tests also report how many do not.
"""

import dataclasses
import os

import numpy as np
import pytest
import torch

from paper_2601_17654_amd import inputs as I

pytestmark = pytest.mark.gpu

RT_TE = 1e-9
RT_MINPLUS = 1e-6


@pytest.fixture(scope="module")
def kr():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2601_17654_amd import binding

    return binding


_cache = {}


def workload(cfg, parts=None):
    key = (cfg, None if parts is None else (parts.start, parts.stop))
    if key not in _cache:
        _cache[key] = I.config_workload(cfg, parts=parts)
    return _cache[key]


def dev_tables(w):
    return [torch.from_numpy(getattr(w, k)).cuda() for k in ("t", "pw", "tc", "pc")]


def assert_close(got, ref, rtol, what):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, what
    np.testing.assert_allclose(got, ref, rtol=rtol, atol=0, err_msg=what)
    diff = int(np.count_nonzero(got != ref))
    if diff:
        print("%s: %d of %d values not bit-identical (within rtol %g)" % (what, diff, got.size, rtol))


def check_frontier(fr, part, ref, what):
    """fr: binding.Frontier on host numpy; ref = (idx, T, E) of the oracle."""
    off = fr.off.cpu().numpy()
    lo, hi = int(off[part]), int(off[part + 1])
    idx = fr.idx.cpu().numpy()[lo:hi]
    np.testing.assert_array_equal(idx, ref[0], err_msg=what + " idx")
    assert_close(fr.T.cpu().numpy()[lo:hi], ref[1], RT_TE, what + " T")
    assert_close(fr.E.cpu().numpy()[lo:hi], ref[2], RT_TE, what + " E")


def small_spaces():
    rng = np.random.default_rng(77)
    spaces = []
    for i in range(10):
        spaces.append(I.random_space(rng, n_comm=1 + (i % 2), max_kernels=8, max_sm=5,
                                     max_freq=3, n_parts=3))
    # edge shapes: one kernel, one position, one SM choice, one frequency; n_pos = N + 1
    spaces.append(I.Space(2, 1, 1, 1, (8,), (1500.0,)))
    spaces.append(I.Space(2, 1, 2, 2, (8, 16), (1500.0,)))
    spaces.append(I.Space(2, 9, 1, 10, (1, 2, 3), (1005.0, 1980.0)))
    spaces.append(I.Space(2, 9, 2, 10, (1, 32), (1005.0, 1980.0)))
    # more SM choices than half a wave: one run of 33 positions per lane, evaluated as
    # two register chunks per frequency
    spaces.append(I.Space(2, 32, 1, 33, tuple(range(1, 41)), (1005.0, 1500.0, 1980.0)))
    spaces.append(I.Space(2, 32, 1, 33, tuple(range(2, 98, 2)), (1005.0, 1980.0)))
    # two comm kernels beyond the one-wave kernel's reach (more than 8 SM choices, or a
    # slab whose tables do not fit its LDS): the block-per-slab kernel
    spaces.append(I.Space(2, 9, 2, 10, tuple(range(1, 10)), (1005.0, 1980.0)))
    spaces.append(I.Space(2, 6, 2, 7, tuple(range(2, 26, 2)), (1500.0,)))
    spaces.append(I.Space(1, 206, 2, 5, tuple(range(2, 18, 2)), (1500.0,)))
    return spaces


@pytest.mark.parametrize("case", range(19))
@pytest.mark.parametrize("tc_scale", [1.0, 1e-3, 1e3])
def test_evaluate_small_spaces(kr, oracle_lib, case, tc_scale):
    space = small_spaces()[case]
    tab = I.make_tables(space, seed=case, comm_bytes=(4e6, 64e6))
    tab["tc"] = tab["tc"] * tc_scale
    d = [torch.from_numpy(tab[k]).cuda() for k in ("t", "pw", "tc", "pc")]
    T, E = kr.evaluate_partition(space, *d)
    fr = kr.evaluate_and_filter(space, *d)
    T, E = T.cpu().numpy(), E.cpu().numpy()
    for p in range(space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], p)
        assert_close(T[p], Tr, RT_TE, "T case %d part %d" % (case, p))
        assert_close(E[p], Er, RT_TE, "E case %d part %d" % (case, p))
        ix = oracle_lib.pareto(Tr, Er)
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "frontier case %d part %d" % (case, p))


def quantised_tables(space, seed):
    """Tables with many exact ties and zeros: times on a coarse binary grid (kernels of
    equal length), powers of 0, 100 or 200 W, comm times of 0 for some SM choices and
    comm powers of 0 for others."""
    rng = np.random.default_rng(seed)
    tab = I.make_tables(space, seed=seed, comm_bytes=(4e6, 64e6))
    tab["t"] = rng.integers(1, 5, tab["t"].shape) * 2.0 ** -12
    tab["pw"] = rng.integers(0, 3, tab["pw"].shape) * 100.0
    tc = rng.integers(0, 4, tab["tc"].shape) * 2.0 ** -11
    tc[..., ::3] = 0.0
    tab["tc"] = tc
    pc = rng.integers(0, 3, tab["pc"].shape) * 50.0
    pc[..., 1::4] = 0.0
    tab["pc"] = pc
    return tab


@pytest.mark.parametrize("case", range(4))
def test_evaluate_degenerate_tables(kr, oracle_lib, case):
    """Exact ties everywhere (equal kernels, equal comm times, zero powers and zero comm
    times) on each evaluation kernel: the one-comm wave kernel, the two-comm pair kernel,
    and the block kernel for each comm count.  Time and energy match the oracle and the
    frontier indices (smallest index among exact duplicates) are bit-exact."""
    space = [I.Space(3, 12, 1, 13, tuple(range(1, 17)), (1005.0, 1500.0, 1980.0)),
             I.Space(3, 9, 2, 10, (4, 8, 12, 16), (1005.0, 1980.0)),
             I.Space(2, 7, 2, 8, tuple(range(1, 10)), (1500.0,)),
             I.Space(2, 5, 1, 6, tuple(range(1, 70)), (1500.0, 1980.0))][case]
    tab = quantised_tables(space, 40 + case)
    d = [torch.from_numpy(tab[k]).cuda() for k in ("t", "pw", "tc", "pc")]
    T, E = kr.evaluate_partition(space, *d)
    fr = kr.evaluate_and_filter(space, *d)
    T, E = T.cpu().numpy(), E.cpu().numpy()
    for p in range(space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], p)
        assert_close(T[p], Tr, RT_TE, "T case %d part %d" % (case, p))
        assert_close(E[p], Er, RT_TE, "E case %d part %d" % (case, p))
        ix = oracle_lib.pareto(Tr, Er)
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "frontier case %d part %d" % (case, p))


@pytest.mark.parametrize("cfg", [0, 1])
def test_evaluate_and_filter_full(kr, oracle_lib, cfg):
    w = workload(cfg)
    d = dev_tables(w)
    T, E = kr.evaluate_partition(w.space, *d)
    fr = kr.evaluate_and_filter(w.space, *d)
    T, E = T.cpu().numpy(), E.cpu().numpy()
    ref = oracle_lib.evaluate_and_filter(w.space, w.t, w.pw, w.tc, w.pc)
    for p in range(w.space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(w.space, w.t, w.pw, w.tc, w.pc, p)
        assert_close(T[p], Tr, RT_TE, "cfg%d T part %d" % (cfg, p))
        assert_close(E[p], Er, RT_TE, "cfg%d E part %d" % (cfg, p))
        check_frontier(fr, p, ref[p], "cfg%d part %d" % (cfg, p))


@pytest.mark.parametrize("cfg,parts", [(2, range(0, 2)), (2, range(255, 256)),
                                       (3, range(0, 8)), (3, range(1020, 1024))])
def test_evaluate_sampled_partitions(kr, oracle_lib, cfg, parts):
    """Unfused evaluation on a sub-batch (the tables are those of the full batch)."""
    w = workload(cfg, parts)
    T, E = kr.evaluate_partition(w.space, *dev_tables(w))
    T, E = T.cpu().numpy(), E.cpu().numpy()
    for p in range(len(parts)):
        Tr, Er = oracle_lib.evaluate_partition(w.space, w.t, w.pw, w.tc, w.pc, p)
        assert_close(T[p], Tr, RT_TE, "cfg%d T part %d" % (cfg, parts.start + p))
        assert_close(E[p], Er, RT_TE, "cfg%d E part %d" % (cfg, parts.start + p))


def test_evaluate_and_filter_eval_stress_all(kr, oracle_lib):
    """The fused kernel at the eval-stress batch size, in the benchmark's launch
    configuration (several frequencies per block, so the staging of the next slab
    during the current one runs), against the oracle on every partition."""
    w = workload(3)
    fr = kr.evaluate_and_filter(w.space, *dev_tables(w))
    ref = oracle_lib.evaluate_and_filter(w.space, w.t, w.pw, w.tc, w.pc)
    off = fr.off.cpu().numpy()
    idx, T, E = fr.idx.cpu().numpy(), fr.T.cpu().numpy(), fr.E.cpu().numpy()
    assert off[-1] == sum(len(r[0]) for r in ref), "total frontier points"
    for p in range(w.space.n_parts):
        lo, hi = int(off[p]), int(off[p + 1])
        np.testing.assert_array_equal(idx[lo:hi], ref[p][0], err_msg="eval-stress part %d" % p)
        assert_close(T[lo:hi], ref[p][1], RT_TE, "eval-stress part %d T" % p)
        assert_close(E[lo:hi], ref[p][2], RT_TE, "eval-stress part %d E" % p)


@pytest.mark.parametrize("cfg,sample", [(3, [0, 1, 333, 512, 1023]), (2, [0, 131, 255])])
def test_evaluate_and_filter_full_size_sampled(kr, oracle_lib, cfg, sample):
    """The fused kernel at the full batch size (the benchmark's launch), checked on
    sampled partitions; every partition's output is a strict staircase."""
    w = workload(cfg)
    fr = kr.evaluate_and_filter(w.space, *dev_tables(w))
    for p in sample:
        Tr, Er = oracle_lib.evaluate_partition(w.space, w.t, w.pw, w.tc, w.pc, p)
        ix = oracle_lib.pareto(Tr, Er)
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "cfg%d part %d" % (cfg, p))
    off = fr.off.cpu().numpy()
    T, E, idx = fr.T.cpu().numpy(), fr.E.cpu().numpy(), fr.idx.cpu().numpy()
    C = w.space.n_cand
    for p in range(w.space.n_parts):
        lo, hi = off[p], off[p + 1]
        assert hi > lo
        assert np.all(np.diff(T[lo:hi]) > 0) and np.all(np.diff(E[lo:hi]) < 0)
        assert idx[lo:hi].min() >= 0 and idx[lo:hi].max() < C


def test_fused_equals_unfused(kr):
    w = workload(1)
    d = dev_tables(w)
    T, E = kr.evaluate_partition(w.space, *d)
    C = w.space.n_cand
    seg = np.arange(w.space.n_parts + 1, dtype=np.int64) * C
    a = kr.pareto_filter(T, E, seg)
    b = kr.evaluate_and_filter(w.space, *d)
    for x, y in ((a.off, b.off), (a.idx, b.idx), (a.T, b.T), (a.E, b.E)):
        assert torch.equal(x, y)


def _tied(rng, n):
    T = rng.integers(1, 40, size=n).astype(np.float64) * 0.125
    E = rng.integers(1, 40, size=n).astype(np.float64) * 0.25
    dup = rng.integers(0, max(n, 1), size=n // 8)
    if len(dup):
        T[dup] = T[dup[0]]
        E[dup] = E[dup[0]]
    return T, E


@pytest.mark.parametrize("kind", ["tied", "continuous", "staircase", "mixed-lengths",
                                  "many-segments"])
def test_pareto_filter(kr, oracle_lib, kind):
    rng = np.random.default_rng({"tied": 1, "continuous": 2, "staircase": 3,
                                 "many-segments": 5}.get(kind, 4))
    if kind == "many-segments":  # more segments than one output block scans for itself
        lens = list(rng.integers(0, 24, size=5000))
    elif kind == "tied":
        lens = [0, 1, 2, 7, 2047, 2048, 2049, 5000, 0, 12345]
    elif kind == "continuous":
        lens = [100000, 3, 65536, 1]
    elif kind == "staircase":
        lens = [9000, 4096, 1]  # every point survives: large runs through every merge level
    else:
        lens = list(rng.integers(0, 9000, size=40))
    Ts, Es = [], []
    for n in lens:
        if kind == "tied":
            T, E = _tied(rng, n)
        elif kind == "staircase":
            T = np.sort(rng.uniform(1.0, 2.0, size=n))
            T = np.unique(T)
            T = np.concatenate([T, 3.0 + np.arange(n - len(T))])
            E = 10.0 - np.arange(n) * 1e-3
            perm = rng.permutation(n)
            T, E = T[perm], E[perm]
        else:
            T = rng.lognormal(size=n)
            E = 1.0 / T + rng.random(n)
        Ts.append(T)
        Es.append(E)
    seg = np.zeros(len(lens) + 1, dtype=np.int64)
    seg[1:] = np.cumsum(lens)
    T = np.concatenate(Ts) if Ts else np.zeros(0)
    E = np.concatenate(Es) if Es else np.zeros(0)
    fr = kr.pareto_filter(torch.from_numpy(T).cuda(), torch.from_numpy(E).cuda(), seg)
    for g in range(len(lens)):
        Tg, Eg = T[seg[g]:seg[g + 1]], E[seg[g]:seg[g + 1]]
        ix = oracle_lib.pareto(Tg, Eg)
        check_frontier(fr, g, (ix, Tg[ix], Eg[ix]), "%s seg %d (n=%d)" % (kind, g, lens[g]))


@pytest.mark.parametrize("n_below", [0, 1, 255, 256, 257, 1000, 2047])
def test_pareto_filter_tile_survivor_paths(kr, oracle_lib, n_below):
    """One 2,048-point tile whose least-time point A has n_below points with lower energy.
    Up to 256 such survivors take the LDS survivor list; more defer the tile to the
    second pass, which sorts them.  Half of the survivors are dominated by others, and
    a second tile of the segment is all on one staircase."""
    rng = np.random.default_rng(500 + n_below)
    n = 2048
    T = 1.0 + rng.permutation(n).astype(np.float64)  # distinct; A is the point with T = 1
    E = np.empty(n)
    a = int(np.argmin(T))
    E[a] = 100.0
    others = np.delete(np.arange(n), a)
    pick = rng.choice(others, n_below, replace=False)
    E[others] = rng.uniform(100.0, 200.0, n - 1)  # at or above A: never kept
    E[pick] = rng.uniform(1.0, 99.0, n_below)
    T2 = np.sort(rng.uniform(5000.0, 6000.0, 900))
    E2 = np.linspace(50.0, 1.0, 900)
    T, E = np.concatenate([T, T2]), np.concatenate([E, E2])
    seg = np.array([0, len(T)], dtype=np.int64)
    fr = kr.pareto_filter(torch.from_numpy(T).cuda(), torch.from_numpy(E).cuda(), seg)
    ix = oracle_lib.pareto(T, E)
    check_frontier(fr, 0, (ix, T[ix], E[ix]), "tile survivors %d" % n_below)


def test_pareto_filter_capacity(kr):
    T = torch.linspace(1.0, 2.0, 5000, dtype=torch.float64).cuda()
    E = torch.linspace(2.0, 1.0, 5000, dtype=torch.float64).cuda()
    seg = np.array([0, 5000], dtype=np.int64)
    fr = kr.pareto_filter(T, E, seg, cap=100, sync=False)
    torch.cuda.synchronize()
    assert int(fr.off[-1]) == 5000  # the required size is reported
    assert torch.equal(fr.idx[:100].cpu(), torch.arange(100, dtype=torch.int32))
    fr = kr.pareto_filter(T, E, seg)  # grows its capacity and retries
    assert fr.idx.numel() == 5000
    # several segments, the capacity ending inside the second: the entries up to it match
    # the uncapped output and the offsets are complete
    seg = np.array([0, 2000, 3000, 5000], dtype=np.int64)
    full = kr.pareto_filter(T, E, seg)
    part = kr.pareto_filter(T, E, seg, cap=2500, sync=False)
    torch.cuda.synchronize()
    assert torch.equal(part.off.cpu(), full.off.cpu())
    for x, y in ((part.idx, full.idx), (part.T, full.T), (part.E, full.E)):
        assert torch.equal(x[:2500].cpu(), y[:2500].cpu())


def compare_composed(kr, comp, ref, off, T, E, what):
    assert int(comp.status.item()) == 0
    info = comp.info.cpu().numpy()
    assert info[0] == ref.delta and info[1] == ref.tmin_sum, what
    assert int(comp.L.item()) == ref.L
    assert_close(comp.F.cpu().numpy(), ref.F, RT_MINPLUS, what + " F")
    np.testing.assert_array_equal(comp.pt_bin.cpu().numpy()[:len(ref.pt_bin)], ref.pt_bin)
    np.testing.assert_array_equal(comp.bp.cpu().numpy(), ref.bp, err_msg=what + " bp")
    # the recorded offsets are the chosen points' offsets in the oracle's binning
    want = np.full(ref.bp.shape, -1, dtype=np.int64)
    for k in range(ref.bp.shape[0]):
        sel = ref.bp[k] >= 0
        want[k, sel] = ref.pt_bin[off[k] + ref.bp[k, sel]]
    np.testing.assert_array_equal(comp.bp_off.cpu().numpy(), want, err_msg=what + " bp_off")


@pytest.fixture(scope="module")
def config4():
    return I.compose_frontiers()


def test_compose_config4(kr, oracle_lib, config4):
    off, T, E = config4
    B = I.COMPOSE_SPACE["bins"]
    comp = kr.compose_frontiers(torch.from_numpy(off).cuda(), torch.from_numpy(T).cuda(),
                                torch.from_numpy(E).cuda(), B)
    ref = oracle_lib.compose(off, T, E, B)
    compare_composed(kr, comp, ref, off, T, E, "cfg4")
    sb, st, se = comp.staircase()
    rb, rt, re_ = oracle_lib.staircase(ref.F, ref.delta, ref.tmin_sum)
    np.testing.assert_array_equal(sb.cpu().numpy(), rb)
    assert_close(st.cpu().numpy(), rt, RT_TE, "cfg4 stair T")
    assert_close(se.cpu().numpy(), re_, RT_MINPLUS, "cfg4 stair E")
    # schedules behind every staircase bin and some other reachable bins
    reach = np.flatnonzero(np.isfinite(ref.F))
    rng = np.random.default_rng(4)
    bins = np.concatenate([rb, rng.choice(reach, size=24, replace=False), [ref.L, B - 1]])
    ch, _, Ts, Es, ok = kr.extract_schedule(comp, off, T, E, torch.from_numpy(
        bins.astype(np.int32)).cuda())
    ch, Ts, Es, ok = ch.cpu().numpy(), Ts.cpu().numpy(), Es.cpu().numpy(), ok.cpu().numpy()
    for q, b in enumerate(bins):
        if b >= ref.L or not np.isfinite(ref.F[b]):
            assert ok[q] == 0
            continue
        rc, rts, res = oracle_lib.extract(off, T, E, ref, int(b))
        assert ok[q] == 1
        np.testing.assert_array_equal(ch[q], rc)
        assert_close(Ts[q], rts, RT_TE, "extract T bin %d" % b)
        assert_close(Es[q], res, RT_TE, "extract E bin %d" % b)


ORACLE_THREADS = min(16, os.cpu_count() or 1)


@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_end_to_end_path(kr, oracle_lib, cfg):
    """Tables -> fused frontiers of every partition -> composition -> staircase ->
    extracted schedule of every staircase bin -> decoded (positions, SM choices,
    frequency), against the oracle run on the same tables (partition-parallel over the
    host's cores; each partition is the plain single-threaded oracle)."""
    w = workload(cfg)
    sp = w.space
    print("end-to-end cfg %d: %d partitions" % (cfg, sp.n_parts), flush=True)
    fr = kr.evaluate_and_filter(sp, *dev_tables(w))
    ref_fr = oracle_lib.evaluate_and_filter(sp, w.t, w.pw, w.tc, w.pc, threads=ORACLE_THREADS)
    off = fr.off.cpu().numpy()
    gidx, gT, gE = fr.idx.cpu().numpy(), fr.T.cpu().numpy(), fr.E.cpu().numpy()
    for p in range(sp.n_parts):
        lo, hi = int(off[p]), int(off[p + 1])
        np.testing.assert_array_equal(gidx[lo:hi], ref_fr[p][0], err_msg="cfg%d part %d" % (cfg, p))
        assert_close(gT[lo:hi], ref_fr[p][1], RT_TE, "cfg%d part %d T" % (cfg, p))
        assert_close(gE[lo:hi], ref_fr[p][2], RT_TE, "cfg%d part %d E" % (cfg, p))
    roff = np.zeros(sp.n_parts + 1, dtype=np.int64)
    roff[1:] = np.cumsum([len(x[0]) for x in ref_fr])
    np.testing.assert_array_equal(off, roff)
    rT = np.concatenate([x[1] for x in ref_fr])
    rE = np.concatenate([x[2] for x in ref_fr])
    ridx = np.concatenate([x[0] for x in ref_fr])
    comp = kr.compose_frontiers(fr.off, fr.T, fr.E, w.bins)
    ref = oracle_lib.compose(roff, rT, rE, w.bins)
    compare_composed(kr, comp, ref, roff, rT, rE, "cfg%d" % cfg)
    sb, st, se = comp.staircase()
    rb, rt, re_ = oracle_lib.staircase(ref.F, ref.delta, ref.tmin_sum)
    np.testing.assert_array_equal(sb.cpu().numpy(), rb)
    assert_close(st.cpu().numpy(), rt, RT_TE, "cfg%d stair T" % cfg)
    assert_close(se.cpu().numpy(), re_, RT_MINPLUS, "cfg%d stair E" % cfg)
    ch, cc, Ts, Es, ok = kr.extract_schedule(comp, fr.off, fr.T, fr.E, sb, cand_idx=fr.idx)
    assert ok.cpu().numpy().all()
    ch, cc, Ts, Es = ch.cpu().numpy(), cc.cpu().numpy(), Ts.cpu().numpy(), Es.cpu().numpy()
    rch = np.empty_like(ch)
    rts, res = np.empty(len(rb)), np.empty(len(rb))
    for q, b in enumerate(rb):
        rch[q], rts[q], res[q] = oracle_lib.extract(roff, rT, rE, ref, int(b))
    np.testing.assert_array_equal(ch, rch, err_msg="cfg%d extracted choices" % cfg)
    assert_close(Ts, rts, RT_TE, "cfg%d extracted T" % cfg)
    assert_close(Es, res, RT_TE, "cfg%d extracted E" % cfg)
    # the candidates behind every choice, decoded on the GPU and by the oracle
    pts = roff[:-1][None, :] + rch  # frontier point of every (query, partition)
    np.testing.assert_array_equal(cc, ridx[pts], err_msg="cfg%d chosen candidates" % cfg)
    f, pos, sm = kr.decode_candidates(sp, torch.from_numpy(cc.reshape(-1)).cuda())
    f, pos, sm = f.cpu().numpy(), pos.cpu().numpy(), sm.cpu().numpy()
    M = sp.n_comm
    df = np.full(len(ridx), -1)
    dpos = np.full((len(ridx), M), -1)
    dsm = np.full((len(ridx), M), -1)
    for x in np.unique(pts):  # the oracle's decode of every point some choice uses
        df[x], dpos[x], dsm[x] = oracle_lib.decode(sp, int(ridx[x]))
    flat = pts.reshape(-1)
    np.testing.assert_array_equal(f, df[flat], err_msg="cfg%d decoded frequency" % cfg)
    np.testing.assert_array_equal(pos.reshape(-1, M), dpos[flat],
                                  err_msg="cfg%d decoded positions" % cfg)
    np.testing.assert_array_equal(sm.reshape(-1, M), dsm[flat],
                                  err_msg="cfg%d decoded SM choices" % cfg)


def test_compose_wavefront_modes(kr, oracle_lib):
    """The min-plus wavefront's record formats and modes against the oracle: occupied
    offsets only (few points over wide spans), a partition wider than the on-chip window,
    and more steps than two chunks of the per-block step metadata."""
    rng = np.random.default_rng(17)
    cases = []
    n = rng.integers(2, 7, 48)
    cases.append(("sparse", n, rng.uniform(1e-3, 1e-2, 48), 16384))
    n = rng.integers(20, 60, 6)
    n[2] = 3000  # more points than the walk stages per partition
    span = rng.uniform(1e-3, 2e-3, 6)
    span[2] = 0.08  # offsets wider than the window and than the walk's look-ahead
    cases.append(("wide", n, span, 8192))
    n = rng.integers(10, 31, 1300)
    cases.append(("long", n, rng.uniform(0.5e-3, 1.5e-3, 1300), 32768))
    # more partitions than the extraction keeps in LDS (the walk that reads offsets and
    # choices from memory)
    n = rng.integers(1, 4, 2100)
    cases.append(("many", n, rng.uniform(1e-5, 2e-5, 2100), 8192))
    for i, (what, n, span, B) in enumerate(cases):
        off, T, E = I.frontier_batch(100 + i, n.tolist(), span.tolist())
        print("compose wavefront case", what, flush=True)
        comp = kr.compose_frontiers(torch.from_numpy(off).cuda(), torch.from_numpy(T).cuda(),
                                    torch.from_numpy(E).cuda(), B)
        ref = oracle_lib.compose(off, T, E, B)
        compare_composed(kr, comp, ref, off, T, E, what)
        # schedules behind the staircase and some other reachable bins
        sb, _, _ = comp.staircase()
        reach = np.flatnonzero(np.isfinite(ref.F))
        bins = np.concatenate([sb.cpu().numpy(), rng.choice(reach, size=8, replace=False),
                               [B - 1]]).astype(np.int32)
        ch, _, Ts, Es, ok = kr.extract_schedule(comp, off, T, E, torch.from_numpy(bins).cuda())
        ch, Ts, Es, ok = ch.cpu().numpy(), Ts.cpu().numpy(), Es.cpu().numpy(), ok.cpu().numpy()
        alt = kr.extract_schedule(comp, off, T, E, torch.from_numpy(bins).cuda(),
                                  use_offsets=False)  # the point-lookup walk: the same
        for x, y in zip((ch, Ts, Es, ok), (alt[0], alt[2], alt[3], alt[4])):
            np.testing.assert_array_equal(x.view(np.uint8), y.cpu().numpy().view(np.uint8))
        for q, bq in enumerate(bins):
            if bq >= ref.L or not np.isfinite(ref.F[bq]):
                assert ok[q] == 0
                continue
            rc, rts, res = oracle_lib.extract(off, T, E, ref, int(bq))
            assert ok[q] == 1, (what, int(bq))
            np.testing.assert_array_equal(ch[q], rc)
            assert_close(Ts[q], rts, RT_TE, "%s extract T bin %d" % (what, bq))
            assert_close(Es[q], res, RT_TE, "%s extract E bin %d" % (what, bq))


def test_compose_edge_cases(kr, oracle_lib):
    cases = []
    rng = np.random.default_rng(11)
    # one partition
    cases.append((np.array([0, 50]), rng.uniform(1e-3, 2e-3, 50), rng.uniform(1, 2, 50), 16, 0.0))
    # single-point partitions: zero range
    cases.append((np.array([0, 1, 2, 3]), np.array([1e-3, 2e-3, 3e-3]), np.array([1., 2., 3.]),
                  4, 0.0))
    # exact ties everywhere
    n = [5, 7, 3, 9]
    off = np.concatenate([[0], np.cumsum(n)])
    cases.append((off, rng.integers(0, 6, off[-1]) * 1e-3 + 1e-3,
                  rng.integers(1, 4, off[-1]) * 0.25, 40, 0.0))
    # a caller-given width
    cases.append((off, rng.uniform(1e-3, 4e-3, off[-1]), rng.uniform(1, 2, off[-1]), 64, 2.5e-4))
    # dense min-plus steps with exact ties: times on a binary grid with the bin width as
    # its step, offset ranges M_k of 128, 122, 64, 200 and 5 (full groups of 8 offsets
    # with and without leftovers), energies on a coarse grid
    spans = [128, 122, 64, 200, 5] * 4
    Ts, Es = [], []
    for m in spans:
        k = rng.integers(0, m + 1, 90)
        k[:2] = (0, m)
        Ts.append((k + 3) * 2.0 ** -10)
        Es.append(rng.integers(1, 6, 90) * 0.25)
    offd = np.concatenate([[0], np.cumsum([len(x) for x in Ts])])
    cases.append((offd, np.concatenate(Ts), np.concatenate(Es), sum(spans) + 8, 2.0 ** -10))
    for i, (off, T, E, B, delta) in enumerate(cases):
        off = off.astype(np.int64)
        comp = kr.compose_frontiers(torch.from_numpy(off).cuda(), torch.from_numpy(T).cuda(),
                                    torch.from_numpy(E).cuda(), B, delta=delta)
        ref = oracle_lib.compose(off, T, E, B, delta=delta)
        compare_composed(kr, comp, ref, off, T, E, "edge %d" % i)
    # a caller-given width that needs too many bins: reported on the device
    off = np.array([0, 3], dtype=np.int64)
    comp = kr.compose_frontiers(torch.from_numpy(off).cuda(),
                                torch.tensor([0.001, 1.0, 2.0], dtype=torch.float64).cuda(),
                                torch.tensor([3.0, 2.0, 1.0], dtype=torch.float64).cuda(), 2,
                                delta=0.5)
    assert int(comp.status.item()) == kr.KR_ECAPACITY
    assert int(comp.n_stair.item()) == 0


def window_hits(bp_off, b, D=16, W=512):
    """(hits, misses) of the offset walk's register windows for a walk from bin b: the
    placement rules of the walk kernel (a window of W bins per row, loaded D rows
    ahead, placed below the bin by the offsets of the last D rows), replayed on the
    host so that a test can show it reaches both the window reads and the direct
    loads."""
    P, B = bp_off.shape
    total = P * B
    base = [0] * D

    def place(d, r0, bk, drift):
        x0 = min(max(r0 + min(bk - drift - W // 2, bk - (W - 1)), 0), total - W)
        base[d] = x0 - r0

    hist = [b] * D
    for d in range(D):
        place(d, max(P - 1 - d, 0) * B, b, d * (b // max(P, 1)))
    hits = misses = 0
    for k in range(P - 1, -1, -1):
        d = (P - 1 - k) % D
        if 0 <= b - base[d] < W:
            hits += 1
        else:
            misses += 1
        b = b - int(bp_off[k, b])
        drift, hist[d] = hist[d] - b, b
        place(d, (k - D) * B, b, drift)
    return hits, misses


def test_extract_walks(kr, oracle_lib, config4):
    """Both schedule walks against the oracle: over the recorded offsets with windows
    read rows ahead (query bins spread over the whole axis, so windows both hit and
    miss), and with each chosen point's offset looked up (Section 5.1)."""
    rng = np.random.default_rng(23)
    cases = [("cfg4",) + tuple(config4) + (I.COMPOSE_SPACE["bins"],)]
    n = rng.integers(20, 60, 40)
    n[[2, 25]] = 3000
    span = rng.uniform(1e-3, 2e-3, 40)
    span[[2, 25]] = 0.04  # offsets wider than a window
    cases.append(("wide",) + tuple(I.frontier_batch(101, n.tolist(), span.tolist())) + (8192,))
    # one partition: the walk is the last-rows path alone (table of exactly one window)
    cases.append(("one",) + tuple(I.frontier_batch(102, [300], [1e-3])) + (512,))
    # a table smaller than a window: the point-lookup walk
    cases.append(("tiny", np.array([0, 2, 5], dtype=np.int64), np.array([1e-3, 2e-3, 1e-3, 3e-3,
                  5e-3]), np.array([2.0, 1.0, 3.0, 2.0, 1.0]), 4))
    hm_all = np.zeros(2, dtype=np.int64)
    for what, off, T, E, B in cases:
        print("extract walks case", what, flush=True)
        Td, Ed, od = torch.from_numpy(T).cuda(), torch.from_numpy(E).cuda(), torch.from_numpy(off).cuda()
        comp = kr.compose_frontiers(od, Td, Ed, B)
        ref = oracle_lib.compose(off, T, E, B)
        reach = np.flatnonzero(np.isfinite(ref.F))
        rb, _, _ = oracle_lib.staircase(ref.F, ref.delta, ref.tmin_sum)
        bins = np.concatenate([rb[:40], rb[-40:], rng.choice(reach, size=min(24, len(reach)),
                               replace=False), [0, ref.L - 1, B - 1]]).astype(np.int32)
        outs = [kr.extract_schedule(comp, od, Td, Ed, torch.from_numpy(bins).cuda(),
                                    use_offsets=u) for u in (True, False)]
        outs = [[x.cpu().numpy() for x in (o[0], o[2], o[3], o[4])] for o in outs]
        for x, y in zip(outs[0], outs[1]):  # the two walks agree bit for bit
            np.testing.assert_array_equal(x.view(np.uint8), y.view(np.uint8), err_msg=what)
        ch, Ts, Es, ok = outs[0]
        if what in ("cfg4", "wide"):  # walks that read windows and load directly
            bo = comp.bp_off.cpu().numpy()
            hm = np.array([window_hits(bo, int(bq)) for bq in bins if bq < ref.L and
                           np.isfinite(ref.F[bq])]).sum(axis=0)
            print("window hits, misses:", hm, flush=True)
            hm_all += hm
        for q, bq in enumerate(bins):
            live = bq < ref.L and np.isfinite(ref.F[bq])
            assert ok[q] == int(live), (what, int(bq))
            if live:
                rc, rts, res = oracle_lib.extract(off, T, E, ref, int(bq))
                np.testing.assert_array_equal(ch[q], rc, err_msg="%s bin %d" % (what, bq))
                assert_close(Ts[q], rts, RT_TE, "%s extract T bin %d" % (what, bq))
                assert_close(Es[q], res, RT_TE, "%s extract E bin %d" % (what, bq))
            else:
                assert (ch[q] == -1).all()
    assert hm_all[0] > 0 and hm_all[1] > 0, hm_all


def test_decode(kr, oracle_lib):
    for sp in (I.SPACES[0]["space"], I.SPACES[2]["space"], I.SPACES[3]["space"]):
        rng = np.random.default_rng(sp.n_kernels)
        idx = rng.integers(0, sp.n_cand, size=500).astype(np.int32)
        f, pos, sm = kr.decode_candidates(sp, torch.from_numpy(idx).cuda())
        f, pos, sm = f.cpu().numpy(), pos.cpu().numpy(), sm.cpu().numpy()
        for q, c in enumerate(idx):
            rf, rpos, rsm = oracle_lib.decode(sp, int(c))
            assert (f[q], tuple(pos[q]), tuple(sm[q])) == (rf, rpos, rsm)


def test_deterministic(kr, config4):
    w = workload(1)
    d = dev_tables(w)
    a = kr.evaluate_and_filter(w.space, *d)
    b = kr.evaluate_and_filter(w.space, *d)
    assert torch.equal(a.idx, b.idx) and torch.equal(a.T, b.T) and torch.equal(a.E, b.E)
    off, T, E = (torch.from_numpy(x).cuda() for x in config4)
    c1 = kr.compose_frontiers(off, T, E, 65536)
    F1, bp1 = c1.F.clone(), c1.bp.clone()
    c2 = kr.compose_frontiers(off, T, E, 65536)
    assert torch.equal(F1, c2.F) and torch.equal(bp1, c2.bp)


def test_adversarial_frontiers(kr, oracle_lib):
    """Comm time dominating and comm energy falling steeply with comm time: almost every
    candidate beats the fastest one's energy (more survivors than the on-chip list
    holds) and the frontiers run to thousands of points (more than the finalize step
    sorts on chip), so every fallback path runs."""
    space = I.Space(2, 4, 1, 5, tuple(range(1, 65)), tuple(1005.0 + 15.0 * j for j in range(64)),
                    p_static=0.0)
    tab = I.make_tables(space, seed=21, comm_bytes=(4e6, 64e6))
    F, S = space.n_freq, space.n_sm
    tc = 10.0 + 1e-3 * np.arange(F * S, dtype=np.float64).reshape(F, S)
    tab["tc"] = np.broadcast_to(tc[None, :, None, :], tab["tc"].shape).copy()
    tab["pc"] = np.broadcast_to((1e6 / tc ** 2)[None, :, None, :], tab["pc"].shape).copy()
    d = [torch.from_numpy(tab[k]).cuda() for k in ("t", "pw", "tc", "pc")]
    fr = kr.evaluate_and_filter(space, *d)
    T, E = kr.evaluate_partition(space, *d)
    seg = np.arange(space.n_parts + 1, dtype=np.int64) * space.n_cand
    un = kr.pareto_filter(T, E, seg)
    sizes = []
    for p in range(space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], p)
        ix = oracle_lib.pareto(Tr, Er)
        sizes.append(len(ix))
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "fused part %d" % p)
        check_frontier(un, p, (ix, Tr[ix], Er[ix]), "unfused part %d" % p)
    assert min(sizes) > 2560


@pytest.mark.parametrize("n", [300, 2048, 20000, 9000, 30000])
def test_pareto_filter_union_paths(kr, oracle_lib, n):
    """One segment: small unions are sorted on chip; unions larger than the on-chip
    capacity (the sorted staircase, every point kept) go through the chunked merge."""
    rng = np.random.default_rng(n)
    if n in (9000, 30000):
        T = np.arange(n, dtype=np.float64) + 1.0
        E = 1e5 - np.arange(n, dtype=np.float64)
        if n == 30000:
            perm = rng.permutation(n)
            T, E = T[perm], E[perm]
    else:
        T = rng.lognormal(size=n)
        E = 1.0 / T + rng.random(n)
    seg = np.array([0, n], dtype=np.int64)
    fr = kr.pareto_filter(torch.from_numpy(T).cuda(), torch.from_numpy(E).cuda(), seg)
    ix = oracle_lib.pareto(T, E)
    check_frontier(fr, 0, (ix, T[ix], E[ix]), "n=%d" % n)


@pytest.mark.parametrize("shape", [(6, 7, 96), (16, 17, 96), (4, 5, 256), (8, 9, 130)])
def test_one_comm_many_sm_choices(kr, oracle_lib, shape):
    """One comm kernel with more SM choices than a wave has lanes (65 .. 256): the fused
    block-per-slab kernel with one thread per (SM choice, run of positions), with one
    tile per frequency (7 positions x 96, 5 x 256) or several (17 x 96, 9 x 130), against
    the oracle; the unfused evaluation too."""
    N, n_pos, S = shape
    K = tuple(1 + (7 * s) % 131 for s in range(S))  # SM counts 1 .. 131, repeats allowed
    space = I.Space(2, N, 1, n_pos, K, (1005.0, 1492.5, 1980.0))
    tab = I.make_tables(space, seed=N * 1000 + S, comm_bytes=(4e6, 64e6))
    d = [torch.from_numpy(tab[k]).cuda() for k in ("t", "pw", "tc", "pc")]
    fr = kr.evaluate_and_filter(space, *d)
    T, E = kr.evaluate_partition(space, *d)
    T, E = T.cpu().numpy(), E.cpu().numpy()
    for p in range(space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], p)
        assert_close(T[p], Tr, RT_TE, "T %s part %d" % (shape, p))
        assert_close(E[p], Er, RT_TE, "E %s part %d" % (shape, p))
        ix = oracle_lib.pareto(Tr, Er)
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "frontier %s part %d" % (shape, p))


@pytest.mark.parametrize("where,value", [("t", float("nan")), ("t", float("inf")),
                                         ("t", -1e-6), ("pw", float("nan")), ("pw", -5.0),
                                         ("tc", float("inf")), ("pc", -0.5)])
def test_nonfinite_tables_rejected(kr, where, value):
    """A NaN, infinite or negative table entry gives KR_ENONFINITE from the input check
    of the evaluation entry points (Sections 2.1, 4.5 define the cost model for finite,
    non-negative profiles)."""
    for cfg_space, n_comm in ((0, 1), (2, 2)):
        space = dataclasses.replace(I.SPACES[cfg_space]["space"], n_parts=2) if n_comm == 1 else \
            I.Space(2, 5, 2, 4, (4, 8), (1005.0, 1980.0))
        tab = I.make_tables(space, seed=3, comm_bytes=(4e6, 64e6))
        arr = tab[where]
        arr.reshape(-1)[arr.size // 2 + 1] = value
        d = [torch.from_numpy(tab[k]).cuda() for k in ("t", "pw", "tc", "pc")]
        with pytest.raises(kr.KrError) as e1:
            kr.evaluate_partition(space, *d)
        assert e1.value.status == kr.KR_ENONFINITE
        with pytest.raises(kr.KrError) as e2:
            kr.evaluate_and_filter(space, *d)
        assert e2.value.status == kr.KR_ENONFINITE
        kr.evaluate_and_filter(space, *d, validate=False)  # unchecked: runs, memory-safe
        torch.cuda.synchronize()


def test_negative_zero_table_entries_accepted(kr, oracle_lib):
    """-0.0 counts as 0: a table with -0.0 comm powers passes the check and matches the
    oracle on the same tables."""
    space = dataclasses.replace(I.SPACES[0]["space"], n_parts=2)
    tab = I.make_tables(space, seed=5, comm_bytes=(4e6, 64e6))
    tab["pc"][:, :, :, ::3] = -0.0
    d = [torch.from_numpy(tab[k]).cuda() for k in ("t", "pw", "tc", "pc")]
    fr = kr.evaluate_and_filter(space, *d)
    for p in range(space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], p)
        ix = oracle_lib.pareto(Tr, Er)
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "-0 tables part %d" % p)


@pytest.mark.parametrize("bad", ["nan_T", "inf_E", "neg_E", "nan_E", "neg_T"])
def test_nonfinite_points_rejected(kr, bad):
    """GetFrontier's input check: a NaN or infinite value or a negative one gives
    KR_ENONFINITE; the composition flags non-finite times and energies that are not
    finite values >= 0 in its status word and reports no staircase."""
    rng = np.random.default_rng(9)
    off = np.array([0, 40, 90, 130], dtype=np.int64)
    T = rng.uniform(1e-3, 2e-3, 130)
    E = rng.uniform(1.0, 2.0, 130)
    x = 57
    if bad == "nan_T":
        T[x] = np.nan
    elif bad == "inf_E":
        E[x] = np.inf
    elif bad == "neg_E":
        E[x] = -1e-9
    elif bad == "nan_E":
        E[x] = np.nan
    else:
        T[x] = -1e-3
    Td, Ed = torch.from_numpy(T).cuda(), torch.from_numpy(E).cuda()
    with pytest.raises(kr.KrError) as e:
        kr.pareto_filter(Td, Ed, off)
    assert e.value.status == kr.KR_ENONFINITE
    comp = kr.compose_frontiers(torch.from_numpy(off).cuda(), Td, Ed, 256)
    if bad == "neg_T":  # a negative time is finite: composition only shifts by tmin
        assert int(comp.status.item()) == kr.KR_OK
    else:
        assert int(comp.status.item()) == kr.KR_ENONFINITE
        assert int(comp.n_stair.item()) == 0


def test_negative_zero_energies(kr, oracle_lib):
    """-0.0 energies are read as +0.0: GetFrontier and the composition keep the oracle's
    points and back-pointers (the oracle compares -0.0 == +0.0)."""
    rng = np.random.default_rng(10)
    n = [30, 45, 12, 60]
    off = np.concatenate([[0], np.cumsum(n)]).astype(np.int64)
    T = rng.integers(1, 20, off[-1]) * 1e-4
    E = rng.integers(0, 6, off[-1]) * 0.5
    E[E == 0.0] = np.where(rng.random(int(np.sum(E == 0.0))) < 0.5, -0.0, 0.0)
    assert np.any(np.signbit(E) & (E == 0.0))
    fr = kr.pareto_filter(torch.from_numpy(T).cuda(), torch.from_numpy(E).cuda(), off)
    for g in range(len(n)):
        Tg, Eg = T[off[g]:off[g + 1]], E[off[g]:off[g + 1]]
        ix = oracle_lib.pareto(Tg, Eg)
        check_frontier(fr, g, (ix, Tg[ix], Eg[ix]), "-0 energies seg %d" % g)
    comp = kr.compose_frontiers(torch.from_numpy(off).cuda(), torch.from_numpy(T).cuda(),
                                torch.from_numpy(E).cuda(), 128)
    ref = oracle_lib.compose(off, T, E, 128)
    compare_composed(kr, comp, ref, off, T, E, "-0 energies")


@pytest.mark.parametrize("shape", [(32, 33, 5), (32, 32, 2), (32, 20, 2), (8, 9, 3), (20, 17, 2),
                                   (35, 36, 2), (40, 41, 2), (12, 8, 4), (1, 2, 3)])
@pytest.mark.parametrize("tc_scale", [1.0, 1e-3, 30.0])
def test_fused_32_sm_choices_shapes(kr, oracle_lib, shape, tc_scale):
    """One comm kernel with 32 SM choices (the SM-choice count of the evaluation stress
    workload): kernel counts 1 to 40, launch positions from 2 to N + 1 (32 kernels with
    33 positions take the kernel instance with the fixed sizes, with 32 or 20 the
    general one), short and long comm, every partition's fused frontier against the
    oracle."""
    N, n_pos, F = shape
    K = tuple(range(1, 33))
    freqs = tuple(1005.0 + 975.0 * q / max(F - 1, 1) for q in range(F))
    space = I.Space(3, N, 1, n_pos, K, freqs)
    tab = I.make_tables(space, seed=N * 7 + n_pos, comm_bytes=(4e6, 64e6))
    tab["tc"] = tab["tc"] * tc_scale
    d = [torch.from_numpy(tab[k]).cuda() for k in ("t", "pw", "tc", "pc")]
    fr = kr.evaluate_and_filter(space, *d)
    for p in range(space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], p)
        ix = oracle_lib.pareto(Tr, Er)
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "S=32 %s x%g part %d" % (shape, tc_scale, p))


def test_fused_many_box_members(kr, oracle_lib):
    """32 SM choices with comm time dominating and comm energy falling steeply with comm
    time: most candidates are frontier points (thousands per partition), so the fused
    filter's per-wave outputs overflow every on-chip list."""
    space = I.Space(2, 4, 1, 5, tuple(range(1, 33)), tuple(1005.0 + 15.0 * j for j in range(64)),
                    p_static=0.0)
    tab = I.make_tables(space, seed=23, comm_bytes=(4e6, 64e6))
    F, S = space.n_freq, space.n_sm
    tc = 10.0 + 1e-3 * np.arange(F * S, dtype=np.float64).reshape(F, S)
    tab["tc"] = np.broadcast_to(tc[None, :, None, :], tab["tc"].shape).copy()
    tab["pc"] = np.broadcast_to((1e6 / tc ** 2)[None, :, None, :], tab["pc"].shape).copy()
    d = [torch.from_numpy(tab[k]).cuda() for k in ("t", "pw", "tc", "pc")]
    fr = kr.evaluate_and_filter(space, *d)
    sizes = []
    for p in range(space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], p)
        ix = oracle_lib.pareto(Tr, Er)
        sizes.append(len(ix))
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "many box members part %d" % p)
    assert min(sizes) > 1000


@pytest.mark.parametrize("sort_cap", [None, "0", "5", "40"])
def test_two_comm_slab_reduction(kr, oracle_lib, monkeypatch, sort_cap):
    """Two comm kernels with at most 8 SM choices (the wave kernel): each wave's chunk
    frontiers of a slab are reduced to their frontier on chip when they fit the sort room.
    The test-only switch KR_TEST_PAIR_SORT_CAP lowers that room (0: never reduce), so
    slabs with more chunk outputs keep them all and the merge after the kernel sees
    them; every partition's frontier against the oracle either way."""
    if sort_cap is not None:
        monkeypatch.setenv("KR_TEST_PAIR_SORT_CAP", sort_cap)
    for k, space in enumerate([I.Space(4, 24, 2, 17, tuple(range(4, 36, 4)), (1005.0, 1500.0, 1980.0)),
                               I.Space(3, 7, 2, 8, (2, 5, 9), (1200.0, 1700.0))]):
        tab = I.make_tables(space, seed=40 + k, comm_bytes=(8e6, 512e6))
        d = [torch.from_numpy(tab[x]).cuda() for x in ("t", "pw", "tc", "pc")]
        fr = kr.evaluate_and_filter(space, *d)
        for p in range(space.n_parts):
            Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"],
                                                   tab["pc"], p)
            ix = oracle_lib.pareto(Tr, Er)
            check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "cap %s space %d part %d" % (sort_cap, k, p))


@pytest.mark.parametrize("shape", [(1, 1, 1), (1, 2, 8), (3, 1, 8), (5, 6, 3), (12, 13, 8),
                                   (20, 9, 7), (48, 33, 8), (9, 10, 2)])
@pytest.mark.parametrize("tc_scale", [1.0, 1e-3, 30.0])
def test_two_comm_wave_kernel_shapes(kr, oracle_lib, shape, tc_scale):
    """Two comm kernels with at most 8 SM choices (the wave kernel whose lanes are SM
    choice pairs): one or all launch positions, one kernel, one SM choice (lanes past
    S * S idle), short and long comm, every partition's fused frontier against the
    oracle."""
    N, n_pos, S = shape
    K = tuple(4 * (i + 1) for i in range(S))
    space = I.Space(3, N, 2, n_pos, K, (1005.0, 1490.0, 1980.0))
    tab = I.make_tables(space, seed=N * 11 + n_pos + S, comm_bytes=(8e6, 512e6))
    tab["tc"] = tab["tc"] * tc_scale
    d = [torch.from_numpy(tab[x]).cuda() for x in ("t", "pw", "tc", "pc")]
    fr = kr.evaluate_and_filter(space, *d)
    for p in range(space.n_parts):
        Tr, Er = oracle_lib.evaluate_partition(space, tab["t"], tab["pw"], tab["tc"], tab["pc"], p)
        ix = oracle_lib.pareto(Tr, Er)
        check_frontier(fr, p, (ix, Tr[ix], Er[ix]), "M=2 %s x%g part %d" % (shape, tc_scale, p))

