"""GPU parity of the Bayesian optimisation's scores and batch selection (Section 4.3,
Algorithm 1; Appendix C) against the oracle.

  * HV and the reference point are bit-exact (same staircase strips, same order).
  * HVI: the kernel sums the area a candidate adds, the oracle takes the difference of
    two hypervolumes, so they differ by rounding only.  Each hypervolume is a sum of at
    most m = n_obs + 1 strips, each a product of two differences: a strip carries at most
    3 roundings and the running sum m - 1, so each side's HV is within (m + 2) u of
    exact; the oracle's difference adds one more rounding, the kernel's strip sum is
    within (m + 2) u of its own (smaller) total.  Bound used:
        |gpu - oracle| <= (3 m + 8) u (HV(P) + HVI),   u = 2^-53.
    A zero from the kernel (dominated or outside the box) is a zero of the oracle.
  * Selection is exact on the same scores; the uncertainty score agrees to 2 ulps
    (square roots).
  * End to end (evaluated llama-layer and stress tables -> scores -> selection): scores
    within the bound above, and every pass of the batch is the top-k of the scores the
    kernel was given.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2601_17654_amd import inputs as I

pytestmark = pytest.mark.gpu

U = 2.0 ** -53


@pytest.fixture(scope="module")
def kr():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2601_17654_amd import binding

    return binding


def _cuda(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _check_hvi(gh, ghv, gref, rh, rhv, rref, cand_off, obs_off, what):
    np.testing.assert_array_equal(ghv, rhv, err_msg=what + " hv")
    np.testing.assert_array_equal(gref, rref, err_msg=what + " ref")
    for g in range(len(cand_off) - 1):
        c0, c1 = cand_off[g], cand_off[g + 1]
        if c1 == c0:
            continue
        m = obs_off[g + 1] - obs_off[g] + 1
        for v in range(3):
            a, b = gh[v, c0:c1], rh[v, c0:c1]
            tol = (3 * m + 8) * U * (rhv[g, v] + np.maximum(np.abs(a), np.abs(b)))
            bad = np.abs(a - b) > tol
            assert not bad.any(), "%s part %d v %d: %d off, first %s" % (
                what, g, v, bad.sum(), (a[bad][:3], b[bad][:3]))
            assert np.all(b[a == 0.0] == 0.0), "%s part %d v %d: kernel zero" % (what, g, v)


def _random_hvi_case(seed, n_cand, n_obs):
    rng = np.random.default_rng(seed)
    cand_off = np.concatenate([[0], np.cumsum(n_cand)]).astype(np.int64)
    obs_off = np.concatenate([[0], np.cumsum(n_obs)]).astype(np.int64)
    To = rng.uniform(1e-3, 4e-3, obs_off[-1])
    Eo = rng.uniform(0.3, 0.9, obs_off[-1])
    Th = rng.uniform(0.5e-3, 5e-3, cand_off[-1])
    Eh = rng.uniform(0.2, 1.0, cand_off[-1])
    # exact ties with measured points and on the box's edges
    if cand_off[-1] >= 8 and obs_off[-1] >= 2:
        Th[:2], Eh[:2] = To[:2], Eo[:2]
        Th[2], Eh[2] = To[0], Eo[0] * 0.5
        Th[3], Eh[3] = To[0] * 0.5, Eo[0]
    return cand_off, Th, Eh, obs_off, To, Eo


@pytest.mark.parametrize("n_cand,n_obs", [
    ([700], [12]),
    ([1500, 3, 0, 1025, 64], [40, 1, 5, 96, 2]),       # ragged tiles, empty partition
    ([5000, 4000], [512, 300]),                        # the largest measured sample
    ([17] * 200, [3] * 200),                           # many partitions per tile
])
def test_hvi_parity(kr, n_cand, n_obs):
    print("hvi case", n_cand[:5], n_obs[:5], flush=True)
    cand_off, Th, Eh, obs_off, To, Eo = _random_hvi_case(len(n_cand) * 7 + n_obs[0], n_cand,
                                                         n_obs)
    got = kr.hvi_scores(cand_off, _cuda(Th), _cuda(Eh), obs_off, _cuda(To), _cuda(Eo),
                        I.P_STATIC_W)
    rh, rhv, rref = oracle.hvi(cand_off, Th, Eh, obs_off, To, Eo, I.P_STATIC_W)
    _check_hvi(got.hvi.cpu().numpy(), got.hv.cpu().numpy(), got.ref.cpu().numpy(), rh, rhv, rref,
               cand_off, obs_off, "random")


def test_hvi_bad_partition_status(kr):
    cand_off = np.array([0, 10, 20], dtype=np.int64)
    obs_off = np.array([0, 4, 4], dtype=np.int64)  # second partition: no measured point
    Th = np.linspace(1e-3, 2e-3, 20)
    got = kr.hvi_scores(cand_off, _cuda(Th), _cuda(Th * 300), obs_off, _cuda(Th[:4]),
                        _cuda(Th[:4] * 310), I.P_STATIC_W, check=False)
    torch.cuda.synchronize()
    assert int(got.status.item()) == kr.KR_EINVAL
    h = got.hvi.cpu().numpy()
    assert np.isnan(h[:, 10:]).all() and not np.isnan(h[:, :10]).any()
    assert np.isnan(got.hv.cpu().numpy()[1]).all()
    with pytest.raises(kr.KrError):
        kr.hvi_scores(cand_off, _cuda(Th), _cuda(Th * 300), obs_off, _cuda(Th[:4]),
                      _cuda(Th[:4] * 310), I.P_STATIC_W)


def test_uncertainty_parity(kr):
    rng = np.random.default_rng(5)
    for M, n in ((5, 10007), (5, 10008), (1, 300), (16, 64)):
        Tm = rng.uniform(1e-3, 2e-3, (M, n))
        Em = rng.uniform(0.2, 0.8, (M, n))
        got = kr.uncertainty(_cuda(Tm), _cuda(Em)).cpu().numpy()
        ref = oracle.uncertainty(Tm, Em)
        np.testing.assert_allclose(got, ref, rtol=4 * U, atol=0)
        if M == 1:
            assert np.all(got == 0.0)


def _selection_case(seed, n_cand, n_obs, ties=True):
    rng = np.random.default_rng(seed)
    cand_off = np.concatenate([[0], np.cumsum(n_cand)]).astype(np.int64)
    n = cand_off[-1]
    s = rng.uniform(0, 1, (3, n))
    if ties:
        s = np.round(s * 50) / 50  # many exact ties
        s[:, rng.random(n) < 0.4] = 0.0
        s[0, rng.random(n) < 0.1] = -0.0
    unc = rng.uniform(0, 1, n)
    obs_off = np.concatenate([[0], np.cumsum(n_obs)]).astype(np.int64)
    obs = np.concatenate([rng.integers(-2, max(c, 1) + 2, o) for c, o in zip(n_cand, n_obs)]
                         ).astype(np.int64) if obs_off[-1] else np.zeros(0, np.int64)
    return cand_off, s, unc, obs_off, obs


@pytest.mark.parametrize("n_cand,n_obs,ks", [
    ([5000], [96], (13, 6, 6, 32)),
    ([9000, 1, 0, 4097, 63, 4096], [96, 1, 3, 50, 70, 0], (13, 6, 6, 32)),
    ([3000, 3000], [10, 10], (64, 0, 0, 64)),
    ([3000, 200], [10, 10], (20, 20, 20, 64)),
    ([3000, 200], [10, 10], (0, 0, 0, 17)),
    ([3000, 200], [10, 10], (0, 0, 0, 0)),
    ([40] * 300, [5] * 300, (2, 2, 2, 8)),
])
@pytest.mark.parametrize("with_unc", [True, False])
def test_select_parity(kr, n_cand, n_obs, ks, with_unc):
    print("select case", n_cand[:6], ks, with_unc, flush=True)
    cand_off, s, unc, obs_off, obs = _selection_case(sum(n_cand) + ks[0], n_cand, n_obs)
    u = unc if with_unc else None
    got = kr.select_batch(cand_off, _cuda(s), None if u is None else _cuda(u), obs_off,
                          obs, *ks).lists()
    ref = oracle.select(cand_off, s, u, obs_off, obs, *ks)
    for g in range(len(n_cand)):
        np.testing.assert_array_equal(got[g], ref[g], err_msg="part %d" % g)


def test_select_nan_status(kr):
    cand_off, s, unc, obs_off, obs = _selection_case(3, [5000, 100], [10, 10])
    unc[4000] = np.nan
    b = kr.select_batch(cand_off, _cuda(s), _cuda(unc), obs_off, obs, 13, 6, 6, 32, check=False)
    torch.cuda.synchronize()
    assert int(b.status.item()) == kr.KR_EINVAL
    assert np.all(b.count.cpu().numpy() == 0)
    # the same call without the exploration pass is fine, and a later good call resets
    b = kr.select_batch(cand_off, _cuda(s), None, obs_off, obs, 13, 6, 6, 32)
    assert int(b.status.item()) == kr.KR_OK


def _top(s, excluded, m):
    """The m best of s outside `excluded` (score descending, index ascending)."""
    x = np.setdiff1d(np.arange(s.shape[0]), np.asarray(list(excluded), dtype=np.int64))
    return x[np.lexsort((x, -s[x]))][:m]


def _check_batch(C, s, unc, D, ks, k, what):
    """C holds each exploitation pass's top-k_p in pass order (repeats dropped), then the
    best uncertainties outside D and those passes, up to k members."""
    D = set(D.tolist())
    front = []
    for p in range(3):
        for x in _top(s[p], D, ks[p]).tolist():
            if x not in front:
                front.append(x)
    rest = _top(unc, D | set(front), k - len(front)).tolist()
    assert C.tolist() == front + rest, what


def _mbo_chain(kr, w, parts_check, seed=11):
    """Evaluated tables -> measured sample and ensembles -> scores -> selection, on the
    GPU for all partitions and in the oracle for the partitions checked."""
    space = w.space
    d = [torch.from_numpy(getattr(w, k)).cuda() for k in ("t", "pw", "tc", "pc")]
    T, E = kr.evaluate_partition(space, *d)
    T, E = T.reshape(-1), E.reshape(-1)
    C, P = space.n_cand, space.n_parts
    cand_off = np.arange(P + 1, dtype=np.int64) * C
    obs_off, idx, z = I.mbo_observations(seed, [C] * P, I.MBO_N_INIT)
    gidx = np.repeat(cand_off[:-1], I.MBO_N_INIT) + idx
    gi, zd = _cuda(gidx), _cuda(z)
    To = I.perturb(T[gi], zd[:, 0], 0.02)
    Eo = I.perturb(E[gi], zd[:, 1], 0.02)
    tab = _cuda(I.noise_table(seed + 1))
    x = torch.arange(C * P, device="cuda", dtype=torch.int64)
    Tm = torch.stack([I.perturb(T, tab[I.noise_index(2 * m, x)], 0.05)
                      for m in range(I.MBO_MEMBERS)])
    Em = torch.stack([I.perturb(E, tab[I.noise_index(2 * m + 1, x)], 0.05)
                      for m in range(I.MBO_MEMBERS)])
    sc = kr.hvi_scores(cand_off, T, E, obs_off, To, Eo, space.p_static)
    unc = kr.uncertainty(Tm, Em)
    k1, k2, k3 = I.MBO_PASSES
    batch = kr.select_batch(cand_off, sc.hvi, unc, obs_off, idx, k1, k2, k3, I.MBO_BATCH)
    gh, ghv, gref = sc.hvi.cpu().numpy(), sc.hv.cpu().numpy(), sc.ref.cpu().numpy()
    gu = unc.cpu().numpy()
    sel = batch.lists()
    tabh = I.noise_table(seed + 1)
    for p in parts_check:
        print("mbo chain partition", p, flush=True)
        Tr, Er = oracle.evaluate_partition(space, w.t, w.pw, w.tc, w.pc, p)
        o = slice(p * I.MBO_N_INIT, (p + 1) * I.MBO_N_INIT)
        Tor = I.perturb(Tr[idx[o]], z[o, 0], 0.02)
        Eor = I.perturb(Er[idx[o]], z[o, 1], 0.02)
        rh, rhv, rref = oracle.hvi([0, C], Tr, Er, [0, I.MBO_N_INIT], Tor, Eor, space.p_static)
        c0 = p * C
        _check_hvi(gh[:, c0:c0 + C], ghv[p:p + 1], gref[p:p + 1], rh, rhv, rref, [0, C],
                   [0, I.MBO_N_INIT], "chain part %d" % p)
        xs = np.arange(c0, c0 + C, dtype=np.int64)
        Tmr = np.stack([I.perturb(Tr, tabh[I.noise_index(2 * m, xs)], 0.05)
                        for m in range(I.MBO_MEMBERS)])
        Emr = np.stack([I.perturb(Er, tabh[I.noise_index(2 * m + 1, xs)], 0.05)
                        for m in range(I.MBO_MEMBERS)])
        np.testing.assert_allclose(gu[c0:c0 + C], oracle.uncertainty(Tmr, Emr), rtol=4 * U,
                                   atol=0)
        # the batch is the multi-pass selection of the scores the kernel was given
        _check_batch(sel[p], gh[:, c0:c0 + C], gu[c0:c0 + C], idx[o], (k1, k2, k3),
                     I.MBO_BATCH, "chain part %d" % p)
    for p in range(P):
        C_ = sel[p]
        assert len(C_) == I.MBO_BATCH and len(set(C_.tolist())) == I.MBO_BATCH
        assert not set(C_.tolist()) & set(idx[p * I.MBO_N_INIT:(p + 1) * I.MBO_N_INIT].tolist())
    return sc, batch


def test_mbo_chain_llama(kr):
    w = I.config_workload(1, parts=range(0, 4))
    _mbo_chain(kr, w, range(4))


def test_mbo_chain_eval_stress_sampled(kr):
    """The benchmark's launch: all 1,024 partitions of the stress tables at once, the
    oracle on sampled partitions."""
    w = I.config_workload(3)
    _mbo_chain(kr, w, [0, 517, 1023])


def test_empty_candidate_sets(kr):
    """No candidates at all: HV and r still come from the measured points; the batch is
    empty."""
    cand_off = np.zeros(3, dtype=np.int64)
    obs_off = np.array([0, 2, 5], dtype=np.int64)
    To = np.array([1e-3, 2e-3, 1e-3, 3e-3, 2e-3])
    Eo = np.array([0.5, 0.4, 0.9, 0.3, 0.6])
    empty = torch.zeros(0, dtype=torch.float64, device="cuda")
    got = kr.hvi_scores(cand_off, empty, empty, obs_off, _cuda(To), _cuda(Eo), I.P_STATIC_W)
    _, rhv, rref = oracle.hvi(cand_off, np.zeros(0), np.zeros(0), obs_off, To, Eo, I.P_STATIC_W)
    np.testing.assert_array_equal(got.hv.cpu().numpy(), rhv)
    np.testing.assert_array_equal(got.ref.cpu().numpy(), rref)
    b = kr.select_batch(cand_off, torch.zeros((3, 0), dtype=torch.float64, device="cuda"),
                        empty, obs_off, np.array([0, 1, 0, 1, 2]), 13, 6, 6, 32)
    assert all(len(x) == 0 for x in b.lists())
