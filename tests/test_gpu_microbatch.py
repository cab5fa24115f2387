"""GPU parity of the microbatch frontier (Algorithm 2 with one frequency per microbatch
and one configuration per partition type) against the oracle: points, frequencies and
per-type choices bit-exact, on random point sets, on per-(type, frequency) frontiers of
evaluated llama-layer tables, and on the degenerate cases (a used type without points at a
frequency, types not in the sequence, one type repeated)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2601_17654_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kr():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2601_17654_amd import binding

    return binding


def _random_case(rng, K, F, nmax, empty=None):
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


def _compare_exact(kr, seg_off, T, E, K, F, seq, cT, cE, what):
    print("microbatch enumeration case", what, flush=True)
    got = kr.microbatch_enumerate(seg_off, torch.from_numpy(T).cuda(),
                                  torch.from_numpy(E).cuda(), K, F, seq,
                                  None if cT is None else torch.from_numpy(cT).cuda(),
                                  None if cE is None else torch.from_numpy(cE).cuda())
    rT, rE, rf, rch = oracle.microbatch_exact(seg_off, T, E, K, F, seq, cT, cE)
    assert got.T.numel() == len(rT), what
    np.testing.assert_array_equal(got.f.cpu().numpy(), rf, err_msg=what)
    np.testing.assert_array_equal(got.choice.cpu().numpy(), rch, err_msg=what)
    np.testing.assert_array_equal(got.T.cpu().numpy(), rT, err_msg=what)
    np.testing.assert_array_equal(got.E.cpu().numpy(), rE, err_msg=what)
    return len(rT)


def _compare(kr, seg_off, T, E, K, F, seq, cT, cE, B, what):
    print("microbatch case", what, flush=True)
    got = kr.microbatch_frontier(seg_off, torch.from_numpy(T).cuda(), torch.from_numpy(E).cuda(),
                                 K, F, seq, None if cT is None else torch.from_numpy(cT).cuda(),
                                 None if cE is None else torch.from_numpy(cE).cuda(), n_bins=B)
    rT, rE, rf, rch = oracle.microbatch(seg_off, T, E, K, F, seq, cT, cE, n_bins=B)
    gT, gE = got.T.cpu().numpy(), got.E.cpu().numpy()
    gf, gch = got.f.cpu().numpy(), got.choice.cpu().numpy()
    assert len(gT) == len(rT), what
    np.testing.assert_array_equal(gf, rf, err_msg=what)
    np.testing.assert_array_equal(gch, rch, err_msg=what)
    np.testing.assert_array_equal(gT, rT, err_msg=what)
    np.testing.assert_array_equal(gE, rE, err_msg=what)
    return len(gT)


@pytest.mark.parametrize("seed", range(8))
def test_microbatch_random(kr, seed):
    rng = np.random.default_rng(300 + seed)
    K, F = int(rng.integers(1, 5)), int(rng.integers(1, 6))
    seg_off, T, E = _random_case(rng, K, F, 12)
    seq = [int(x) for x in rng.integers(0, K, int(rng.integers(1, 9)))]
    nc = int(rng.integers(0, 3))
    cT = rng.uniform(1e-4, 1e-3, (nc, F)) if nc else None
    cE = rng.uniform(0.01, 0.1, (nc, F)) if nc else None
    B = int(rng.choice([64, 512, 4096]))
    _compare(kr, seg_off, T, E, K, F, seq, cT, cE, B, "random %d" % seed)
    _compare_exact(kr, seg_off, T, E, K, F, seq, cT, cE, "random %d" % seed)


@pytest.mark.parametrize("B", [4097, 9000, 20000])
def test_microbatch_wide_grids(kr, B):
    """More bins than one on-chip binning window (4,096 offsets) and thousands of points
    per type and frequency: a type's offsets are binned in several windows, and its
    occupied offsets run to thousands."""
    rng = np.random.default_rng(B)
    K, F = 2, 3
    seg_off, T, E = _random_case(rng, K, F, 3000)
    _compare(kr, seg_off, T, E, K, F, [0, 1, 0], None, None, B, "wide grid %d" % B)
    _compare(kr, seg_off, T, E, K, F, [1], None, None, B, "wide grid %d, one type" % B)


def test_microbatch_degenerate(kr):
    rng = np.random.default_rng(17)
    K, F = 3, 4
    seg_off, T, E = _random_case(rng, K, F, 6, empty=(1, 2))
    # a used type without points at frequency 2, an unused type
    _compare(kr, seg_off, T, E, K, F, [0, 1, 0], None, None, 256, "empty segment")
    _compare_exact(kr, seg_off, T, E, K, F, [0, 1, 0], None, None, "empty segment")
    # one type, repeated, with components
    cT, cE = I.microbatch_components(5, 2, [1005.0, 1200.0, 1500.0, 1980.0])
    _compare(kr, seg_off, T, E, K, F, [2] * 5, cT, cE, 1024, "one type repeated")
    _compare_exact(kr, seg_off, T, E, K, F, [2] * 5, cT, cE, "one type repeated")


def test_microbatch_llama_layers(kr):
    """Types = the first four partitions of the llama-layer tables; per-(type, frequency)
    frontiers by the library's filter and by the oracle's; a sequence of 8 layers of
    (type 0, type 1) plus one of each other type; two components."""
    w = I.config_workload(1, parts=range(0, 4))
    sp = w.space
    K, F = sp.n_parts, sp.n_freq
    Cf = sp.cand_per_freq
    d = [torch.from_numpy(getattr(w, k)).cuda() for k in ("t", "pw", "tc", "pc")]
    Tg, Eg = kr.evaluate_partition(sp, *d)
    seg = np.arange(K * F + 1, dtype=np.int64) * Cf
    fr = kr.pareto_filter(Tg.reshape(-1), Eg.reshape(-1), seg)
    # the oracle's per-(type, frequency) frontiers
    rT, rE, rsegs = [], [], [0]
    for t in range(K):
        Tt, Et = oracle.evaluate_partition(sp, w.t, w.pw, w.tc, w.pc, t)
        for f in range(F):
            idx = oracle.pareto(Tt[f * Cf:(f + 1) * Cf], Et[f * Cf:(f + 1) * Cf])
            rT.extend(Tt[f * Cf + idx])
            rE.extend(Et[f * Cf + idx])
            rsegs.append(rsegs[-1] + len(idx))
    rseg = np.array(rsegs, dtype=np.int64)
    np.testing.assert_array_equal(fr.off.cpu().numpy(), rseg)
    np.testing.assert_array_equal(fr.T.cpu().numpy(), np.array(rT))
    np.testing.assert_array_equal(fr.E.cpu().numpy(), np.array(rE))
    seq = [0, 1] * 8 + [2, 3]
    cT, cE = I.microbatch_components(1, 2, sp.freqs_mhz)
    n = _compare(kr, rseg, np.array(rT), np.array(rE), K, F, seq, cT, cE, 2048, "llama layers")
    assert n > 10
    assert _compare_exact(kr, rseg, np.array(rT), np.array(rE), K, F, seq, cT, cE,
                          "llama layers") > 10


def test_microbatch_kept_buffers(kr):
    """Calls given kept buffers and check=False return the same points as the default
    calls, also when the buffers are used again with other inputs of the same shape."""
    rng = np.random.default_rng(41)
    K, F, B = 3, 4, 512
    seq = [0, 1, 2, 1, 0]
    seg_off, T, E = _random_case(rng, K, F, 6)
    cT = rng.uniform(1e-4, 5e-4, (2, F))
    cE = rng.uniform(0.05, 0.2, (2, F))
    cT_d, cE_d = torch.from_numpy(cT).cuda(), torch.from_numpy(cE).cuda()
    sizes = np.diff(seg_off).reshape(K, F)
    n_cfg = int(np.sum(np.prod(sizes, axis=0)))
    gbuf = kr.microbatch_buffers(seg_off, K, F * B)
    xbuf = kr.microbatch_buffers(seg_off, K, n_cfg)
    for rep in range(2):
        T2 = T * (1.0 + 0.25 * rep)
        T_d, E_d = torch.from_numpy(T2).cuda(), torch.from_numpy(E).cuda()
        ref = kr.microbatch_frontier(seg_off, T_d, E_d, K, F, seq, cT_d, cE_d, n_bins=B)
        got = kr.microbatch_frontier(seg_off, T_d, E_d, K, F, seq, cT_d, cE_d, n_bins=B,
                                     check=False, out=gbuf)
        n = int(got.n.item())
        assert n == ref.T.numel()
        np.testing.assert_array_equal(got.T[:n].cpu().numpy(), ref.T.cpu().numpy())
        np.testing.assert_array_equal(got.E[:n].cpu().numpy(), ref.E.cpu().numpy())
        np.testing.assert_array_equal(got.choice[:n].cpu().numpy(), ref.choice.cpu().numpy())
        refx = kr.microbatch_enumerate(seg_off, T_d, E_d, K, F, seq, cT_d, cE_d)
        gotx = kr.microbatch_enumerate(seg_off, T_d, E_d, K, F, seq, cT_d, cE_d, check=False,
                                       out=xbuf)
        assert int(gotx.status.item()) == kr.KR_OK
        n = int(gotx.n.item())
        assert n == refx.T.numel()
        np.testing.assert_array_equal(gotx.T[:n].cpu().numpy(), refx.T.cpu().numpy())
        np.testing.assert_array_equal(gotx.f[:n].cpu().numpy(), refx.f.cpu().numpy())
        np.testing.assert_array_equal(gotx.choice[:n].cpu().numpy(), refx.choice.cpu().numpy())
        # and the checked call on the kept buffers trims as the default one does
        chk = kr.microbatch_enumerate(seg_off, T_d, E_d, K, F, seq, cT_d, cE_d, out=xbuf)
        np.testing.assert_array_equal(chk.E.cpu().numpy(), refx.E.cpu().numpy())
    # buffers made for other segments are refused
    seg2, T3, E3 = _random_case(np.random.default_rng(42), K, F, 6)
    assert not np.array_equal(seg2, seg_off)
    with pytest.raises(ValueError):
        kr.microbatch_enumerate(seg2, torch.from_numpy(T3).cuda(), torch.from_numpy(E3).cuda(),
                                K, F, seq, cT_d, cE_d, out=xbuf)
