"""GPU parity of the launch-timing dynamic program (Appendix B) against the oracle:
frontier times and energies, sizes and schedules bit-exact, on random instances of many
shapes (lone sequences, no communication, kmax = 0, several communications, repeated
structure across a batch), on two-nanobatch transformer blocks built from the two-comm
tables, and with a frontier larger than the output capacity."""

import numpy as np
import pytest
import torch

import oracle
from paper_2601_17654_amd import inputs as I

pytestmark = pytest.mark.gpu

# the kernel's on-chip limits: points of one cell, points of all cells, candidates of a cell
LIMITS = (64, 2048, 1024)


@pytest.fixture(scope="module")
def kr():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2601_17654_amd import binding

    return binding


def _random_batch(rng, kind1, kind2, n):
    kind = list(kind1) + list(kind2)
    ops = np.zeros((n, len(kind), 4))
    for x in range(n):
        for o, k in enumerate(kind):
            if k == 0:
                t0 = rng.uniform(1e-4, 2e-3)
                p0 = rng.uniform(300, 700)
                ops[x, o] = [t0, p0, t0 * rng.uniform(1.05, 1.6), p0 * rng.uniform(0.6, 0.95)]
            else:
                ops[x, o] = [rng.uniform(2e-4, 4e-3), rng.uniform(80, 200), 0.0, 0.0]
    return ops


def _compare(kr, kind1, kind2, ops, ps, kmax, what, out_cap=64):
    print("launch-timing case", what, flush=True)
    got = kr.launch_timing_frontier(kind1, kind2, torch.from_numpy(ops).cuda(), ps, kmax,
                                    out_cap=out_cap, check=False)
    gT, gE = got.T.cpu().numpy(), got.E.cpu().numpy()
    gS, gn = got.sched.cpu().numpy(), got.n.cpu().numpy()
    fits = 0
    for x in range(ops.shape[0]):
        rT, rE, rS, (mcell, total, mcand) = oracle.launch_dp(kind1, kind2, ops[x], ps, kmax)
        if mcell > LIMITS[0] or total > LIMITS[1] or mcand > LIMITS[2]:
            assert gn[x] == -1, (what, x)  # beyond the on-chip limits: reported, not solved
            continue
        fits += 1
        assert gn[x] == len(rT), (what, x)
        m = min(len(rT), out_cap)
        np.testing.assert_array_equal(gT[x, :m], rT[:m], err_msg="%s %d T" % (what, x))
        np.testing.assert_array_equal(gE[x, :m], rE[:m], err_msg="%s %d E" % (what, x))
        np.testing.assert_array_equal(gS[x, :m], rS[:m], err_msg="%s %d sched" % (what, x))
    st = int(got.status.item())
    assert st == (kr.KR_OK if fits == ops.shape[0] else kr.KR_ECAPACITY)
    return fits


@pytest.mark.parametrize("kind1,kind2,kmax", [
    ([0], [1], 1),
    ([0, 0, 1], [0, 1, 0], 3),
    ([0, 0, 0, 0, 1, 0, 0, 0, 0, 0, 1], [0, 0, 0, 0, 1, 0, 0, 0, 0, 0, 1], 9),
    ([1, 0, 0, 1, 0, 1], [0, 0, 0, 1, 0, 0, 0], 4),
    ([0, 0, 0], [0, 0], 2),                   # no communication
    ([0, 1, 0, 0], [1, 0, 0, 0], 0),          # no overlap allowed
    ([0, 0, 0, 0, 0, 0], [], 3),              # one sequence only
    ([], [1, 0, 0], 2),
    ([0] * 24, [1] * 2, 16),                  # the longest sequence, the largest kmax
    ([0, 1] * 6, [1, 0] * 6, 16),             # many instances past the first pass's budget
    ([0, 1] * 12, [1, 0] * 12, 16),           # some past the full budget
])
def test_random_instances(kr, kind1, kind2, kmax):
    rng = np.random.default_rng(len(kind1) * 31 + len(kind2) + kmax)
    ops = _random_batch(rng, kind1, kind2, 24)
    _compare(kr, kind1, kind2, ops, I.P_STATIC_W, kmax, "random %s/%s k%d" % (kind1, kind2, kmax))


def test_two_nanobatch_blocks(kr):
    w = I.config_workload(2, parts=range(0, 2))
    kind1, kind2, ops, idx = I.dp_instances(w, [0, 1])
    sel = np.random.default_rng(3).choice(len(ops), 96, replace=False)
    assert _compare(kr, kind1, kind2, ops[sel], w.space.p_static, I.DP_KMAX,
                    "two-nanobatch") == len(sel)


def test_output_capacity(kr):
    rng = np.random.default_rng(8)
    kind1, kind2 = [0, 0, 1, 0, 0, 1], [0, 0, 1, 0, 0, 1]
    ops = _random_batch(rng, kind1, kind2, 16)
    _compare(kr, kind1, kind2, ops, 0.0, 4, "capacity 1", out_cap=1)


def test_no_instances(kr):
    ops = torch.zeros((0, 4, 4), dtype=torch.float64, device="cuda")
    got = kr.launch_timing_frontier([0, 1], [0, 0], ops, I.P_STATIC_W, 2)
    assert got.T.shape[0] == 0 and int(got.status.item()) == kr.KR_OK
