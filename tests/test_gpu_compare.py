"""GPU parity of the frontier comparison metrics (Section 6.1, "Metrics") against the
oracle: all ten outputs bit-exact (they are minima under predicates and one division),
including NaN for an unreachable deadline or budget, on hand-made, random, tie-heavy and
multi-block point sets."""

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kr():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2601_17654_amd import binding

    return binding


def _both(kr, TA, EA, TB, EB, what):
    print("compare case", what, flush=True)
    got = kr.compare_frontiers(*(torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))
                                 .cuda() for x in (TA, EA, TB, EB))).cpu().numpy()
    ref = oracle.compare(TA, EA, TB, EB)
    np.testing.assert_array_equal(got, ref, err_msg=what)
    return got


def test_hand_case(kr):
    r = _both(kr, [1, 2, 4], [10, 5, 2], [0.8, 1.5, 3], [9, 4, 1], "hand")
    np.testing.assert_allclose(r[:4], [20, 10, 10, 25], rtol=1e-13)


def test_unreachable(kr):
    r = _both(kr, [1.0, 2.0], [2.0, 1.0], [1.5, 3.0], [1.8, 1.2], "unreachable")
    assert np.isnan(r[2]) and np.isnan(r[3])


@pytest.mark.parametrize("nA,nB", [(1, 1), (1, 700), (300, 5), (4097, 3000),
                                   (1 << 20, 3 << 20), (5_000_000, 17)])
def test_random_sets(kr, nA, nB):
    rng = np.random.default_rng(nA + 7 * nB)
    TA = np.round(rng.uniform(1, 3, nA), 3)  # ties in time and energy
    EA = np.round(rng.uniform(1, 3, nA), 3)
    TB = np.round(rng.uniform(0.9, 3, nB), 3)
    EB = np.round(rng.uniform(0.9, 3, nB), 3)
    _both(kr, TA, EA, TB, EB, "random %d/%d" % (nA, nB))


def test_self_and_scaled(kr):
    i = np.arange(1, 2001, dtype=float)
    r = _both(kr, i, 1 / i, i, 1 / i, "self")
    assert np.all(r[:4] == 0.0)
    _both(kr, i, 1 / i, 0.5 * i, 0.5 / i, "scaled")
