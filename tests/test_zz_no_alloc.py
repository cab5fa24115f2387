"""The allocation-free GetFrontier entry point (kr_pareto_filter_noalloc, library-held
workspace) against kr_pareto_filter with a caller workspace: identical CSR output on
two calls in a row, the second with a smaller input, and the size limits refused on
the host before any launch."""

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kr():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2601_17654_amd import binding

    return binding


def _points(seed, lens):
    rng = np.random.default_rng(seed)
    T = np.concatenate([rng.lognormal(size=n) for n in lens])
    E = np.concatenate([1.0 / T[sum(lens[:i]):sum(lens[:i + 1])] + rng.random(n)
                        for i, n in enumerate(lens)])
    # ties and duplicates in every segment
    T[::7] = np.round(T[::7], 1)
    E[::5] = np.round(E[::5], 1)
    seg = np.zeros(len(lens) + 1, dtype=np.int64)
    seg[1:] = np.cumsum(lens)
    return torch.from_numpy(T).cuda(), torch.from_numpy(E).cuda(), seg


def test_noalloc_matches_pareto_filter(kr):
    big = [60000, 0, 1, 250000, 31, 2048, 2049, 180000, 300000, 77, 5000]  # 799,206 points
    cases = [("large", 11, big), ("smaller", 12, [700, 3, 0, 5000, 2])]
    assert sum(big) <= kr.NOALLOC_MAX_POINTS
    for what, seed, lens in cases:
        print("no-alloc case", what, sum(lens), "points", flush=True)
        T, E, seg = _points(seed, lens)
        a = kr.pareto_filter(T, E, seg, noalloc=True)
        b = kr.pareto_filter(T, E, seg)
        for x, y in ((a.off, b.off), (a.idx, b.idx), (a.T, b.T), (a.E, b.E)):
            assert torch.equal(x, y), what


def test_noalloc_limits(kr):
    one = torch.zeros(1, dtype=torch.float64, device="cuda")
    with pytest.raises(kr.KrError) as e:
        kr._check("kr_pareto_filter_noalloc",
                  kr._lib.kr_pareto_filter_noalloc(kr.NOALLOC_MAX_POINTS + 1, kr._ptr(one),
                                                   kr._ptr(one), kr._ptr(one), 1, 1, kr._ptr(one),
                                                   kr._ptr(one), kr._ptr(one), kr._ptr(one), None,
                                                   kr._stream()))
    assert e.value.status == kr.KR_ECAPACITY
    with pytest.raises(kr.KrError) as e:
        kr._check("kr_pareto_filter_noalloc",
                  kr._lib.kr_pareto_filter_noalloc(10, kr._ptr(one), kr._ptr(one), kr._ptr(one),
                                                   kr.NOALLOC_MAX_SEGS + 1, 1, kr._ptr(one),
                                                   kr._ptr(one), kr._ptr(one), kr._ptr(one), None,
                                                   kr._stream()))
    assert e.value.status == kr.KR_ECAPACITY
