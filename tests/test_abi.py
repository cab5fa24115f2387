"""The C ABI library loads and exports every symbol that include/kareus.h declares;
host-side argument validation answers without touching a GPU."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kareus.h")
LIB = os.path.join(ROOT, "paper_2601_17654_amd", "libkareus_mi355x.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kr_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2601_17654_amd import build

        build.build()
    return ctypes.CDLL(LIB)


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    lib.kr_status_string.restype = ctypes.c_char_p
    assert lib.kr_status_string(0) == b"ok"
    assert b"capacity" in lib.kr_status_string(-3)
    assert b"non-finite" in lib.kr_status_string(-2)
    assert b"unknown" in lib.kr_status_string(42)


def test_host_validation_without_gpu():
    from paper_2601_17654_amd import binding as b
    from paper_2601_17654_amd import inputs as I

    L = b._lib
    sp = b._space(I.SPACES[0]["space"])
    null = ctypes.c_void_p(0)
    assert L.kr_evaluate_partition(ctypes.byref(sp), null, null, null, null, null, null,
                                   null, null) == b.KR_EINVAL
    bad = b.KrSpace(1, 4, 3, 1, 1, 5, 90.0)  # three comm kernels
    assert L.kr_candidates_per_partition(ctypes.byref(bad)) == 0
    bad = b.KrSpace(1, 4, 1, 1, 1, 6, 90.0)  # n_pos > N + 1
    assert L.kr_candidates_per_partition(ctypes.byref(bad)) == 0
    # a slab that cannot fit on chip is refused before any launch
    huge = b.KrSpace(1, 400, 1, 1, 40, 401, 90.0)
    one = ctypes.c_void_p(8)
    assert L.kr_evaluate_partition(ctypes.byref(huge), one, one, one, one, one, one,
                                   null, null) == b.KR_EUNSUPPORTED
    assert L.kr_evaluate_and_filter_workspace(ctypes.byref(huge)) == 0
    # workspace sizes grow with the problem
    assert L.kr_pareto_filter_workspace(10, 1) < L.kr_pareto_filter_workspace(10 ** 6, 8)
    assert L.kr_compose_frontiers_workspace(4, 1024) < L.kr_compose_frontiers_workspace(512, 65536)
    assert L.kr_compose_frontiers_workspace(0, 1024) == 0
    # too small a workspace is refused on the host
    assert L.kr_compose_frontiers(4, one, one, one, 1024, 0.0, one, one, one, one, one, one, one,
                                  one, one, one, one, one, 16, null) == b.KR_ECAPACITY
    assert L.kr_compose_frontiers(4, one, one, one, 1024, -1.0, one, one, one, one, one, one, one,
                                  one, one, one, one, one, 1 << 30, null) == b.KR_EINVAL
    assert b.candidates_per_partition(I.SPACES[2]["space"]) == 1148928
    # scores and selection: shapes and counts are checked before any launch
    assert L.kr_hvi_scores_workspace(0, 10) == 0 and L.kr_hvi_scores_workspace(4, 0) == 0
    assert L.kr_select_batch_workspace(0, 10) == 0
    assert L.kr_hvi_scores(2, 10, one, one, one, 8, one, one, one, 90.0, one, one, one, one, one,
                           16, null) == b.KR_ECAPACITY
    assert L.kr_hvi_scores(2, 10, null, one, one, 8, one, one, one, 90.0, one, one, one, one, one,
                           1 << 20, null) == b.KR_EINVAL
    big = 1 << 20
    for ks in ((13, 6, 6, 32), (0, 0, 0, 0), (64, 0, 0, 64)):
        assert L.kr_select_batch(1, 10, one, one, one, one, one, *ks, one, one, one, one, 16,
                                 null) == b.KR_ECAPACITY
    for ks in ((13, 6, 6, 24), (-1, 0, 0, 4), (0, 0, 0, 65)):
        assert L.kr_select_batch(1, 10, one, one, one, one, one, *ks, one, one, one, one, big,
                                 null) == b.KR_EINVAL
    assert L.kr_uncertainty(0, 10, one, one, one, null) == b.KR_EINVAL
    assert L.kr_compare_frontiers(0, one, one, 1, one, one, one, one, big, null) == b.KR_EINVAL
    assert L.kr_compare_frontiers(1, one, one, 1, one, one, one, one, 8, null) == b.KR_ECAPACITY
    kind = (ctypes.c_int32 * 30)(*([0] * 29 + [2]))
    for n, I_, J_, kmax, cap in ((1, 25, 1, 1, 8), (1, 0, 0, 1, 8), (1, 3, 3, 17, 8),
                                 (1, 3, 3, 1, 65), (1, 3, 3, 1, 0), (1, 29, 1, 1, 8)):
        assert L.kr_launch_timing_frontier(n, I_, J_, kind, one, 90.0, kmax, cap, one, one, one,
                                           one, one, one, big, null) == b.KR_EINVAL
    assert L.kr_launch_timing_frontier(4, 3, 3, kind, one, 90.0, 2, 8, one, one, one, one, one,
                                       one, 4, null) == b.KR_ECAPACITY
    assert L.kr_uncertainty(65, 10, one, one, one, null) == b.KR_EINVAL


def test_hv_stopping_rule_matches_oracle():
    """The library's host stopping rule against the oracle's on hand-made histories."""
    import oracle
    from paper_2601_17654_amd import binding as b

    cases = [[1.0, 1.0005, 1.0006], [1.0, 1.1, 1.1001], [1.0, 1.0], [1.0, 1.0, 1.0],
             [0.0, 0.0, 1.0, 1.0], [0.0, 1.0, 1.0, 1.0], [2.0, 2.001, 2.0021, 2.0022, 2.00225]]
    for h in cases:
        for R in (1, 2, 3):
            for eps in (1e-3, 1e-4):
                assert b.hv_converged(h, R, eps) == oracle.hv_converged(h, R, eps), (h, R, eps)


def test_oracle_and_library_share_nothing():
    """The oracle neither includes the library's header nor loads it, and the library's
    sources never mention the oracle."""
    src = open(os.path.join(ROOT, "oracle", "kareus_oracle.c")).read()
    assert "kareus.h" not in src and "libkareus" not in src
    py = open(os.path.join(ROOT, "oracle", "__init__.py")).read()
    assert "paper_2601_17654_amd" not in py and "libkareus" not in py
    csrc = os.path.join(ROOT, "paper_2601_17654_amd", "csrc")
    for f in os.listdir(csrc):
        assert "oracle" not in open(os.path.join(csrc, f)).read().lower(), f
    for f in ("binding.py", "build.py", "__init__.py", "inputs.py"):
        text = open(os.path.join(ROOT, "paper_2601_17654_amd", f)).read()
        assert not re.search(r"^\s*(import|from)\s+oracle", text, flags=re.M), f
