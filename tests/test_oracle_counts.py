"""Search-space size pins (Section 4.1 and Appendix B) and the workload shapes."""

import os

from paper_2601_17654_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    vals = {}
    with open(os.path.join(GOLDEN, "search_space_counts.txt")) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            k, v = line.split()
            vals[k] = int(v)
    return vals


def test_paper_solution_space_size():
    """Appendix B: 35 frequencies x 30 SM allocations x 81 launch groupings = 85,050
    candidates, and ~13 s of profiling each makes 307 h, 4,912 GPU-hours on 16 GPUs."""
    g = _golden()
    freqs = range(g["freq_lo_mhz"], g["freq_hi_mhz"] + 1, g["freq_stride_mhz"])
    assert len(freqs) == g["freq_choices"]
    sp = I.Space(1, g["launch_groupings"] - 1, 1, g["launch_groupings"],
                 tuple(range(1, g["sm_choices"] + 1)), tuple(float(f) for f in freqs))
    assert sp.n_cand == g["total_candidates"]
    hours = sp.n_cand * g["seconds_per_candidate"] / 3600.0
    assert round(hours) == g["exhaustive_hours"]
    assert g["exhaustive_hours"] * g["gpus"] == g["exhaustive_gpu_hours"]


def test_workload_candidate_counts(oracle_lib):
    expect = {0: 896, 1: 25600, 2: 1148928, 3: 135168}
    for cfg, n in expect.items():
        sp = I.SPACES[cfg]["space"]
        assert sp.n_cand == n
    assert I.SPACES[2]["space"].n_pairs == 561
    assert I.SPACES[3]["space"].n_cand * I.SPACES[3]["space"].n_parts == 138412032
    # the oracle enumerates exactly that many candidates
    w = I.config_workload(0)
    T, E = oracle_lib.evaluate_partition(w.space, w.t, w.pw, w.tc, w.pc, 0)
    assert len(T) == 896


def test_generator_is_deterministic_and_in_range():
    a = I.config_workload(0)
    b = I.config_workload(0)
    for k in ("t", "pw", "tc", "pc"):
        assert (getattr(a, k) == getattr(b, k)).all()
    sp = a.space
    t_max_all = a.t[:, -1, :, 0]  # top frequency, all SMs: t0 itself
    assert (t_max_all >= 20e-6 * (1 - 1e-12)).all() and (t_max_all <= 2e-3 * (1 + 1e-12)).all()
    assert (a.pc > 0).all() and (a.tc > 0).all()
    # a sub-range of partitions draws the same numbers as the full batch
    part = I.config_workload(0, parts=range(2, 4))
    assert (part.t == a.t[2:4]).all() and (part.tc == a.tc[2:4]).all()
    off, T, E = I.compose_frontiers(n_parts=8)
    assert off[-1] == len(T) and (T > 0).all() and (E <= 1.0).all() and (E >= 0.5 - 1e-12).all()
