"""CPU oracle for the Kareus schedule-search hot path -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
package.  It loads `liboracle.so`, built from `kareus_oracle.c` with gcc (no FMA
contraction, no fast-math), and wraps it with numpy arrays.  It shares no code with
the HIP library and never imports it.

The C source cites, per function, the passage of the paper it follows.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kareus_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc; returns the library path."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        lp = ctypes.POINTER(ctypes.c_int64)
        i, d = ctypes.c_int, ctypes.c_double
        lib.oracle_evaluate.argtypes = [i, i, i, i, i, d, dp, dp, dp, dp, dp, dp]
        lib.oracle_pareto.argtypes = [ctypes.c_int64, dp, dp, ip, lp]
        lib.oracle_compose.argtypes = [i, lp, dp, dp, i, d, dp, ip, ip, dp, ip]
        lib.oracle_staircase.argtypes = [i, dp, d, d, ip, dp, dp, ip]
        lib.oracle_extract.argtypes = [i, i, lp, dp, dp, ip, ip, ctypes.c_int32, ip, dp, dp]
        lib.oracle_microbatch.argtypes = [i, i, lp, dp, dp, i, ip, i, dp, dp, i,
                                          ctypes.c_int64, dp, dp, ip, ip, lp]
        lib.oracle_microbatch_exact.argtypes = [i, i, lp, dp, dp, i, ip, i, dp, dp,
                                                ctypes.c_int64, dp, dp, ip, ip, lp]
        lib.oracle_hypervolume.argtypes = [ctypes.c_int64, dp, dp, d, d, dp]
        lib.oracle_hvi.argtypes = [i, lp, dp, dp, lp, dp, dp, d, dp, dp, dp]
        lib.oracle_uncertainty.argtypes = [i, ctypes.c_int64, dp, dp, dp]
        lib.oracle_select.argtypes = [i, lp, dp, dp, lp, lp, i, i, i, i, lp, ip]
        lib.oracle_hv_converged.argtypes = [i, dp, i, d]
        lib.oracle_compare.argtypes = [ctypes.c_int64, dp, dp, ctypes.c_int64, dp, dp, dp]
        lib.oracle_launch_dp.argtypes = [i, i, ip, dp, d, i, ctypes.c_int64, dp, dp, ip, lp, lp]
        for fn in ("oracle_evaluate", "oracle_pareto", "oracle_compose", "oracle_staircase",
                   "oracle_extract", "oracle_microbatch", "oracle_microbatch_exact",
                   "oracle_hypervolume", "oracle_hvi", "oracle_uncertainty", "oracle_select",
                   "oracle_hv_converged", "oracle_compare", "oracle_launch_dp"):
            getattr(lib, fn).restype = ctypes.c_int
        _lib = lib
    return _lib


def _p(a: np.ndarray, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


class OracleError(RuntimeError):
    pass


def evaluate_partition(space, t, pw, tc, pc, part: int = 0):
    """Time and energy of every candidate of partition `part`: (T, E) float64[n_cand]."""
    lib = _load()
    tp, pwp = _f64(t[part]), _f64(pw[part])
    tcp, pcp = _f64(tc[part]), _f64(pc[part])
    n = space.n_cand
    T = np.empty(n)
    E = np.empty(n)
    rc = lib.oracle_evaluate(space.n_kernels, space.n_comm, space.n_freq, space.n_sm,
                             space.n_pos, float(space.p_static), _p(tp, ctypes.c_double),
                             _p(pwp, ctypes.c_double), _p(tcp, ctypes.c_double),
                             _p(pcp, ctypes.c_double), _p(T, ctypes.c_double),
                             _p(E, ctypes.c_double))
    if rc != 0:
        raise OracleError("oracle_evaluate failed: %d" % rc)
    return T, E


def pareto(T, E):
    """Indices of the non-dominated points, in ascending time."""
    lib = _load()
    T, E = _f64(T), _f64(E)
    out = np.empty(max(len(T), 1), dtype=np.int32)
    n_out = ctypes.c_int64(0)
    rc = lib.oracle_pareto(len(T), _p(T, ctypes.c_double), _p(E, ctypes.c_double),
                           _p(out, ctypes.c_int32), ctypes.byref(n_out))
    if rc != 0:
        raise OracleError("oracle_pareto failed: %d" % rc)
    return out[: n_out.value].copy()


def evaluate_and_filter(space, t, pw, tc, pc, parts: Optional[range] = None,
                        threads: int = 1):
    """Per partition: (frontier candidate indices, T, E).  With threads > 1 the partitions
    (independent) are spread over that many threads; each partition still runs the plain
    single-threaded evaluation and GetFrontier, so the results are the same."""
    ps = list(parts if parts is not None else range(space.n_parts))

    def one(p):
        T, E = evaluate_partition(space, t, pw, tc, pc, p)
        idx = pareto(T, E)
        return idx, T[idx], E[idx]

    if threads <= 1:
        return [one(p) for p in ps]
    import concurrent.futures as cf

    _load()  # load once, before the threads
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(one, ps))


class Composed:
    def __init__(self, F, bp, pt_bin, delta, tmin_sum, L):
        self.F, self.bp, self.pt_bin = F, bp, pt_bin
        self.delta, self.tmin_sum, self.L = delta, tmin_sum, L


def compose(off, T, E, n_bins: int, delta: float = 0.0) -> Composed:
    lib = _load()
    off = np.ascontiguousarray(off, dtype=np.int64)
    T, E = _f64(T), _f64(E)
    P = len(off) - 1
    F = np.empty(n_bins)
    bp = np.empty((P, n_bins), dtype=np.int32)
    pt = np.empty(max(int(off[-1]), 1), dtype=np.int32)
    info = np.empty(2)
    L = ctypes.c_int32(0)
    rc = lib.oracle_compose(P, _p(off, ctypes.c_int64), _p(T, ctypes.c_double),
                            _p(E, ctypes.c_double), n_bins, float(delta),
                            _p(F, ctypes.c_double), _p(bp, ctypes.c_int32),
                            _p(pt, ctypes.c_int32), _p(info, ctypes.c_double), ctypes.byref(L))
    if rc != 0:
        raise OracleError("oracle_compose failed: %d" % rc)
    return Composed(F, bp, pt[: int(off[-1])], float(info[0]), float(info[1]), int(L.value))


def staircase(F, delta: float, tmin_sum: float):
    """(bins int32, T_lo float64, E float64) of the non-dominated composite bins."""
    lib = _load()
    F = _f64(F)
    B = len(F)
    bins = np.empty(B, dtype=np.int32)
    tlo = np.empty(B)
    e = np.empty(B)
    n = ctypes.c_int32(0)
    lib.oracle_staircase(B, _p(F, ctypes.c_double), float(delta), float(tmin_sum),
                         _p(bins, ctypes.c_int32), _p(tlo, ctypes.c_double),
                         _p(e, ctypes.c_double), ctypes.byref(n))
    k = n.value
    return bins[:k].copy(), tlo[:k].copy(), e[:k].copy()


def extract(off, T, E, comp: Composed, bin_: int):
    """(choice int32[P], T_sum, E_sum) behind composite bin `bin_`."""
    lib = _load()
    off = np.ascontiguousarray(off, dtype=np.int64)
    T, E = _f64(T), _f64(E)
    P = len(off) - 1
    B = comp.bp.shape[1]
    choice = np.empty(P, dtype=np.int32)
    ts = ctypes.c_double(0.0)
    es = ctypes.c_double(0.0)
    bp = np.ascontiguousarray(comp.bp, dtype=np.int32)
    pt = np.ascontiguousarray(comp.pt_bin, dtype=np.int32)
    rc = lib.oracle_extract(P, B, _p(off, ctypes.c_int64), _p(T, ctypes.c_double),
                            _p(E, ctypes.c_double), _p(bp, ctypes.c_int32),
                            _p(pt, ctypes.c_int32), int(bin_), _p(choice, ctypes.c_int32),
                            ctypes.byref(ts), ctypes.byref(es))
    if rc != 0:
        raise OracleError("oracle_extract failed for bin %d: %d" % (bin_, rc))
    return choice, ts.value, es.value


def microbatch(seg_off, T, E, n_types: int, n_freq: int, seq, comp_T=None, comp_E=None,
               n_bins: int = 4096):
    """Microbatch frontier (Algorithm 2 with one frequency per microbatch and one choice
    per partition type).  seg_off [K*F+1]: segment t*F+f holds type t's points at
    frequency f.  comp_T, comp_E [n_comp][F] or None.
    Returns (T, E, f int32, choice int32[n][K]) in ascending time."""
    lib = _load()
    seg_off = np.ascontiguousarray(seg_off, dtype=np.int64)
    T, E = _f64(T), _f64(E)
    seq = np.ascontiguousarray(seq, dtype=np.int32)
    if comp_T is None:
        cT = np.zeros((0, n_freq))
        cE = np.zeros((0, n_freq))
    else:
        cT, cE = _f64(comp_T).reshape(-1, n_freq), _f64(comp_E).reshape(-1, n_freq)
    cap = n_freq * n_bins
    oT, oE = np.empty(cap), np.empty(cap)
    of = np.empty(cap, dtype=np.int32)
    och = np.empty((cap, n_types), dtype=np.int32)
    n = ctypes.c_int64(0)
    rc = lib.oracle_microbatch(n_types, n_freq, _p(seg_off, ctypes.c_int64),
                               _p(T, ctypes.c_double), _p(E, ctypes.c_double), len(seq),
                               _p(seq, ctypes.c_int32), cT.shape[0], _p(cT, ctypes.c_double),
                               _p(cE, ctypes.c_double), n_bins, cap, _p(oT, ctypes.c_double),
                               _p(oE, ctypes.c_double), _p(of, ctypes.c_int32),
                               _p(och, ctypes.c_int32), ctypes.byref(n))
    if rc != 0:
        raise OracleError("oracle_microbatch failed: %d" % rc)
    k = min(n.value, cap)
    return oT[:k].copy(), oE[:k].copy(), of[:k].copy(), och[:k].copy()


def microbatch_exact(seg_off, T, E, n_types: int, n_freq: int, seq, comp_T=None, comp_E=None):
    """Microbatch frontier by enumerating every configuration (Algorithm 2 as written).
    Returns (T, E, f int32, choice int32[n][K]) in ascending time."""
    lib = _load()
    seg_off = np.ascontiguousarray(seg_off, dtype=np.int64)
    T, E = _f64(T), _f64(E)
    seq = np.ascontiguousarray(seq, dtype=np.int32)
    if comp_T is None:
        cT = np.zeros((0, n_freq))
        cE = np.zeros((0, n_freq))
    else:
        cT, cE = _f64(comp_T).reshape(-1, n_freq), _f64(comp_E).reshape(-1, n_freq)
    sizes = np.diff(seg_off).reshape(n_types, n_freq)
    used = sorted(set(seq.tolist()))
    cap = max(int(np.sum(np.prod(sizes[used], axis=0))), 1)
    oT, oE = np.empty(cap), np.empty(cap)
    of = np.empty(cap, dtype=np.int32)
    och = np.empty((cap, n_types), dtype=np.int32)
    n = ctypes.c_int64(0)
    rc = lib.oracle_microbatch_exact(n_types, n_freq, _p(seg_off, ctypes.c_int64),
                                     _p(T, ctypes.c_double), _p(E, ctypes.c_double), len(seq),
                                     _p(seq, ctypes.c_int32), cT.shape[0],
                                     _p(cT, ctypes.c_double), _p(cE, ctypes.c_double), cap,
                                     _p(oT, ctypes.c_double), _p(oE, ctypes.c_double),
                                     _p(of, ctypes.c_int32), _p(och, ctypes.c_int32),
                                     ctypes.byref(n))
    if rc != 0:
        raise OracleError("oracle_microbatch_exact failed: %d" % rc)
    k = min(n.value, cap)
    return oT[:k].copy(), oE[:k].copy(), of[:k].copy(), och[:k].copy()


def hypervolume(T, E, rT: float, rE: float) -> float:
    """HV of the points (T, E) against the reference point (rT, rE) (Section 4.3)."""
    lib = _load()
    T, E = _f64(T), _f64(E)
    out = ctypes.c_double(0.0)
    rc = lib.oracle_hypervolume(T.shape[0], _p(T, ctypes.c_double), _p(E, ctypes.c_double),
                                float(rT), float(rE), ctypes.byref(out))
    if rc != 0:
        raise OracleError("oracle_hypervolume failed: %d" % rc)
    return out.value


def hvi(cand_off, T_hat, E_hat, obs_off, T_obs, E_obs, p_static: float):
    """Exploitation scores of Algorithm 1 (total, dynamic, static energy).
    Returns (hvi float64[3][n_cand], hv float64[n_seg][3], ref float64[n_seg][4])."""
    lib = _load()
    cand_off = np.ascontiguousarray(cand_off, dtype=np.int64)
    obs_off = np.ascontiguousarray(obs_off, dtype=np.int64)
    T_hat, E_hat, T_obs, E_obs = _f64(T_hat), _f64(E_hat), _f64(T_obs), _f64(E_obs)
    n_seg = cand_off.shape[0] - 1
    n = int(cand_off[-1]) if n_seg > 0 else 0
    out = np.empty((3, n))
    hv = np.empty((max(n_seg, 0), 3))
    ref = np.empty((max(n_seg, 0), 4))
    rc = lib.oracle_hvi(n_seg, _p(cand_off, ctypes.c_int64), _p(T_hat, ctypes.c_double),
                        _p(E_hat, ctypes.c_double), _p(obs_off, ctypes.c_int64),
                        _p(T_obs, ctypes.c_double), _p(E_obs, ctypes.c_double),
                        float(p_static), _p(out, ctypes.c_double), _p(hv, ctypes.c_double),
                        _p(ref, ctypes.c_double))
    if rc != 0:
        raise OracleError("oracle_hvi failed: %d" % rc)
    return out, hv, ref


def uncertainty(Tm, Em):
    """Exploration score: population std over ensemble members of T plus that of E.
    Tm, Em: [M][n]."""
    lib = _load()
    Tm, Em = _f64(Tm), _f64(Em)
    M, n = Tm.shape
    out = np.empty(n)
    rc = lib.oracle_uncertainty(M, n, _p(Tm, ctypes.c_double), _p(Em, ctypes.c_double),
                                _p(out, ctypes.c_double))
    if rc != 0:
        raise OracleError("oracle_uncertainty failed: %d" % rc)
    return out


def select(cand_off, score, unc, obs_off, obs_idx, k1: int, k2: int, k3: int, k: int):
    """Multi-pass candidate selection of Algorithm 1.  score [3][n_cand], unc [n_cand] or
    None, obs_idx local indices.  Returns a list of int64 arrays, one per partition."""
    lib = _load()
    cand_off = np.ascontiguousarray(cand_off, dtype=np.int64)
    obs_off = np.ascontiguousarray(obs_off, dtype=np.int64)
    obs_idx = np.ascontiguousarray(obs_idx, dtype=np.int64)
    score = _f64(score)
    n_seg = cand_off.shape[0] - 1
    uncp = None if unc is None else _f64(unc)
    sel = np.full((max(n_seg, 1), max(k, 1)), -1, dtype=np.int64)
    cnt = np.zeros(max(n_seg, 1), dtype=np.int32)
    rc = lib.oracle_select(n_seg, _p(cand_off, ctypes.c_int64), _p(score, ctypes.c_double),
                           None if uncp is None else _p(uncp, ctypes.c_double),
                           _p(obs_off, ctypes.c_int64), _p(obs_idx, ctypes.c_int64),
                           k1, k2, k3, k, _p(sel, ctypes.c_int64), _p(cnt, ctypes.c_int32))
    if rc != 0:
        raise OracleError("oracle_select failed: %d" % rc)
    return [sel[g, :cnt[g]].copy() for g in range(n_seg)]


def hv_converged(hv_history, R: int = 2, eps: float = 1e-3) -> bool:
    """Stopping rule of Algorithm 1 (Appendix C)."""
    lib = _load()
    h = _f64(hv_history)
    return bool(lib.oracle_hv_converged(h.shape[0], _p(h, ctypes.c_double), R, float(eps)))


def compare(TA, EA, TB, EB) -> np.ndarray:
    """Frontier metrics of B against baseline A (Section 6.1): float64[10] =
    (leftmost time red. %, leftmost energy red. %, iso-time energy red. %,
     iso-energy time red. %, d, E_A(d), E_B(d), b, T_A(b), T_B(b))."""
    lib = _load()
    TA, EA, TB, EB = _f64(TA), _f64(EA), _f64(TB), _f64(EB)
    out = np.empty(10)
    rc = lib.oracle_compare(TA.shape[0], _p(TA, ctypes.c_double), _p(EA, ctypes.c_double),
                            TB.shape[0], _p(TB, ctypes.c_double), _p(EB, ctypes.c_double),
                            _p(out, ctypes.c_double))
    if rc != 0:
        raise OracleError("oracle_compare failed: %d" % rc)
    return out


def launch_dp(kind1, kind2, ops, p_static: float, kmax: int):
    """Launch-timing frontier of two operation sequences (Appendix B).  kind1 [I],
    kind2 [J]: 0 computation, 1 communication; ops [I + J][4] (S1's ops, then S2's).
    Returns (T, E, schedules int32[n][I + J], stats) with stats = (largest cell
    frontier, frontier points of all cells, most candidates of a cell)."""
    lib = _load()
    kind = np.ascontiguousarray(np.concatenate([np.asarray(kind1), np.asarray(kind2)]),
                                dtype=np.int32)
    I, J = len(kind1), len(kind2)
    ops = _f64(ops).reshape(I + J, 4)
    cap = 4096
    oT, oE = np.empty(cap), np.empty(cap)
    sched = np.empty((cap, I + J), dtype=np.int32)
    n = ctypes.c_int64(0)
    st = np.zeros(3, dtype=np.int64)
    rc = lib.oracle_launch_dp(I, J, _p(kind, ctypes.c_int32), _p(ops, ctypes.c_double),
                              float(p_static), kmax, cap, _p(oT, ctypes.c_double),
                              _p(oE, ctypes.c_double), _p(sched, ctypes.c_int32),
                              ctypes.byref(n), _p(st, ctypes.c_int64))
    if rc != 0:
        raise OracleError("oracle_launch_dp failed: %d" % rc)
    k = min(n.value, cap)
    return oT[:k].copy(), oE[:k].copy(), sched[:k].copy(), tuple(int(x) for x in st)


def decode(space, idx: int):
    """Candidate index -> (f, positions tuple, SM-choice tuple), the oracle's order."""
    S = space.n_sm
    if space.n_comm == 1:
        s = idx % S
        rest = idx // S
        return rest // space.n_pos, (rest % space.n_pos,), (s,)
    s2 = idx % S
    s1 = (idx // S) % S
    rest = idx // (S * S)
    f, pp = divmod(rest, space.n_pairs)
    for p1 in range(space.n_pos):
        width = space.n_pos - p1
        if pp < width:
            return f, (p1, p1 + pp), (s1, s2)
        pp -= width
    raise ValueError(idx)
