"""Python binding of libkareus_mi355x.so (the C ABI in include/kareus.h).

Argument marshalling only: every step runs in the library's HIP kernels.  PyTorch
provides device memory and the current HIP stream.  The functions carry the C names
without the `kr_` prefix.  Importing this module loads the library and fails loudly
if it has not been built.
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkareus_mi355x.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError("libkareus_mi355x.so is not built (run __graft_entry__.build() or "
                      "python paper_2601_17654_amd/build.py)")
_lib = ctypes.CDLL(_LIB_PATH)

KR_OK, KR_EINVAL, KR_ENONFINITE, KR_ECAPACITY, KR_EHIP, KR_EUNSUPPORTED = 0, -1, -2, -3, -4, -5


class KrSpace(ctypes.Structure):
    _fields_ = [("n_parts", ctypes.c_int32), ("n_kernels", ctypes.c_int32),
                ("n_comm", ctypes.c_int32), ("n_freq", ctypes.c_int32),
                ("n_sm", ctypes.c_int32), ("n_pos", ctypes.c_int32),
                ("p_static", ctypes.c_double)]


_vp, _i32, _i64, _f64, _sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                              ctypes.c_double, ctypes.c_size_t)
_SP = ctypes.POINTER(KrSpace)
_SIGS = {
    "kr_evaluate_partition": (_i32, [_SP, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "kr_candidates_per_partition": (_i64, [_SP]),
    "kr_pareto_filter": (_i32, [_i64, _vp, _vp, _vp, _i32, _i64, _vp, _vp, _vp, _vp, _vp, _vp,
                                _sz, _vp]),
    "kr_pareto_filter_workspace": (_sz, [_i64, _i32]),
    "kr_pareto_filter_noalloc": (_i32, [_i64, _vp, _vp, _vp, _i32, _i64, _vp, _vp, _vp, _vp, _vp,
                                        _vp]),
    "kr_evaluate_and_filter": (_i32, [_SP, _vp, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp,
                                      _vp, _sz, _vp]),
    "kr_evaluate_and_filter_workspace": (_sz, [_SP]),
    "kr_compose_frontiers": (_i32, [_i32, _vp, _vp, _vp, _i32, _f64, _vp, _vp, _vp, _vp, _vp, _vp,
                                    _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "kr_compose_frontiers_workspace": (_sz, [_i32, _i32]),
    "kr_extract_schedule": (_i32, [_i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp,
                                   _vp, _vp, _vp, _vp, _vp]),
    "kr_decode_candidates": (_i32, [_SP, _vp, _i64, _vp, _vp, _vp, _vp]),
    "kr_microbatch_frontier": (_i32, [_i32, _i32, _vp, _vp, _vp, _i64, _i32, _vp, _i32, _vp, _vp,
                                      _i32, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "kr_microbatch_frontier_workspace": (_sz, [_i32, _i32, _i64, _i32, _i32]),
    "kr_microbatch_enumerate": (_i32, [_i32, _i32, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _i64,
                                       _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "kr_microbatch_enumerate_workspace": (_sz, [_i32, _i32, _i64]),
    "kr_hvi_scores": (_i32, [_i32, _i64, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _f64, _vp, _vp, _vp,
                             _vp, _vp, _sz, _vp]),
    "kr_hvi_scores_workspace": (_sz, [_i32, _i64]),
    "kr_uncertainty": (_i32, [_i32, _i64, _vp, _vp, _vp, _vp]),
    "kr_select_batch": (_i32, [_i32, _i64, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _vp,
                               _vp, _vp, _vp, _sz, _vp]),
    "kr_select_batch_workspace": (_sz, [_i32, _i64]),
    "kr_hv_converged": (_i32, [_i32, _vp, _i32, _f64]),
    "kr_compare_frontiers": (_i32, [_i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _sz, _vp]),
    "kr_compare_frontiers_workspace": (_sz, []),
    "kr_launch_timing_frontier": (_i32, [_i64, _i32, _i32, _vp, _vp, _f64, _i32, _i32, _vp, _vp,
                                         _vp, _vp, _vp, _vp, _sz, _vp]),
    "kr_launch_timing_frontier_workspace": (_sz, [_i64]),
    "kr_status_string": (ctypes.c_char_p, [_i32]),
    "kr_set_phase_events": (_i32, [_i32, _vp, _vp]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args


class KrError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__("%s: %s (%d)" % (fn, status_string(status), status))
        self.status = status


def status_string(status: int) -> str:
    return _lib.kr_status_string(int(status)).decode()


def _check(fn: str, status: int) -> None:
    if status != KR_OK:
        raise KrError(fn, status)


def _status_word(validate: bool):
    """Device status word for an entry point's input check, or None to skip it."""
    return torch.empty(1, dtype=torch.int32, device="cuda") if validate else None


def _check_status(fn: str, status: Optional[torch.Tensor]) -> None:
    """Raises KrError if the device status word of an input check is not KR_OK (reads it
    back, so the stream is synchronised)."""
    if status is not None:
        _check(fn, int(status.item()))


def _space(space) -> KrSpace:
    return KrSpace(space.n_parts, space.n_kernels, space.n_comm, space.n_freq, space.n_sm,
                   space.n_pos, float(space.p_static))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(x, dtype, name: str) -> torch.Tensor:
    if not isinstance(x, torch.Tensor):
        x = torch.as_tensor(np.ascontiguousarray(x))
    if x.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, x.dtype))
    if not x.is_cuda:
        x = x.cuda()
    return x.contiguous()


_ws_cache = {}


def _workspace(nbytes: int) -> torch.Tensor:
    dev = torch.cuda.current_device()
    buf = _ws_cache.get(dev)
    if buf is None or buf.numel() < nbytes:
        buf = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")
        _ws_cache[dev] = buf
    return buf


PHASE_EVAL_TILE, PHASE_MERGE, PHASE_MINPLUS, PHASE_HVI, PHASE_SELECT, PHASE_UNC = range(6)


def set_phase_events(phase: int, start=None, stop=None) -> None:
    """Record torch.cuda.Event pairs around a library phase (None switches it off)."""
    a = ctypes.c_void_p(start.cuda_event) if start is not None else None
    b = ctypes.c_void_p(stop.cuda_event) if stop is not None else None
    _check("kr_set_phase_events", _lib.kr_set_phase_events(phase, a, b))


def candidates_per_partition(space) -> int:
    return int(_lib.kr_candidates_per_partition(ctypes.byref(_space(space))))


def evaluate_partition(space, t, pw, tc, pc, T_out=None, E_out=None, validate: bool = True):
    """Time and energy of every candidate: (T, E), float64 [P][C] on the device.  With
    validate, the library checks the tables first and a non-finite or negative value
    raises KrError(KR_ENONFINITE) (the call then waits for the stream)."""
    sp = _space(space)
    C = candidates_per_partition(space)
    t, pw = _dev(t, torch.float64, "t"), _dev(pw, torch.float64, "pw")
    tc, pc = _dev(tc, torch.float64, "tc"), _dev(pc, torch.float64, "pc")
    _check_tables(space, t, pw, tc, pc)
    if T_out is None:
        T_out = torch.empty((space.n_parts, C), dtype=torch.float64, device="cuda")
    if E_out is None:
        E_out = torch.empty((space.n_parts, C), dtype=torch.float64, device="cuda")
    status = _status_word(validate)
    _check("kr_evaluate_partition",
           _lib.kr_evaluate_partition(ctypes.byref(sp), _ptr(t), _ptr(pw), _ptr(tc), _ptr(pc),
                                      _ptr(T_out), _ptr(E_out), _ptr(status), _stream()))
    _check_status("kr_evaluate_partition", status)
    return T_out, E_out


def _check_tables(space, t, pw, tc, pc):
    P, F, N, S, M = space.n_parts, space.n_freq, space.n_kernels, space.n_sm, space.n_comm
    if tuple(t.shape) != (P, F, N, S + 1) or tuple(pw.shape) != (P, F, N, S + 1):
        raise ValueError("t/pw must be [P][F][N][S+1] = %s" % ((P, F, N, S + 1),))
    if tuple(tc.shape) != (P, F, M, S) or tuple(pc.shape) != (P, F, M, S):
        raise ValueError("tc/pc must be [P][F][M][S] = %s" % ((P, F, M, S),))


@dataclasses.dataclass
class Frontier:
    """Per-segment frontiers in CSR form (device tensors)."""
    off: torch.Tensor   # int64 [n_seg + 1]
    idx: torch.Tensor   # int32 [total]
    T: torch.Tensor     # float64 [total]
    E: torch.Tensor     # float64 [total]


def _finish_frontier(off, idx, T, E, cap, sync):
    if not sync:
        return Frontier(off, idx, T, E), True
    torch.cuda.current_stream().synchronize()
    total = int(off[-1].item())
    if total > cap:
        return None, total
    return Frontier(off, idx[:total], T[:total], E[:total]), True


NOALLOC_MAX_POINTS, NOALLOC_MAX_SEGS = 1 << 20, 1 << 16


def pareto_filter(T, E, seg_off, cap: Optional[int] = None, sync: bool = True,
                  validate: Optional[bool] = None, noalloc: bool = False) -> Frontier:
    """GetFrontier of every segment [seg_off[g], seg_off[g+1]) of (T, E).  validate
    (default: sync) has the library check T and E, raising KrError(KR_ENONFINITE).
    noalloc calls kr_pareto_filter_noalloc (library-held workspace, bounded sizes)."""
    seg_host = np.asarray(seg_off.cpu() if isinstance(seg_off, torch.Tensor) else seg_off,
                          dtype=np.int64)
    n_seg = len(seg_host) - 1
    if n_seg < 0 or seg_host[0] != 0 or np.any(np.diff(seg_host) < 0):
        raise ValueError("seg_off must start at 0 and be non-decreasing")
    T = _dev(T, torch.float64, "T").reshape(-1)
    E = _dev(E, torch.float64, "E").reshape(-1)
    n_total = int(seg_host[-1])
    if T.numel() != n_total or E.numel() != n_total:
        raise ValueError("T/E must hold seg_off[-1] points")
    seg_dev = torch.from_numpy(seg_host).cuda()
    while True:
        c = int(cap) if cap is not None else min(n_total, max(4096 * max(n_seg, 1), 1))
        off = torch.empty(n_seg + 1, dtype=torch.int64, device="cuda")
        idx = torch.empty(max(c, 1), dtype=torch.int32, device="cuda")
        oT = torch.empty(max(c, 1), dtype=torch.float64, device="cuda")
        oE = torch.empty(max(c, 1), dtype=torch.float64, device="cuda")
        status = _status_word(sync if validate is None else validate)
        if noalloc:
            fn = "kr_pareto_filter_noalloc"
            rc = _lib.kr_pareto_filter_noalloc(n_total, _ptr(T), _ptr(E), _ptr(seg_dev), n_seg, c,
                                               _ptr(off), _ptr(idx), _ptr(oT), _ptr(oE),
                                               _ptr(status), _stream())
        else:
            fn = "kr_pareto_filter"
            wsb = _lib.kr_pareto_filter_workspace(n_total, n_seg)
            ws = _workspace(wsb)
            rc = _lib.kr_pareto_filter(n_total, _ptr(T), _ptr(E), _ptr(seg_dev), n_seg, c,
                                       _ptr(off), _ptr(idx), _ptr(oT), _ptr(oE), _ptr(status),
                                       _ptr(ws), wsb, _stream())
        _check(fn, rc)
        _check_status(fn, status)
        fr, ok = _finish_frontier(off, idx, oT, oE, c, sync)
        if fr is not None:
            return fr
        cap = ok  # the exact size


def evaluate_and_filter(space, t, pw, tc, pc, cap: Optional[int] = None,
                        sync: bool = True, validate: Optional[bool] = None) -> Frontier:
    """Fused evaluation + GetFrontier, one segment per partition; idx = candidate index.
    validate (default: sync) has the library check the tables first, raising
    KrError(KR_ENONFINITE)."""
    sp = _space(space)
    t, pw = _dev(t, torch.float64, "t"), _dev(pw, torch.float64, "pw")
    tc, pc = _dev(tc, torch.float64, "tc"), _dev(pc, torch.float64, "pc")
    _check_tables(space, t, pw, tc, pc)
    C = candidates_per_partition(space)
    wsb = _lib.kr_evaluate_and_filter_workspace(ctypes.byref(sp))
    if wsb == 0:
        raise KrError("kr_evaluate_and_filter_workspace", KR_EUNSUPPORTED)
    while True:
        c = int(cap) if cap is not None else min(space.n_parts * C, 4096 * space.n_parts)
        off = torch.empty(space.n_parts + 1, dtype=torch.int64, device="cuda")
        idx = torch.empty(max(c, 1), dtype=torch.int32, device="cuda")
        oT = torch.empty(max(c, 1), dtype=torch.float64, device="cuda")
        oE = torch.empty(max(c, 1), dtype=torch.float64, device="cuda")
        ws = _workspace(wsb)
        status = _status_word(sync if validate is None else validate)
        _check("kr_evaluate_and_filter",
               _lib.kr_evaluate_and_filter(ctypes.byref(sp), _ptr(t), _ptr(pw), _ptr(tc), _ptr(pc),
                                           c, _ptr(off), _ptr(idx), _ptr(oT), _ptr(oE),
                                           _ptr(status), _ptr(ws), wsb, _stream()))
        _check_status("kr_evaluate_and_filter", status)
        fr, ok = _finish_frontier(off, idx, oT, oE, c, sync)
        if fr is not None:
            return fr
        cap = ok


@dataclasses.dataclass
class Composed:
    F: torch.Tensor          # float64 [B]
    bp: torch.Tensor         # int32 [P][B]
    bp_off: torch.Tensor     # int32 [P][B]: offset of each chosen point
    pt_bin: torch.Tensor     # int32 [n_points]
    info: torch.Tensor       # float64 [2]: delta, tmin_sum
    L: torch.Tensor          # int32 [1]
    stair_bin: torch.Tensor  # int32 [B]
    stair_Tlo: torch.Tensor  # float64 [B]
    stair_E: torch.Tensor    # float64 [B]
    n_stair: torch.Tensor    # int32 [1]
    status: torch.Tensor     # int32 [1]

    def staircase(self):
        n = int(self.n_stair.item())
        return self.stair_bin[:n], self.stair_Tlo[:n], self.stair_E[:n]


def compose_frontiers(off, T, E, n_bins: int, delta: float = 0.0, out: Optional[Composed] = None
                      ) -> Composed:
    """Min-plus composition of partition frontiers [off[k], off[k+1]) of (T, E)."""
    off = _dev(off, torch.int64, "off")
    T = _dev(T, torch.float64, "T").reshape(-1)
    E = _dev(E, torch.float64, "E").reshape(-1)
    P = off.numel() - 1
    B = int(n_bins)
    if out is None:
        f64 = dict(dtype=torch.float64, device="cuda")
        i32 = dict(dtype=torch.int32, device="cuda")
        out = Composed(torch.empty(B, **f64), torch.empty((P, B), **i32),
                       torch.empty((P, B), **i32),
                       torch.empty(max(T.numel(), 1), **i32), torch.empty(2, **f64),
                       torch.empty(1, **i32), torch.empty(B, **i32), torch.empty(B, **f64),
                       torch.empty(B, **f64), torch.empty(1, **i32), torch.empty(1, **i32))
    wsb = _lib.kr_compose_frontiers_workspace(P, B)
    ws = _workspace(wsb)
    _check("kr_compose_frontiers",
           _lib.kr_compose_frontiers(P, _ptr(off), _ptr(T), _ptr(E), B, float(delta), _ptr(out.F),
                                     _ptr(out.bp), _ptr(out.bp_off), _ptr(out.pt_bin),
                                     _ptr(out.info), _ptr(out.L),
                                     _ptr(out.stair_bin), _ptr(out.stair_Tlo), _ptr(out.stair_E),
                                     _ptr(out.n_stair), _ptr(out.status), _ptr(ws), wsb,
                                     _stream()))
    return out


def extract_schedule(comp: Composed, off, T, E, bins, cand_idx=None, use_offsets: bool = True):
    """Per-partition choice behind each query bin (use_offsets=False walks without the
    recorded offsets, looking each point's offset up instead).
    Returns (choice [n_q][P], choice_cand [n_q][P] or None, T [n_q], E [n_q], ok [n_q])."""
    off = _dev(off, torch.int64, "off")
    T = _dev(T, torch.float64, "T").reshape(-1)
    E = _dev(E, torch.float64, "E").reshape(-1)
    bins = _dev(bins, torch.int32, "bins").reshape(-1)
    P, B = comp.bp.shape
    nq = bins.numel()
    choice = torch.empty((nq, P), dtype=torch.int32, device="cuda")
    cc = None
    if cand_idx is not None:
        cand_idx = _dev(cand_idx, torch.int32, "cand_idx")
        cc = torch.empty((nq, P), dtype=torch.int32, device="cuda")
    Ts = torch.empty(nq, dtype=torch.float64, device="cuda")
    Es = torch.empty(nq, dtype=torch.float64, device="cuda")
    ok = torch.empty(nq, dtype=torch.int32, device="cuda")
    _check("kr_extract_schedule",
           _lib.kr_extract_schedule(P, B, _ptr(comp.bp),
                                    _ptr(comp.bp_off) if use_offsets else None,
                                    _ptr(comp.pt_bin), _ptr(off), _ptr(T),
                                    _ptr(E), _ptr(bins), nq, _ptr(cand_idx), _ptr(choice), _ptr(cc),
                                    _ptr(Ts), _ptr(Es), _ptr(ok), _stream()))
    return choice, cc, Ts, Es, ok


class Microbatch:
    """Microbatch frontier: T, E [n], f int32 [n] frequency index, choice int32 [n][K]."""

    def __init__(self, T, E, f, choice):
        self.T, self.E, self.f, self.choice = T, E, f, choice


@dataclasses.dataclass
class MicrobatchBuffers:
    """Caller-kept buffers of a microbatch call: outputs of capacity `cap`, the device
    point count n [1] and status [1], and the device copy of seg_off.  A call given them
    allocates nothing and copies nothing from the host; with check=False it also reads
    nothing back, so it only enqueues work on the stream.  Results of a checked call are
    views into the buffers, valid until the buffers are used again."""
    T: torch.Tensor
    E: torch.Tensor
    f: torch.Tensor
    choice: torch.Tensor
    n: torch.Tensor
    status: torch.Tensor
    seg: torch.Tensor
    seg_host: np.ndarray


def microbatch_buffers(seg_off, n_types: int, cap: int) -> MicrobatchBuffers:
    """Buffers for microbatch_frontier / microbatch_enumerate calls on segments seg_off
    (host) with output capacity cap."""
    seg_host = np.ascontiguousarray(np.asarray(seg_off, dtype=np.int64))
    c = max(int(cap), 1)
    return MicrobatchBuffers(
        torch.empty(c, dtype=torch.float64, device="cuda"),
        torch.empty(c, dtype=torch.float64, device="cuda"),
        torch.empty(c, dtype=torch.int32, device="cuda"),
        torch.empty((c, n_types), dtype=torch.int32, device="cuda"),
        torch.empty(1, dtype=torch.int64, device="cuda"),
        torch.empty(1, dtype=torch.int32, device="cuda"),
        torch.from_numpy(seg_host.copy()).cuda(), seg_host)


def _mb_buffers(out, seg_host, n_types, c):
    if out is None:
        return microbatch_buffers(seg_host, n_types, c)
    if (out.T.numel() < max(c, 1) or out.choice.shape[1] != n_types
            or not np.array_equal(out.seg_host, seg_host)):
        raise ValueError("buffers were made for another shape, capacity or seg_off")
    return out


def microbatch_frontier(seg_off, T, E, n_types: int, n_freq: int, seq, comp_T=None, comp_E=None,
                        n_bins: int = 4096, cap: Optional[int] = None, check: bool = True,
                        out: Optional[MicrobatchBuffers] = None):
    """Microbatch frontier of Algorithm 2 (one frequency per microbatch, one configuration
    per partition type).  seg_off [K*F+1] (segment t*F+f = type t's points at frequency f),
    seq: host list of partition types in execution order, comp_T/comp_E [n_comp][F].
    With check=False the buffers are returned untrimmed (out.n holds the count)."""
    seg_host = np.asarray(seg_off.cpu() if isinstance(seg_off, torch.Tensor) else seg_off,
                          dtype=np.int64)
    if len(seg_host) != n_types * n_freq + 1:
        raise ValueError("seg_off must have n_types * n_freq + 1 entries")
    n_points = int(seg_host[-1])
    T = _dev(T, torch.float64, "T").reshape(-1)
    E = _dev(E, torch.float64, "E").reshape(-1)
    seq_h = np.ascontiguousarray(np.asarray(seq, dtype=np.int32))
    if comp_T is None:
        n_comp, cT, cE = 0, None, None
    else:
        cT = _dev(comp_T, torch.float64, "comp_T").reshape(-1, n_freq)
        cE = _dev(comp_E, torch.float64, "comp_E").reshape(-1, n_freq)
        n_comp = cT.shape[0]
    c = int(cap) if cap is not None else n_freq * n_bins
    out = _mb_buffers(out, seg_host, n_types, c)
    wsb = _lib.kr_microbatch_frontier_workspace(n_types, n_freq, n_points, len(seq_h), n_bins)
    if wsb == 0:
        raise ValueError("unsupported microbatch shape")
    ws = _workspace(wsb)
    _check("kr_microbatch_frontier",
           _lib.kr_microbatch_frontier(n_types, n_freq, _ptr(out.seg), _ptr(T), _ptr(E), n_points,
                                       len(seq_h), seq_h.ctypes.data_as(ctypes.c_void_p), n_comp,
                                       _ptr(cT), _ptr(cE), n_bins, c, _ptr(out.T), _ptr(out.E),
                                       _ptr(out.f), _ptr(out.choice), _ptr(out.n), _ptr(ws), wsb,
                                       _stream()))
    if not check:
        return out
    k = min(int(out.n.item()), c)
    return Microbatch(out.T[:k], out.E[:k], out.f[:k], out.choice[:k])


def microbatch_enumerate(seg_off, T, E, n_types: int, n_freq: int, seq, comp_T=None,
                         comp_E=None, cap: Optional[int] = None, check: bool = True,
                         out: Optional[MicrobatchBuffers] = None):
    """Microbatch frontier by enumerating every configuration (Algorithm 2 as written).
    With check=False the buffers are returned untrimmed and the status is not read
    (out.n holds the count, out.status the status)."""
    seg_host = np.asarray(seg_off.cpu() if isinstance(seg_off, torch.Tensor) else seg_off,
                          dtype=np.int64)
    if len(seg_host) != n_types * n_freq + 1:
        raise ValueError("seg_off must have n_types * n_freq + 1 entries")
    seq_h = np.ascontiguousarray(np.asarray(seq, dtype=np.int32))
    sizes = np.diff(seg_host).reshape(n_types, n_freq)
    used = sorted(set(seq_h.tolist()))
    n_configs = max(int(np.sum(np.prod(sizes[used], axis=0))), 1)
    T = _dev(T, torch.float64, "T").reshape(-1)
    E = _dev(E, torch.float64, "E").reshape(-1)
    if comp_T is None:
        n_comp, cT, cE = 0, None, None
    else:
        cT = _dev(comp_T, torch.float64, "comp_T").reshape(-1, n_freq)
        cE = _dev(comp_E, torch.float64, "comp_E").reshape(-1, n_freq)
        n_comp = cT.shape[0]
    c = int(cap) if cap is not None else n_configs
    out = _mb_buffers(out, seg_host, n_types, c)
    wsb = _lib.kr_microbatch_enumerate_workspace(n_types, n_freq, n_configs)
    if wsb == 0:
        raise ValueError("unsupported microbatch shape")
    ws = _workspace(wsb)
    _check("kr_microbatch_enumerate",
           _lib.kr_microbatch_enumerate(n_types, n_freq, _ptr(out.seg), _ptr(T), _ptr(E),
                                        len(seq_h), seq_h.ctypes.data_as(ctypes.c_void_p),
                                        n_comp, _ptr(cT), _ptr(cE), n_configs, c, _ptr(out.T),
                                        _ptr(out.E), _ptr(out.f), _ptr(out.choice), _ptr(out.n),
                                        _ptr(out.status), _ptr(ws), wsb, _stream()))
    if not check:
        return out
    st = int(out.status.item())
    if st != KR_OK:
        raise KrError("kr_microbatch_enumerate", st)
    k = min(int(out.n.item()), c)
    return Microbatch(out.T[:k], out.E[:k], out.f[:k], out.choice[:k])


def decode_candidates(space, idx):
    """Candidate index -> (f [n], pos [n][M], sm [n][M]) on the device."""
    sp = _space(space)
    idx = _dev(idx, torch.int32, "idx").reshape(-1)
    n = idx.numel()
    f = torch.empty(n, dtype=torch.int32, device="cuda")
    pos = torch.empty((n, space.n_comm), dtype=torch.int32, device="cuda")
    sm = torch.empty((n, space.n_comm), dtype=torch.int32, device="cuda")
    _check("kr_decode_candidates",
           _lib.kr_decode_candidates(ctypes.byref(sp), _ptr(idx), n, _ptr(f), _ptr(pos), _ptr(sm),
                                     _stream()))
    return f, pos, sm


@dataclasses.dataclass
class HviScores:
    hvi: torch.Tensor     # [3][n_cand]: total, dynamic, static energy
    hv: torch.Tensor      # [n_seg][3]
    ref: torch.Tensor     # [n_seg][4]: rT, rE per variant
    status: torch.Tensor  # [1]


def _offsets(off, name: str) -> torch.Tensor:
    return _dev(np.asarray(off.cpu() if isinstance(off, torch.Tensor) else off, dtype=np.int64),
                torch.int64, name).reshape(-1)


def hvi_scores(cand_off, T_hat, E_hat, obs_off, T_obs, E_obs, p_static: float,
               check: bool = True, out: Optional[HviScores] = None) -> HviScores:
    """Exploitation scores of Algorithm 1 (kr_hvi_scores).  With check=False the device
    status is left for the caller (no synchronisation)."""
    co = cand_off if isinstance(cand_off, torch.Tensor) and cand_off.is_cuda else \
        _offsets(cand_off, "cand_off")
    oo = obs_off if isinstance(obs_off, torch.Tensor) and obs_off.is_cuda else \
        _offsets(obs_off, "obs_off")
    n_seg = co.numel() - 1
    T_hat = _dev(T_hat, torch.float64, "T_hat").reshape(-1)
    E_hat = _dev(E_hat, torch.float64, "E_hat").reshape(-1)
    T_obs = _dev(T_obs, torch.float64, "T_obs").reshape(-1)
    E_obs = _dev(E_obs, torch.float64, "E_obs").reshape(-1)
    n, no = T_hat.numel(), T_obs.numel()
    if out is None:
        out = HviScores(torch.empty((3, n), dtype=torch.float64, device="cuda"),
                        torch.empty((n_seg, 3), dtype=torch.float64, device="cuda"),
                        torch.empty((n_seg, 4), dtype=torch.float64, device="cuda"),
                        torch.empty(1, dtype=torch.int32, device="cuda"))
    wsb = _lib.kr_hvi_scores_workspace(n_seg, no)
    if wsb == 0:
        raise ValueError("hvi_scores needs at least one partition and one measured point")
    ws = _workspace(wsb)
    _check("kr_hvi_scores",
           _lib.kr_hvi_scores(n_seg, n, _ptr(co), _ptr(T_hat), _ptr(E_hat), no, _ptr(oo),
                              _ptr(T_obs), _ptr(E_obs), float(p_static), _ptr(out.hvi),
                              _ptr(out.hv), _ptr(out.ref), _ptr(out.status), _ptr(ws), wsb,
                              _stream()))
    if check and int(out.status.item()) != KR_OK:
        raise KrError("kr_hvi_scores", int(out.status.item()))
    return out


def uncertainty(T_m, E_m, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Exploration score of Algorithm 1 (kr_uncertainty); T_m, E_m [M][n]."""
    T_m = _dev(T_m, torch.float64, "T_m")
    E_m = _dev(E_m, torch.float64, "E_m")
    if T_m.dim() != 2 or T_m.shape != E_m.shape:
        raise ValueError("T_m and E_m must both be [M][n]")
    M, n = T_m.shape
    if out is None:
        out = torch.empty(n, dtype=torch.float64, device="cuda")
    _check("kr_uncertainty",
           _lib.kr_uncertainty(M, n, _ptr(T_m), _ptr(E_m), _ptr(out), _stream()))
    return out


@dataclasses.dataclass
class Batch:
    sel: torch.Tensor     # [n_seg][k] int64 local indices
    count: torch.Tensor   # [n_seg] int32
    status: torch.Tensor  # [1]

    def lists(self):
        c = self.count.cpu().numpy()
        s = self.sel.cpu().numpy()
        return [s[g, :c[g]].copy() for g in range(len(c))]


def select_batch(cand_off, score, unc, obs_off, obs_idx, k1: int, k2: int, k3: int, k: int,
                 check: bool = True, out: Optional[Batch] = None) -> Batch:
    """Multi-pass candidate selection of Algorithm 1 (kr_select_batch)."""
    co = cand_off if isinstance(cand_off, torch.Tensor) and cand_off.is_cuda else \
        _offsets(cand_off, "cand_off")
    oo = obs_off if isinstance(obs_off, torch.Tensor) and obs_off.is_cuda else \
        _offsets(obs_off, "obs_off")
    oi = _dev(np.asarray(obs_idx, dtype=np.int64) if not isinstance(obs_idx, torch.Tensor)
              else obs_idx, torch.int64, "obs_idx").reshape(-1)
    if oi.numel() == 0:
        oi = torch.zeros(1, dtype=torch.int64, device="cuda")
    n_seg = co.numel() - 1
    score = _dev(score, torch.float64, "score").reshape(3, -1)
    n = score.shape[1]
    u = None if unc is None else _dev(unc, torch.float64, "unc").reshape(-1)
    if out is None:
        out = Batch(torch.full((n_seg, max(k, 1)), -1, dtype=torch.int64, device="cuda"),
                    torch.empty(n_seg, dtype=torch.int32, device="cuda"),
                    torch.empty(1, dtype=torch.int32, device="cuda"))
    wsb = _lib.kr_select_batch_workspace(n_seg, n)
    if wsb == 0:
        raise ValueError("select_batch needs at least one partition")
    ws = _workspace(wsb)
    _check("kr_select_batch",
           _lib.kr_select_batch(n_seg, n, _ptr(co), _ptr(score), _ptr(u), _ptr(oo), _ptr(oi),
                                k1, k2, k3, k, _ptr(out.sel), _ptr(out.count), _ptr(out.status),
                                _ptr(ws), wsb, _stream()))
    if check and int(out.status.item()) != KR_OK:
        raise KrError("kr_select_batch", int(out.status.item()))
    return out


def hv_converged(hv_history, R: int = 2, eps: float = 1e-3) -> bool:
    """Stopping rule of Algorithm 1 (kr_hv_converged, host)."""
    h = np.ascontiguousarray(np.asarray(hv_history, dtype=np.float64))
    return bool(_lib.kr_hv_converged(h.shape[0], h.ctypes.data_as(ctypes.c_void_p), R, float(eps)))


def compare_frontiers(TA, EA, TB, EB, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Frontier metrics of B against baseline A (kr_compare_frontiers): float64[10] on the
    device (leftmost time and energy reduction %, iso-time energy reduction %, iso-energy
    time reduction %, d, E_A(d), E_B(d), b, T_A(b), T_B(b))."""
    TA = _dev(TA, torch.float64, "TA").reshape(-1)
    EA = _dev(EA, torch.float64, "EA").reshape(-1)
    TB = _dev(TB, torch.float64, "TB").reshape(-1)
    EB = _dev(EB, torch.float64, "EB").reshape(-1)
    if out is None:
        out = torch.empty(10, dtype=torch.float64, device="cuda")
    wsb = _lib.kr_compare_frontiers_workspace()
    ws = _workspace(wsb)
    _check("kr_compare_frontiers",
           _lib.kr_compare_frontiers(TA.numel(), _ptr(TA), _ptr(EA), TB.numel(), _ptr(TB),
                                     _ptr(EB), _ptr(out), _ptr(ws), wsb, _stream()))
    return out


@dataclasses.dataclass
class LaunchFrontier:
    T: torch.Tensor       # [n_inst][out_cap]
    E: torch.Tensor
    sched: Optional[torch.Tensor]  # [n_inst][out_cap][I + J] decision codes, -1 padded
    n: torch.Tensor       # [n_inst] frontier sizes (-1: an on-chip limit was hit)
    status: torch.Tensor  # [1]


def launch_timing_frontier(kind1, kind2, ops, p_static: float, kmax: int, out_cap: int = 64,
                           sched: bool = True, check: bool = True,
                           out: Optional[LaunchFrontier] = None) -> LaunchFrontier:
    """Launch-timing frontier of two operation sequences (kr_launch_timing_frontier).
    kind1 [I], kind2 [J]: 0 computation, 1 communication; ops [n_inst][I + J][4]."""
    kind = np.ascontiguousarray(np.concatenate([np.asarray(kind1), np.asarray(kind2)]),
                                dtype=np.int32)
    I, J = len(kind1), len(kind2)
    ops = _dev(ops, torch.float64, "ops").reshape(-1, I + J, 4)
    n = ops.shape[0]
    if out is None:
        out = LaunchFrontier(
            torch.empty((n, out_cap), dtype=torch.float64, device="cuda"),
            torch.empty((n, out_cap), dtype=torch.float64, device="cuda"),
            torch.empty((n, out_cap, I + J), dtype=torch.int32, device="cuda") if sched else None,
            torch.empty(max(n, 1), dtype=torch.int32, device="cuda"),
            torch.empty(1, dtype=torch.int32, device="cuda"))
    wsb = _lib.kr_launch_timing_frontier_workspace(n)
    ws = _workspace(wsb)
    _check("kr_launch_timing_frontier",
           _lib.kr_launch_timing_frontier(n, I, J, kind.ctypes.data_as(ctypes.c_void_p),
                                          _ptr(ops), float(p_static), kmax, out_cap,
                                          _ptr(out.T), _ptr(out.E), _ptr(out.sched),
                                          _ptr(out.n), _ptr(out.status), _ptr(ws), wsb,
                                          _stream()))
    if check and int(out.status.item()) != KR_OK:
        raise KrError("kr_launch_timing_frontier", int(out.status.item()))
    return out
