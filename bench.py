"""Benchmark of the schedule-search hot path on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
  1. fused evaluation + frontier filter of the eval-stress batch: 1,024 partitions x
     135,168 candidates (32 compute kernels, 33 launch positions, 32 SM choices, 128
     frequencies) = 138,412,032 candidates;
  2. composition of the compose-stress batch (512 precomputed frontiers of 256-2,048
     points) over 65,536 time bins, staircase, and extraction of the leftmost
     (max-throughput) schedule.
Inputs are device-resident before the timed region.  `value` is candidates evaluated
and Pareto-filtered per second (step 1's candidates over step 1's time, HIP events on
the library's stream); `frontier_cells_per_s` is the composition's DP cells (sum over
partitions of the reachable bins) over step 2's time.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--skip-cpu]
       python bench.py --part eval|compose|eval2|mbo|dp   (one leg only, no bench line: for
                                                           profilers)
       python bench.py --copy-calibration   (plain 1 GiB device copy, for counters)
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP64_VECTOR_TFLOPS = 78.6
COUNTERS = os.path.join(ROOT, "profiles", "eval_filter_counters_eval_stress.txt")
KERNEL_SOURCES = ["eval_wave.hip", "kr_filter.h", "kr_device.h", "kr_wave.h"]
METRIC = "schedule candidates evaluated+filtered/sec and frontier cells/sec on 1 MI355X"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _between(text: str, start: str, end: str) -> str:
    i = text.index(start)
    return text[i:text.index(end, i) + len(end)]


def kernel_source_hash() -> str:
    """sha256 (first 16 hex) of what the fused eval kernel is built from: its source files,
    its argument struct, and the host code that plans its launch."""
    csrc = os.path.join(ROOT, "paper_2601_17654_amd", "csrc")
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(csrc, "kr_launch.h")) as fh:
        h.update(_between(fh.read(), "struct EvalArgs {", "\n};\n").encode())
    with open(os.path.join(csrc, "api.hip")) as fh:
        api = fh.read()
    h.update(_between(api, "bool wave_plan(EvalArgs *a)", "\n}\n").encode())
    h.update(_between(api, "bool eval_plan(const kr_space *s, bool fused, EvalArgs *a)",
                      "\n}\n").encode())
    return h.hexdigest()[:16]


def read_summary(path: str, source_hash: str):
    """key=value pairs of a committed counter summary, or None when it is missing or
    was taken on sources that hash differently from today's."""
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("#", 1)[0].strip().split("=", 1)
            vals[k.strip()] = v.strip()
    return vals if vals.get("source_hash") == source_hash else None


def minplus_source_hash() -> str:
    """sha256 (first 16 hex) of what the composition kernels are built and launched from."""
    csrc = os.path.join(ROOT, "paper_2601_17654_amd", "csrc")
    h = hashlib.sha256()
    for f in ("compose.hip", "kr_device.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(csrc, "kr_launch.h")) as fh:
        lh = fh.read()
    h.update(_between(lh, "struct ComposeArgs {", "\n};\n").encode())
    h.update(_between(lh, "struct ComposeWs {", "\n};\n").encode())
    with open(os.path.join(csrc, "api.hip")) as fh:
        h.update(_between(fh.read(), "kr_status kr_compose_frontiers(", "\n}\n").encode())
    return h.hexdigest()[:16]


def eval2_source_hash() -> str:
    """sha256 (first 16 hex) of what the one-wave-per-slab two-comm evaluation kernel is
    built from and planned by."""
    csrc = os.path.join(ROOT, "paper_2601_17654_amd", "csrc")
    h = hashlib.sha256()
    for f in ("eval_pair.hip", "kr_wave.h", "kr_filter.h", "kr_device.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(csrc, "kr_launch.h")) as fh:
        h.update(_between(fh.read(), "struct EvalArgs {", "\n};\n").encode())
    with open(os.path.join(csrc, "api.hip")) as fh:
        api = fh.read()
    h.update(_between(api, "bool pair_plan(EvalArgs *a)", "\n}\n").encode())
    h.update(_between(api, "bool eval_plan(const kr_space *s, bool fused, EvalArgs *a)",
                      "\n}\n").encode())
    return h.hexdigest()[:16]


MINPLUS_COUNTERS = os.path.join(ROOT, "profiles", "minplus_counters_compose_stress.txt")
EVAL2_COUNTERS = os.path.join(ROOT, "profiles", "eval_two_comm_counters.txt")


MBO_COUNTERS = os.path.join(ROOT, "profiles", "mbo_counters_eval_stress.txt")
MBO_KERNELS = ("hvi_score_kernel", "unc_kernel", "sel_tile_kernel")


def mbo_source_hash() -> str:
    """sha256 (first 16 hex) of what the score, uncertainty and selection kernels are
    built and launched from."""
    csrc = os.path.join(ROOT, "paper_2601_17654_amd", "csrc")
    h = hashlib.sha256()
    for f in ("mbo.hip", "kr_device.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(csrc, "kr_launch.h")) as fh:
        h.update(_between(fh.read(), "// mbo.hip", "launch_select(const SelArgs &a, "
                          "hipEvent_t *ev, hipStream_t st);").encode())
    with open(os.path.join(csrc, "api.hip")) as fh:
        api = fh.read()
        h.update(_between(api, "size_t kr_hvi_scores_workspace",
                          "return launch_select(a, g_phase_ev[KR_PHASE_SELECT]").encode())
    return h.hexdigest()[:16]


def read_mbo_traffic():
    """HBM bytes per launch of each score/selection kernel from the committed counter
    summary, if it was taken on the current sources; else {}."""
    if not os.path.exists(MBO_COUNTERS):
        return {}, "no counter summary"
    vals = {}
    for line in open(MBO_COUNTERS):
        if "=" in line and not line.startswith("#"):
            k, v = line.strip().split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_hash") != mbo_source_hash():
        return {}, "kernels changed since counters were taken"
    return {k: float(vals[k + ".traffic_bytes_per_launch"]) for k in MBO_KERNELS
            if k + ".traffic_bytes_per_launch" in vals}, "counters"


VALU_COUNTERS = os.path.join(ROOT, "profiles", "eval_valu_counters_eval_stress.txt")
VALU_ISSUE_PEAK = 1024 * 2.4e9 / 4  # wave instructions/s: 4 cycles per wave64 instruction


def read_valu():
    """VALU wave instructions and fp64 flops per launch of the fused eval kernel from the
    committed counter summary, if taken on the current sources; else None."""
    if not os.path.exists(VALU_COUNTERS):
        return None
    vals = {}
    for line in open(VALU_COUNTERS):
        if "=" in line and not line.startswith("#"):
            k, v = line.strip().split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_hash") != kernel_source_hash():
        return None
    return float(vals["valu_wave_instructions_per_launch"]), float(vals["fp64_flops_per_launch"])


def read_traffic(n_launch_bytes_alg: float):
    """HBM bytes per launch of the fused kernel from the committed counter summary, if
    it was taken on the current kernel source; else None."""
    if not os.path.exists(COUNTERS):
        return None, "no counter summary"
    vals = {}
    for line in open(COUNTERS):
        if "=" in line and not line.startswith("#"):
            k, v = line.strip().split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_hash") != kernel_source_hash():
        return None, "kernel changed since counters were taken"
    try:
        return float(vals["traffic_bytes_per_launch"]), "counters"
    except (KeyError, ValueError):
        return None, "incomplete counter summary"


def copy_calibration():
    import torch

    n = 1 << 27  # 1 GiB of fp64
    x = torch.ones(n, dtype=torch.float64, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 8, "copy_bytes_written": n * 8, "launches": 3}))


def mk_events(n):
    import torch

    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
    for e in evs:
        e.record()  # creates the HIP event behind the handle
    return evs


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--skip-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--part", choices=["all", "eval", "compose", "eval2", "mbo", "dp"],
                    default="all",
                    help="profiling aid: run only one half of the step (prints no bench line)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        log("bench.py runs on exactly one GPU: the schedule search here is a single-GPU "
            "build (no collectives); --gpus %d is not supported." % args.gpus)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        copy_calibration()
        return

    from paper_2601_17654_amd import binding as kr
    from paper_2601_17654_amd import inputs as I

    torch.cuda.set_device(0)
    t0 = time.time()
    w = I.config_workload(3)
    off4, T4, E4 = I.compose_frontiers()
    B = I.COMPOSE_SPACE["bins"]
    log("inputs generated in %.1f s" % (time.time() - t0))
    sp = w.space
    d = [torch.from_numpy(getattr(w, k)).cuda() for k in ("t", "pw", "tc", "pc")]
    off4_d, T4_d, E4_d = (torch.from_numpy(x).cuda() for x in (off4, T4, E4))
    table_bytes = sum(x.numel() * 8 for x in d)
    n_cand = sp.n_parts * sp.n_cand

    # exact output capacity from one untimed pass
    fr = kr.evaluate_and_filter(sp, *d)
    cap = int(fr.off[-1].item())
    comp = kr.compose_frontiers(off4_d, T4_d, E4_d, B)
    torch.cuda.synchronize()

    if args.part == "eval2":
        res, _ = bench_eval2(kr, I, torch, args, mk_events)
        log("eval2: " + json.dumps(res))
        return
    if args.part == "dp":
        res, _ = bench_dp(kr, I, torch, args, mk_events)
        log("dp: " + json.dumps(res))
        return
    if args.part == "mbo":
        res, _ = bench_mbo(kr, I, torch, sp, d, args, mk_events)
        log("mbo: " + json.dumps(res))
        return
    if args.part != "all":
        for _ in range(args.warmup + args.steps):
            if args.part == "eval":
                kr.evaluate_and_filter(sp, *d, cap=cap, sync=False)
            else:
                kr.compose_frontiers(off4_d, T4_d, E4_d, B, out=comp)
                kr.extract_schedule(comp, off4_d, T4_d, E4_d, comp.stair_bin[:1])
        torch.cuda.synchronize()
        log("ran %d passes of the %s half" % (args.warmup + args.steps, args.part))
        return

    def step(ev, phase_ev):
        ev[0].record()
        kr.set_phase_events(kr.PHASE_EVAL_TILE, *phase_ev[0])
        kr.set_phase_events(kr.PHASE_MINPLUS, *phase_ev[1])
        f = kr.evaluate_and_filter(sp, *d, cap=cap, sync=False)
        ev[1].record()
        kr.compose_frontiers(off4_d, T4_d, E4_d, B, out=comp)
        ev[2].record()
        kr.extract_schedule(comp, off4_d, T4_d, E4_d, comp.stair_bin[:1])
        ev[3].record()
        return f

    mk = mk_events

    for _ in range(args.warmup):
        step(mk(4), [mk(2), mk(2)])
    torch.cuda.synchronize()
    evs = [mk(4) for _ in range(args.steps)]
    pev = [[mk(2), mk(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for k in range(args.steps):
        fr = step(evs[k], pev[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    kr.set_phase_events(kr.PHASE_EVAL_TILE)
    kr.set_phase_events(kr.PHASE_MINPLUS)

    # per-part times: medians over the timed steps (HIP events on the library's stream)
    ef_ms = float(np.median([e[0].elapsed_time(e[1]) for e in evs]))
    co_ms = float(np.median([e[1].elapsed_time(e[2]) for e in evs]))
    ex_ms = float(np.median([e[2].elapsed_time(e[3]) for e in evs]))
    kern_ms = float(np.median([p[0][0].elapsed_time(p[0][1]) for p in pev]))
    mp_ms = float(np.median([p[1][0].elapsed_time(p[1][1]) for p in pev]))
    ms_per_step = wall * 1e3 / args.steps
    assert int(comp.status.item()) == 0 and int(fr.off[-1].item()) == cap

    # composition cells: sum over partitions of the reachable bins after that partition
    pt = comp.pt_bin.cpu().numpy()[: len(T4)]
    Mk = np.maximum.reduceat(pt, off4[:-1]).astype(np.int64)
    cells = int(np.sum(1 + np.cumsum(Mk)))

    achieved = table_bytes / (kern_ms * 1e-3) / 1e9
    traffic, tsrc = read_traffic(table_bytes)
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
            "kernel": "eval_filter_wave_kernel (fused evaluation + frontier, one wave per slab)",
            "kernel_ms": round(kern_ms, 4), "algorithmic_bytes": table_bytes,
            "traffic_GBps": None if traffic is None else round(traffic / (kern_ms * 1e-3) / 1e9, 1),
            "traffic_source": tsrc}

    # composition: the min-plus step for partition k pairs each of the L_{k-1} bins
    # reachable after the partitions before it with each occupied bin of its own
    # frontier; VALU instruction counts come from the committed counter summary
    pairs = 0
    reach = 1 + int(Mk[0])
    for k in range(1, len(Mk)):
        occ = len(np.unique(pt[off4[k]:off4[k + 1]]))
        pairs += min(reach, B) * occ
        reach += int(Mk[k])
    mpc = read_summary(MINPLUS_COUNTERS, minplus_source_hash())
    croof = {"bound": "alu", "kernel": "minplus_wavefront_kernel (min-plus steps, tiles of "
             "bins taken by ticket)", "kernel_ms": round(mp_ms, 4), "pairs": pairs,
             "pairs_per_s": pairs / (mp_ms * 1e-3), "peak": VALU_ISSUE_PEAK / 1e9,
             "unit": "G VALU wave-instructions/s", "achieved": None, "frac": None,
             "source": "kernel changed since counters were taken" if mpc is None else
             "profiles/minplus_counters_compose_stress.txt"}
    if mpc is not None:
        vi = float(mpc["valu_wave_instructions_per_launch"]) / (mp_ms * 1e-3)
        croof.update(achieved=round(vi / 1e9, 2), frac=round(vi / VALU_ISSUE_PEAK, 4),
                     valu_busy=float(mpc["valu_busy"]),
                     valu_per_pair_lane=round(64 * float(mpc["valu_wave_instructions_per_launch"])
                                              / pairs, 2))

    valu = read_valu()
    if valu is not None:
        vi = valu[0] / (kern_ms * 1e-3)
        roof["alu"] = {"bound": "alu", "achieved": round(vi / 1e9, 2), "peak": VALU_ISSUE_PEAK / 1e9,
                       "unit": "G VALU wave-instructions/s", "frac": round(vi / VALU_ISSUE_PEAK, 4),
                       "fp64_TFLOPs": round(valu[1] / (kern_ms * 1e-3) / 1e12, 2),
                       "fp64_peak_TFLOPs": FP64_VECTOR_TFLOPS,
                       "source": "profiles/eval_valu_counters_eval_stress.txt"}

    out = {
        "metric": METRIC,
        "value": n_cand / (ef_ms * 1e-3),
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {
            "workload": "eval-stress (1024 partitions x 135,168 candidates: 32 kernels, "
                        "33 positions, 32 SM choices, 128 frequencies) + compose-stress "
                        "(512 frontiers of 256-2048 points, 65,536 bins)",
            "candidates": n_cand, "frontier_points": cap, "compose_bins": B,
            "compose_partitions": len(off4) - 1, "parallelism": "single GPU"},
        "frontier_cells_per_s": cells / (co_ms * 1e-3),
        "frontier_cells": cells,
        "eval_filter_ms": round(ef_ms, 4),
        "compose_ms": round(co_ms, 4),
        "minplus_ms": round(mp_ms, 4),
        "extract_ms": round(ex_ms, 4),
        "roofline": roof,
        "compose_roofline": croof,
    }

    # Microbatch frontier (Algorithm 2 with one frequency per microbatch and one
    # configuration per partition type): four llama-layer partition types, a 16-layer
    # microbatch of all four, two non-partition components, every frequency.  Timed on
    # its own.
    mb_w = I.config_workload(1, parts=range(0, 4))
    msp = mb_w.space
    mK, mF, mCf = msp.n_parts, msp.n_freq, msp.cand_per_freq
    md = [torch.from_numpy(getattr(mb_w, k)).cuda() for k in ("t", "pw", "tc", "pc")]
    mT, mE = kr.evaluate_partition(msp, *md)
    mfr = kr.pareto_filter(mT.reshape(-1), mE.reshape(-1), np.arange(mK * mF + 1) * mCf)
    mseg = mfr.off.cpu().numpy()
    mseq = [0, 1, 2, 3] * 16
    mcT, mcE = I.microbatch_components(1, 2, msp.freqs_mhz)
    mcT_d, mcE_d = torch.from_numpy(mcT).cuda(), torch.from_numpy(mcE).cuda()
    MB_BINS = 4096
    sizes = np.diff(mseg).reshape(mK, mF)
    n_configs = int(np.sum(np.prod(sizes, axis=0)))
    # Timed calls get device-resident buffers and read nothing back (check=False), so the
    # events bracket only the enqueued work; the checked call after them gives the
    # results that are compared with the oracle.
    mbuf = kr.microbatch_buffers(mseg, mK, mF * MB_BINS)
    xbuf = kr.microbatch_buffers(mseg, mK, n_configs)
    kr.microbatch_frontier(mseg, mfr.T, mfr.E, mK, mF, mseq, mcT_d, mcE_d, n_bins=MB_BINS,
                           check=False, out=mbuf)
    torch.cuda.synchronize()
    mev = mk(2 * args.steps)
    for k in range(args.steps):
        mev[2 * k].record()
        kr.microbatch_frontier(mseg, mfr.T, mfr.E, mK, mF, mseq, mcT_d, mcE_d, n_bins=MB_BINS,
                               check=False, out=mbuf)
        mev[2 * k + 1].record()
    torch.cuda.synchronize()
    mb_ms = float(np.median([mev[2 * k].elapsed_time(mev[2 * k + 1]) for k in range(args.steps)]))
    mres = kr.microbatch_frontier(mseg, mfr.T, mfr.E, mK, mF, mseq, mcT_d, mcE_d,
                                  n_bins=MB_BINS, out=mbuf)
    kr.microbatch_enumerate(mseg, mfr.T, mfr.E, mK, mF, mseq, mcT_d, mcE_d, check=False,
                            out=xbuf)
    torch.cuda.synchronize()
    for k in range(args.steps):
        mev[2 * k].record()
        kr.microbatch_enumerate(mseg, mfr.T, mfr.E, mK, mF, mseq, mcT_d, mcE_d, check=False,
                                out=xbuf)
        mev[2 * k + 1].record()
    torch.cuda.synchronize()
    mx_ms = float(np.median([mev[2 * k].elapsed_time(mev[2 * k + 1]) for k in range(args.steps)]))
    mexa = kr.microbatch_enumerate(mseg, mfr.T, mfr.E, mK, mF, mseq, mcT_d, mcE_d, out=xbuf)
    out["microbatch"] = {
        "workload": "microbatch-llama: 4 partition types (llama-layer tables), 16 layers of "
                    "all four (64 partitions), 64 frequencies, 2 components",
        "configurations": n_configs,
        "enumerate_ms": round(mx_ms, 4), "enumerate_points": int(mexa.T.numel()),
        "configurations_per_s": n_configs / (mx_ms * 1e-3),
        "grid_ms": round(mb_ms, 4), "grid_bins": MB_BINS, "grid_points": int(mres.T.numel())}

    out["mbo"], mbo_ctx = bench_mbo(kr, I, torch, sp, d, args, mk)

    # Frontier comparison metrics (Section 6.1): the eval-stress frontier points against
    # the same points 3 % faster and 5 % cheaper, timed on their own.
    cA_T, cA_E = fr.T[:cap], fr.E[:cap]
    cB_T, cB_E = cA_T * 0.97, cA_E * 0.95
    cmp_out = kr.compare_frontiers(cA_T, cA_E, cB_T, cB_E)
    torch.cuda.synchronize()
    cev = mk(2 * args.steps)
    for k in range(args.steps):
        cev[2 * k].record()
        kr.compare_frontiers(cA_T, cA_E, cB_T, cB_E, out=cmp_out)
        cev[2 * k + 1].record()
    torch.cuda.synchronize()
    cmp_ms = float(np.median([cev[2 * k].elapsed_time(cev[2 * k + 1]) for k in range(args.steps)]))
    cm = cmp_out.cpu().numpy()
    out["frontier_metrics"] = {
        "workload": "eval-stress frontier points (%d) against the same points x (0.97 T, "
                    "0.95 E)" % cap,
        "points": 2 * cap, "call_ms": round(cmp_ms, 4),
        "algorithmic_bytes": 56 * cap,
        "achieved_GBps": round(56 * cap / (cmp_ms * 1e-3) / 1e9, 1),
        "leftmost_time_reduction_pct": float(cm[0]), "leftmost_energy_reduction_pct": float(cm[1]),
        "iso_time_energy_reduction_pct": float(cm[2]),
        "iso_energy_time_reduction_pct": float(cm[3])}

    out["launch_timing"], dp_ctx = bench_dp(kr, I, torch, args, mk)
    out["eval_two_comm"], e2_ctx = bench_eval2(kr, I, torch, args, mk)

    if not args.skip_cpu:
        import oracle

        oracle.build(force=False)
        # the single-threaded legs run on one core: this thread is pinned to the first CPU
        # it may use, and the mask is restored for the partition-parallel leg
        all_cpus = os.sched_getaffinity(0)
        pin_cpu = min(all_cpus)
        os.sched_setaffinity(0, {pin_cpu})
        t0 = time.perf_counter()
        n = 0
        mism = 0
        off = fr.off.cpu().numpy()
        gidx = fr.idx.cpu().numpy()
        while n < sp.n_parts and (time.perf_counter() - t0) < args.cpu_seconds:
            T, E = oracle.evaluate_partition(sp, w.t, w.pw, w.tc, w.pc, n)
            ix = oracle.pareto(T, E)
            mism += int(not np.array_equal(gidx[off[n]:off[n + 1]], ix))
            n += 1
        el = time.perf_counter() - t0
        out["cpu_baseline"] = {
            "value": n * sp.n_cand / el, "unit": "candidates/s", "cores": 1, "kind": "oracle",
            "sample": "first %d of the 1024 eval-stress partitions (%d candidates), evaluate + "
                      "GetFrontier, single-threaded C oracle, %.1f s" % (n, n * sp.n_cand, el)}
        out["parity_check"] = {"partitions": n, "frontier_mismatches": mism}
        # the same oracle, partition-parallel over the host's cores (ctypes calls release
        # the interpreter lock), over the batch from its first partition
        import concurrent.futures as cfu

        os.sched_setaffinity(0, all_cpus)  # worker threads inherit the mask of this thread
        nthreads = len(all_cpus)

        def one(q):
            T, E = oracle.evaluate_partition(sp, w.t, w.pw, w.tc, w.pc, q)
            return oracle.pareto(T, E)

        t0 = time.perf_counter()
        done = 0
        with cfu.ThreadPoolExecutor(max_workers=nthreads) as ex:
            futs = []
            for q in range(sp.n_parts):
                futs.append(ex.submit(one, q))
                if len(futs) >= 4 * nthreads:
                    futs.pop(0).result()
                    done += 1
                    if time.perf_counter() - t0 > args.cpu_seconds:
                        break
            for f in futs:
                f.result()
                done += 1
        el = time.perf_counter() - t0
        os.sched_setaffinity(0, {pin_cpu})
        out["cpu_baseline_parallel"] = {
            "value": done * sp.n_cand / el, "unit": "candidates/s", "cores": nthreads,
            "kind": "oracle",
            "sample": "%d eval-stress partitions, evaluate + GetFrontier, %d threads, %.1f s"
                      % (done, nthreads, el)}
        t0 = time.perf_counter()
        oracle.compose(off4, T4, E4, B)
        el = time.perf_counter() - t0
        out["cpu_baseline_compose"] = {"value": cells / el, "unit": "cells/s", "cores": 1,
                                       "kind": "oracle", "sample": "full compose-stress batch, "
                                       "%.1f s" % el}
        # the oracle's own per-(type, frequency) frontiers of the same tables
        oseg, oT, oE = [0], [], []
        for t in range(mK):
            Tr, Er = oracle.evaluate_partition(msp, mb_w.t, mb_w.pw, mb_w.tc, mb_w.pc, t)
            for f in range(mF):
                ix = oracle.pareto(Tr[f * mCf:(f + 1) * mCf], Er[f * mCf:(f + 1) * mCf])
                oT.append(Tr[f * mCf + ix])
                oE.append(Er[f * mCf + ix])
                oseg.append(oseg[-1] + len(ix))
        oseg, oT, oE = np.array(oseg, dtype=np.int64), np.concatenate(oT), np.concatenate(oE)
        t0 = time.perf_counter()
        rx = oracle.microbatch_exact(oseg, oT, oE, mK, mF, mseq, mcT, mcE)
        el = time.perf_counter() - t0
        t0 = time.perf_counter()
        ro = oracle.microbatch(oseg, oT, oE, mK, mF, mseq, mcT, mcE, n_bins=MB_BINS)
        elg = time.perf_counter() - t0
        out["microbatch"]["cpu_baseline"] = {
            "value": n_configs / el, "unit": "configurations/s", "cores": 1, "kind": "oracle",
            "sample": "the same microbatch by enumeration, %.4f s (grid composition %.2f s)"
                      % (el, elg),
            "parity": bool(np.array_equal(oseg, mseg) and
                           np.array_equal(rx[0], mexa.T.cpu().numpy()) and
                           np.array_equal(rx[3], mexa.choice.cpu().numpy()) and
                           np.array_equal(ro[0], mres.T.cpu().numpy()) and
                           np.array_equal(ro[3], mres.choice.cpu().numpy()))}
        out["mbo"]["cpu_baseline"] = mbo_cpu_baseline(oracle, I, w, mbo_ctx, args.cpu_seconds)
        # the oracle's own frontier points of the same batch (its evaluation + GetFrontier)
        oT, oE = [], []
        for p in range(sp.n_parts):
            Tr, Er = oracle.evaluate_partition(sp, w.t, w.pw, w.tc, w.pc, p)
            ix = oracle.pareto(Tr, Er)
            oT.append(Tr[ix])
            oE.append(Er[ix])
        oT, oE = np.concatenate(oT), np.concatenate(oE)
        t0 = time.perf_counter()
        rc = oracle.compare(oT, oE, oT * 0.97, oE * 0.95)
        el = time.perf_counter() - t0
        out["frontier_metrics"]["cpu_baseline"] = {
            "value": 2 * len(oT) / el, "unit": "points/s", "cores": 1, "kind": "oracle",
            "sample": "the same comparison, %.4f s" % el,
            "parity": bool(np.array_equal(rc, cm, equal_nan=True))}
        out["launch_timing"]["cpu_baseline"] = dp_cpu_baseline(oracle, dp_ctx, args.cpu_seconds)
        out["eval_two_comm"]["cpu_baseline"] = eval2_cpu_baseline(oracle, e2_ctx, args.cpu_seconds)
        os.sched_setaffinity(0, all_cpus)
        host = host_info(pin_cpu)
        for k in ("cpu_baseline", "cpu_baseline_compose"):
            out[k]["host"] = host
    print(json.dumps(out))


def host_info(pin_cpu):
    """CPU model, logical CPUs, the core the single-threaded legs ran on, and the
    oracle's compiler with its version and flags."""
    import subprocess

    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    import oracle

    try:
        gcc = subprocess.run(["gcc", "--version"], capture_output=True, text=True,
                             timeout=30).stdout.splitlines()[0]
    except (OSError, IndexError, subprocess.SubprocessError):
        gcc = "unknown"
    return {"cpu": model, "logical_cpus": os.cpu_count(),
            "usable_cpus": len(os.sched_getaffinity(0)), "pinned_cpu": pin_cpu,
            "compiler": gcc, "oracle_build": "gcc " + " ".join(oracle.CFLAGS),
            "threads_used": 1}


def bench_eval2(kr, I, torch, args, mk):
    """Fused evaluation + frontier filter of the two-comm workload (256 partitions x
    1,148,928 candidates, two comm kernels): VALU-bound, reported as candidates/s."""
    w2 = I.config_workload(2)
    sp2 = w2.space
    d2 = [torch.from_numpy(getattr(w2, k)).cuda() for k in ("t", "pw", "tc", "pc")]
    fr = kr.evaluate_and_filter(sp2, *d2)
    cap = int(fr.off[-1].item())
    for _ in range(args.warmup):
        kr.evaluate_and_filter(sp2, *d2, cap=cap, sync=False)
    torch.cuda.synchronize()
    steps = max(3, args.steps // 4)
    ev = mk(2 * steps)
    kev = [mk(2) for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        kr.set_phase_events(kr.PHASE_EVAL_TILE, *kev[k])
        ev[2 * k].record()
        fr = kr.evaluate_and_filter(sp2, *d2, cap=cap, sync=False)
        ev[2 * k + 1].record()
    torch.cuda.synchronize()
    kr.set_phase_events(kr.PHASE_EVAL_TILE)
    ms = sorted(ev[2 * k].elapsed_time(ev[2 * k + 1]) for k in range(steps))
    kms = float(np.median([e[0].elapsed_time(e[1]) for e in kev]))
    n = sp2.n_parts * sp2.n_cand
    nbytes = sum(x.numel() * 8 for x in d2)
    c2 = read_summary(EVAL2_COUNTERS, eval2_source_hash())
    roof = {"bound": "alu", "kernel": "eval_filter_pair_kernel<8,16,4> (four waves per slab, "
            "two comm kernels)", "kernel_ms": round(kms, 4), "peak": VALU_ISSUE_PEAK / 1e9,
            "unit": "G VALU wave-instructions/s", "achieved": None, "frac": None,
            "hbm_GBps": round(nbytes / (kms * 1e-3) / 1e9, 1),
            "hbm_frac": round(nbytes / (kms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "algorithmic_bytes": nbytes,
            "source": "kernel changed since counters were taken" if c2 is None else
            "profiles/eval_two_comm_counters.txt"}
    if c2 is not None:
        vi = float(c2["valu_wave_instructions_per_launch"]) / (kms * 1e-3)
        roof.update(achieved=round(vi / 1e9, 2), frac=round(vi / VALU_ISSUE_PEAK, 4),
                    valu_busy=float(c2["valu_busy"]),
                    valu_per_wave_candidate=round(64 * float(c2["valu_wave_instructions_per_launch"])
                                                  / n, 1))
    res = {"workload": "two-comm (256 partitions x 1,148,928 candidates: 48 kernels, 561 "
                       "launch-position pairs, 8 x 8 SM choices, 32 frequencies)",
           "candidates": n, "frontier_points": cap, "call_ms_median": round(ms[len(ms) // 2], 4),
           "candidates_per_s": n / (ms[len(ms) // 2] * 1e-3), "roofline": roof}
    return res, dict(w=w2, fr=fr)


def eval2_cpu_baseline(oracle, ctx, seconds):
    """The oracle's evaluation + GetFrontier on the first partitions of the two-comm batch
    (at least one), checked against the GPU's frontiers."""
    w, fr = ctx["w"], ctx["fr"]
    off, idx = fr.off.cpu().numpy(), fr.idx.cpu().numpy()
    t0 = time.perf_counter()
    n, mism = 0, 0
    while n < w.space.n_parts and (n == 0 or time.perf_counter() - t0 < seconds):
        T, E = oracle.evaluate_partition(w.space, w.t, w.pw, w.tc, w.pc, n)
        mism += int(not np.array_equal(idx[off[n]:off[n + 1]], oracle.pareto(T, E)))
        n += 1
    el = time.perf_counter() - t0
    return {"value": n * w.space.n_cand / el, "unit": "candidates/s", "cores": 1,
            "kind": "oracle",
            "sample": "first %d of the 256 partitions, evaluate + GetFrontier, %.1f s" % (n, el),
            "frontier_mismatches": mism}


def bench_dp(kr, I, torch, args, mk):
    """Launch-timing frontiers (Appendix B's dynamic program) of two nanobatches of a
    transformer block for every (partition, frequency, SM choice) of the two-comm tables."""
    w2 = I.config_workload(2)
    sp2 = w2.space
    k1, k2, ops, idx = I.dp_instances(w2, range(sp2.n_parts))
    ops_d = torch.from_numpy(ops).cuda()
    res = kr.launch_timing_frontier(k1, k2, ops_d, sp2.p_static, I.DP_KMAX)
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        kr.launch_timing_frontier(k1, k2, ops_d, sp2.p_static, I.DP_KMAX, check=False, out=res)
    torch.cuda.synchronize()
    ev = mk(2 * args.steps)
    for k in range(args.steps):
        ev[2 * k].record()
        kr.launch_timing_frontier(k1, k2, ops_d, sp2.p_static, I.DP_KMAX, check=False, out=res)
        ev[2 * k + 1].record()
    torch.cuda.synchronize()
    assert int(res.status.item()) == 0
    ms = float(np.median([ev[2 * k].elapsed_time(ev[2 * k + 1]) for k in range(args.steps)]))
    n = ops.shape[0]
    cells = n * ((len(k1) + 1) * (len(k2) + 1) - 1)
    sizes = res.n.cpu().numpy()
    out = {
        "workload": "launch-timing-two-comm: two nanobatches of a transformer block (4 "
                    "computations, a collective, 5 computations, a collective) per "
                    "(partition, frequency, SM choice) of the two-comm tables, overlap runs "
                    "up to %d" % I.DP_KMAX,
        "instances": n, "cells": cells, "call_ms": round(ms, 4),
        "instances_per_s": n / (ms * 1e-3), "cells_per_s": cells / (ms * 1e-3),
        "frontier_points_mean": float(sizes.mean()), "frontier_points_max": int(sizes.max())}
    return out, dict(k1=k1, k2=k2, ops=ops, res=res, ps=sp2.p_static)


def dp_cpu_baseline(oracle, ctx, seconds):
    """The oracle's dynamic program on the first instances of the same batch for about
    `seconds`, checked bit for bit against the GPU's frontiers."""
    import torch  # noqa: F401

    res = ctx["res"]
    gT, gE, gn = res.T.cpu().numpy(), res.E.cpu().numpy(), res.n.cpu().numpy()
    gS = res.sched.cpu().numpy()
    t0 = time.perf_counter()
    n, mism = 0, 0
    while n < len(ctx["ops"]) and time.perf_counter() - t0 < seconds:
        T, E, S, _ = oracle.launch_dp(ctx["k1"], ctx["k2"], ctx["ops"][n], ctx["ps"], 9)
        m = len(T)
        mism += int(not (gn[n] == m and np.array_equal(gT[n, :m], T) and
                         np.array_equal(gE[n, :m], E) and np.array_equal(gS[n, :m], S)))
        n += 1
    el = time.perf_counter() - t0
    return {"value": n / el, "unit": "instances/s", "cores": 1, "kind": "oracle",
            "sample": "first %d of the instances, single-threaded C oracle, %.1f s" % (n, el),
            "mismatches": mism}


def mbo_inputs(kr, I, torch, sp, d, seed=11):
    """Predictions of every eval-stress candidate (the cost model), a measured sample of
    96 per partition and a 5-member ensemble around the predictions, all on the device."""
    T, E = kr.evaluate_partition(sp, *d)
    T, E = T.reshape(-1), E.reshape(-1)
    C, P = sp.n_cand, sp.n_parts
    obs_off, idx, z = I.mbo_observations(seed, [C] * P, I.MBO_N_INIT)
    gidx = torch.from_numpy(np.repeat(np.arange(P, dtype=np.int64) * C, I.MBO_N_INIT) + idx).cuda()
    zd = torch.from_numpy(z).cuda()
    To = I.perturb(T[gidx], zd[:, 0].contiguous(), 0.02)
    Eo = I.perturb(E[gidx], zd[:, 1].contiguous(), 0.02)
    tab = torch.from_numpy(I.noise_table(seed + 1)).cuda()
    x = torch.arange(C * P, device="cuda", dtype=torch.int64)
    Tm = torch.empty((I.MBO_MEMBERS, C * P), dtype=torch.float64, device="cuda")
    Em = torch.empty_like(Tm)
    for m in range(I.MBO_MEMBERS):
        Tm[m] = I.perturb(T, tab[I.noise_index(2 * m, x)], 0.05)
        Em[m] = I.perturb(E, tab[I.noise_index(2 * m + 1, x)], 0.05)
    del x
    return dict(T=T, E=E, To=To, Eo=Eo, Tm=Tm, Em=Em, idx=idx, z=z, seed=seed,
                cand_off=torch.arange(P + 1, dtype=torch.int64, device="cuda") * C,
                obs_off=torch.from_numpy(obs_off).cuda(),
                idx_d=torch.from_numpy(idx).cuda())


def bench_mbo(kr, I, torch, sp, d, args, mk):
    """Scores and batch selection of the Bayesian optimisation (Section 4.3, Algorithm 1)
    over the whole eval-stress candidate space: the three HVI scores of every candidate,
    the ensemble uncertainty, and one batch of 32 per partition."""
    c = mbo_inputs(kr, I, torch, sp, d)
    n = c["T"].numel()
    P = sp.n_parts
    k1, k2, k3 = I.MBO_PASSES
    sc = kr.hvi_scores(c["cand_off"], c["T"], c["E"], c["obs_off"], c["To"], c["Eo"], sp.p_static)
    unc = kr.uncertainty(c["Tm"], c["Em"])
    bt = kr.select_batch(c["cand_off"], sc.hvi, unc, c["obs_off"], c["idx_d"], k1, k2, k3,
                         I.MBO_BATCH)
    torch.cuda.synchronize()

    def run():
        kr.hvi_scores(c["cand_off"], c["T"], c["E"], c["obs_off"], c["To"], c["Eo"],
                      sp.p_static, check=False, out=sc)
        kr.uncertainty(c["Tm"], c["Em"], out=unc)
        kr.select_batch(c["cand_off"], sc.hvi, unc, c["obs_off"], c["idx_d"], k1, k2, k3,
                        I.MBO_BATCH, check=False, out=bt)

    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    steps = args.steps
    ev = [mk(2) for _ in range(steps)]
    ph = [[mk(2) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    for k in range(steps):
        kr.set_phase_events(kr.PHASE_HVI, *ph[k][0])
        kr.set_phase_events(kr.PHASE_UNC, *ph[k][1])
        kr.set_phase_events(kr.PHASE_SELECT, *ph[k][2])
        ev[k][0].record()
        run()
        ev[k][1].record()
    torch.cuda.synchronize()
    for p in (kr.PHASE_HVI, kr.PHASE_UNC, kr.PHASE_SELECT):
        kr.set_phase_events(p)
    assert int(sc.status.item()) == 0 and int(bt.status.item()) == 0
    step_ms = float(np.median([e[0].elapsed_time(e[1]) for e in ev]))
    hvi_ms, unc_ms, sel_ms = (float(np.median([q[i][0].elapsed_time(q[i][1]) for q in ph]))
                              for i in range(3))

    traffic, tsrc = read_mbo_traffic()

    def roof(nbytes, ms, kernel):
        a = nbytes / (ms * 1e-3) / 1e9
        name = kernel.split(" ")[0]
        return {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(a / HBM_PEAK_GBS, 4), "traffic": traffic.get(name),
                "kernel": kernel, "kernel_ms": round(ms, 4), "algorithmic_bytes": nbytes,
                "traffic_source": tsrc}

    M = I.MBO_MEMBERS
    res = {
        "workload": "mbo-eval-stress: every candidate of the 1,024 eval-stress partitions "
                    "(135,168 each) scored against 96 measured points per partition "
                    "(3 HVI variants), a 5-member ensemble, one batch of 32 per partition "
                    "(13 / 6 / 6 by HVI, the rest by uncertainty)",
        "candidates": n, "partitions": P,
        "step_ms": round(step_ms, 4), "candidates_per_s": n / (step_ms * 1e-3),
        "hvi_ms": round(hvi_ms, 4), "uncertainty_ms": round(unc_ms, 4),
        "select_tile_ms": round(sel_ms, 4),
        "roofline": roof(40 * n, hvi_ms, "hvi_score_kernel (2 predictions in, 3 scores out)"),
        "uncertainty_roofline": roof((16 * M + 8) * n, unc_ms,
                                     "unc_kernel (%d members x 2 predictions in, 1 out)" % M),
        "select_roofline": roof(32 * n, sel_ms, "sel_tile_kernel (4 scores in)"),
    }
    ctx = dict(c=c, sc=sc, unc=unc, bt=bt, sp=sp)
    return res, ctx


def mbo_cpu_baseline(oracle, I, w, ctx, seconds):
    """The oracle's scores, uncertainty and selection on whole partitions from the start
    of the batch (its own cost-model predictions), for about `seconds`; scores compared
    with the GPU's within the rounding bound of the parity tests."""
    c, sp = ctx["c"], ctx["sp"]
    C = sp.n_cand
    U = 2.0 ** -53
    gh = ctx["sc"].hvi
    tab = I.noise_table(c["seed"] + 1)
    t0 = time.perf_counter()
    n, worst = 0, 0.0
    while n < sp.n_parts and (time.perf_counter() - t0) < seconds:
        Tr, Er = oracle.evaluate_partition(sp, w.t, w.pw, w.tc, w.pc, n)
        o = slice(n * I.MBO_N_INIT, (n + 1) * I.MBO_N_INIT)
        To = I.perturb(Tr[c["idx"][o]], c["z"][o, 0], 0.02)
        Eo = I.perturb(Er[c["idx"][o]], c["z"][o, 1], 0.02)
        rh, rhv, _ = oracle.hvi([0, C], Tr, Er, [0, I.MBO_N_INIT], To, Eo, sp.p_static)
        xs = np.arange(n * C, (n + 1) * C, dtype=np.int64)
        Tm = np.stack([I.perturb(Tr, tab[I.noise_index(2 * m, xs)], 0.05)
                       for m in range(I.MBO_MEMBERS)])
        Em = np.stack([I.perturb(Er, tab[I.noise_index(2 * m + 1, xs)], 0.05)
                       for m in range(I.MBO_MEMBERS)])
        ru = oracle.uncertainty(Tm, Em)
        k1, k2, k3 = I.MBO_PASSES
        oracle.select([0, C], rh, ru, [0, I.MBO_N_INIT], c["idx"][o], k1, k2, k3, I.MBO_BATCH)
        g = gh[:, n * C:(n + 1) * C].cpu().numpy()
        tol = (3 * (I.MBO_N_INIT + 1) + 8) * U * (rhv[0][:, None] + np.maximum(abs(g), abs(rh)))
        worst = max(worst, float(np.max(np.abs(g - rh) / tol)))
        n += 1
    el = time.perf_counter() - t0
    return {"value": n * C / el, "unit": "candidates/s", "cores": 1, "kind": "oracle",
            "sample": "first %d of the 1024 partitions (%d candidates): cost model, 3 HVI "
                      "scores, uncertainty and selection, single-threaded C oracle, %.1f s"
                      % (n, n * C, el),
            "parity_worst_error_over_bound": worst}


if __name__ == "__main__":
    main()
