"""Seeded synthetic inputs for the schedule search: per-kernel time/power tables and
precomputed partition frontiers.

This module is shared by the HIP path, the CPU oracle, the tests and the benchmark.
It only draws random numbers and expands them into tables; it holds none of the
method's arithmetic (no cost model, no Pareto filter, no composition).

The paper profiles every candidate schedule on A100 GPUs (Section 5.3) and ships no
traces, so these tables stand in for the profiled per-kernel time and power of its
Llama / Qwen partitions (Section 6.1).  The modelled training GPU is a synthetic
132-SM part with a 1005-1980 MHz clock grid; it is a parameter of the generator and
has nothing to do with the GPU that runs the planner.

Random numbers: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014), used as a counter-based stream: draw k of seed s is
mix(s + (k + 1) * 0x9E3779B97F4A7C15); a uniform double is the top 53 bits * 2^-53.

Table layout (row-major, fp64), per partition p and frequency index f:
  t [P][F][N][S+1]   compute-kernel time (s) in SM state s
  pw[P][F][N][S+1]   compute-kernel dynamic power (W) in SM state s
  tc[P][F][M][S]     comm-kernel time (s) with SM choice s
  pc[P][F][M][S]     comm-kernel dynamic power (W) with SM choice s
SM state 0 means no communication is running (all SMs available to compute);
state s >= 1 means communication holds sm_counts[s-1] SMs.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

TOTAL_SMS = 132.0
P_STATIC_W = 90.0


def splitmix64_uniform(seed: int, start: int, count: int) -> np.ndarray:
    """Uniform doubles in [0, 1): draws start .. start+count-1 of stream `seed`."""
    with np.errstate(over="ignore"):
        k = np.arange(start + 1, start + count + 1, dtype=np.uint64)
        z = np.uint64(seed) + k * _GAMMA
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        z = z ^ (z >> np.uint64(31))
    return (z >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)


def _log_uniform(u: np.ndarray, lo: float, hi: float) -> np.ndarray:
    return np.exp(np.log(lo) + u * (np.log(hi) - np.log(lo)))


@dataclasses.dataclass(frozen=True)
class Space:
    """Shape of one batch of partitions and its candidate axes."""

    n_parts: int
    n_kernels: int
    n_comm: int
    n_pos: int
    sm_counts: tuple
    freqs_mhz: tuple
    p_static: float = P_STATIC_W
    total_sms: float = TOTAL_SMS

    @property
    def n_freq(self) -> int:
        return len(self.freqs_mhz)

    @property
    def n_sm(self) -> int:
        return len(self.sm_counts)

    @property
    def n_pairs(self) -> int:
        """Ordered launch-position pairs p1 <= p2 (two comm kernels)."""
        return self.n_pos * (self.n_pos + 1) // 2

    @property
    def cand_per_freq(self) -> int:
        if self.n_comm == 1:
            return self.n_pos * self.n_sm
        return self.n_pairs * self.n_sm * self.n_sm

    @property
    def n_cand(self) -> int:
        """Candidates per partition."""
        return self.n_freq * self.cand_per_freq


@dataclasses.dataclass
class Workload:
    space: Space
    t: np.ndarray
    pw: np.ndarray
    tc: np.ndarray
    pc: np.ndarray
    bins: Optional[int] = None
    name: str = ""


def make_tables(space: Space, seed: int, comm_bytes: Sequence[float],
                parts: Optional[range] = None) -> Dict[str, np.ndarray]:
    """Draw the per-kernel tables of `space` (all partitions, or the range `parts`).

    Per partition, per compute kernel: t0 ~ logU(20 us, 2 ms), alpha ~ U(0.3, 1),
    beta ~ U(0.2, 1), P0 ~ U(300, 700) W, gamma ~ U(1.5, 2.5); then per comm kernel:
    bytes ~ logU(comm_bytes), c ~ U(80, 200) W.
      t  = t0 * (alpha * fmax / f + 1 - alpha) * (132 / k_avail) ** beta
      pw = P0 * (f / fmax) ** gamma * (k_avail / 132)
      tc = bytes / (400 GB/s * min(1, k / 16) * (0.6 + 0.4 * f / fmax))
      pc = c * k / 32
    """
    P, N, M = space.n_parts, space.n_kernels, space.n_comm
    if parts is None:
        parts = range(P)
    per = 5 * N + 2 * M
    u = splitmix64_uniform(seed, parts.start * per, len(parts) * per).reshape(len(parts), per)
    ku = u[:, : 5 * N].reshape(len(parts), N, 5)
    cu = u[:, 5 * N:].reshape(len(parts), M, 2)
    t0 = _log_uniform(ku[..., 0], 20e-6, 2e-3)
    alpha = 0.3 + 0.7 * ku[..., 1]
    beta = 0.2 + 0.8 * ku[..., 2]
    p0 = 300.0 + 400.0 * ku[..., 3]
    gamma = 1.5 + 1.0 * ku[..., 4]
    nbytes = _log_uniform(cu[..., 0], comm_bytes[0], comm_bytes[1])
    cpow = 80.0 + 120.0 * cu[..., 1]

    f = np.asarray(space.freqs_mhz, dtype=np.float64)
    fmax = f.max()
    k = np.asarray(space.sm_counts, dtype=np.float64)
    kav = np.concatenate([[space.total_sms], space.total_sms - k])  # [S+1]

    # [p][f][i] frequency factor, [p][i][s] SM factor
    ffac = t0[:, None, :] * (alpha[:, None, :] * (fmax / f)[None, :, None] + 1.0 - alpha[:, None, :])
    sfac = (space.total_sms / kav)[None, None, :] ** beta[:, :, None]
    t = ffac[:, :, :, None] * sfac[:, None, :, :]
    pf = p0[:, None, :] * (f / fmax)[None, :, None] ** gamma[:, None, :]
    pw = pf[:, :, :, None] * (kav / space.total_sms)[None, None, None, :]

    bw = 400e9 * np.minimum(1.0, k / 16.0)[None, :] * (0.6 + 0.4 * f / fmax)[:, None]  # [F][S]
    tc = nbytes[:, None, :, None] / bw[None, :, None, :]
    pc = np.broadcast_to((cpow[:, :, None] * (k / 32.0)[None, None, :])[:, None, :, :],
                         tc.shape).copy()
    return dict(t=np.ascontiguousarray(t), pw=np.ascontiguousarray(pw),
                tc=np.ascontiguousarray(tc), pc=pc)


def _grid(lo: float, hi: float, n: int) -> tuple:
    return tuple(float(x) for x in np.linspace(lo, hi, n))


# The five workload shapes.  Seeds are the config index.
SPACES = {
    0: dict(space=Space(4, 6, 1, 7, tuple(range(4, 33, 4)), _grid(1005.0, 1980.0, 16)),
            comm_bytes=(4e6, 64e6), bins=1024, name="tiny: 4 partitions x 6 kernels, 896 cand/part"),
    1: dict(space=Space(64, 24, 1, 25, tuple(range(2, 33, 2)),
                        tuple(1005.0 + 15.0 * j for j in range(64))),
            comm_bytes=(16e6, 256e6), bins=16384,
            name="llama-layer: 64 partitions x 24 kernels, 25,600 cand/part"),
    2: dict(space=Space(256, 48, 2, 33, tuple(range(4, 33, 4)), _grid(1005.0, 1980.0, 32)),
            comm_bytes=(8e6, 512e6), bins=32768,
            name="two-comm: 256 partitions x 48 kernels, 2 comm kernels, 1,148,928 cand/part"),
    3: dict(space=Space(1024, 32, 1, 33, tuple(range(1, 33)),
                        tuple(1005.0 + 7.5 * j for j in range(128))),
            comm_bytes=(4e6, 64e6), bins=None,
            name="eval-stress: 1024 partitions x 32 kernels, 135,168 cand/part"),
}

COMPOSE_SPACE = dict(n_parts=512, n_min=256, n_max=2048, t_lo=50e-6, t_hi=50e-3, bins=65536,
                     name="compose-stress: 512 frontiers of 256-2048 points, 65,536 bins")


def config_workload(cfg: int, parts: Optional[range] = None) -> Workload:
    """Tables of workload `cfg` (0..3), seed = cfg."""
    spec = SPACES[cfg]
    space = spec["space"]
    tabs = make_tables(space, seed=cfg, comm_bytes=spec["comm_bytes"], parts=parts)
    if parts is not None:
        space = dataclasses.replace(space, n_parts=len(parts))
    return Workload(space=space, bins=spec["bins"], name=spec["name"], **tabs)


def random_space(rng: np.random.Generator, n_comm: int = 1, max_kernels: int = 6,
                 max_sm: int = 4, max_freq: int = 3, n_parts: int = 2) -> Space:
    """A small random space for property tests."""
    N = int(rng.integers(1, max_kernels + 1))
    S = int(rng.integers(1, max_sm + 1))
    F = int(rng.integers(1, max_freq + 1))
    n_pos = int(rng.integers(1, N + 2))
    sms = tuple(sorted(int(x) for x in rng.choice(np.arange(1, 33), size=S, replace=False)))
    freqs = tuple(float(x) for x in sorted(rng.choice(np.arange(1005, 1981, 15), size=F,
                                                      replace=False)))
    return Space(n_parts, N, n_comm, n_pos, sms, freqs)


def compose_frontiers(seed: int = 4, n_parts: int = 512, n_min: int = 256, n_max: int = 2048,
                      t_lo: float = 50e-6, t_hi: float = 50e-3):
    """Precomputed partition frontiers for the composition stress workload.

    Per partition: n ~ U{n_min..n_max}; times are n sorted logU(t_lo, t_hi) draws;
    energies start at 1 J and fall by decrements d_j whose raw sizes r_j shrink by a
    U(0.5, 1) factor per step (r_1 = 1), scaled so the total fall is 0.5 J.
    Returns (off int64[P+1], T float64[n], E float64[n]).
    """
    T_parts: List[np.ndarray] = []
    E_parts: List[np.ndarray] = []
    cursor = 0
    for _ in range(n_parts):
        n = n_min + int(splitmix64_uniform(seed, cursor, 1)[0] * (n_max - n_min + 1))
        n = min(n, n_max)
        cursor += 1
        T = np.sort(_log_uniform(splitmix64_uniform(seed, cursor, n), t_lo, t_hi))
        cursor += n
        n_ratio = max(n - 2, 0)
        ratios = 0.5 + 0.5 * splitmix64_uniform(seed, cursor, n_ratio)
        cursor += n_ratio
        r = np.ones(max(n - 1, 0))
        r[1:] = np.cumprod(ratios)
        d = 0.5 * r / r.sum() if n > 1 else r
        E = np.empty(n)
        E[0] = 1.0
        acc = 1.0
        for j in range(1, n):
            acc = acc - d[j - 1]
            E[j] = acc
        T_parts.append(T)
        E_parts.append(E)
    off = np.zeros(n_parts + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(x) for x in T_parts])
    return off, np.concatenate(T_parts), np.concatenate(E_parts)


def frontier_batch(seed: int, n_points: Sequence[int], t_span: Sequence[float],
                   t0: float = 1e-3) -> tuple:
    """Frontier-shaped partitions of chosen sizes and time spans.

    Partition k has n_points[k] times t0 + t_span[k] * u (u uniform, sorted, the first
    pinned to 0 and the last to 1 when there are two or more) and energies falling from
    2 J by uniform decrements.  Returns (off int64[P+1], T float64[n], E float64[n]).
    """
    T_parts: List[np.ndarray] = []
    E_parts: List[np.ndarray] = []
    cursor = 0
    for n, span in zip(n_points, t_span):
        u = np.sort(splitmix64_uniform(seed, cursor, n))
        cursor += n
        if n >= 2:
            u[0], u[-1] = 0.0, 1.0
        d = splitmix64_uniform(seed, cursor, n)
        cursor += n
        T_parts.append(t0 + span * u)
        E_parts.append(2.0 - np.cumsum(d) / n)
    off = np.zeros(len(T_parts) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(x) for x in T_parts])
    return off, np.concatenate(T_parts), np.concatenate(E_parts)


def microbatch_components(seed: int, n_comp: int, freqs: Sequence[float]) -> tuple:
    """Non-partition components of a microbatch (kernels outside any partition, such as
    an embedding or a loss), each like a compute kernel running alone: per component
    t0 ~ logU(20 us, 2 ms), alpha ~ U(0.3, 1), P0 ~ U(300, 700) W, gamma ~ U(1.5, 2.5);
    T_c(f) = t0 (alpha fmax / f + 1 - alpha), E_c(f) = P0 (f / fmax)^gamma T_c(f).
    Returns (T [n_comp][F], E [n_comp][F])."""
    f = np.asarray(freqs, dtype=np.float64)
    fmax = f.max()
    u = splitmix64_uniform(seed, 0, 4 * n_comp).reshape(n_comp, 4) if n_comp else np.zeros((0, 4))
    t0 = _log_uniform(u[:, 0], 20e-6, 2e-3)
    alpha = 0.3 + 0.7 * u[:, 1]
    P0 = 300.0 + 400.0 * u[:, 2]
    gamma = 1.5 + u[:, 3]
    T = t0[:, None] * (alpha[:, None] * fmax / f[None, :] + 1.0 - alpha[:, None])
    E = P0[:, None] * (f[None, :] / fmax) ** gamma[:, None] * T
    return T, E


# ---- inputs of the Bayesian optimisation's scores and selection (Section 4.3) --------
# Appendix C's settings for a large partition: 96 initial samples, batches of 32, an
# ensemble of 5; the batch shares 0.4 / 0.2 / 0.2 of total / dynamic / static energy
# rounded to whole candidates, the rest by uncertainty.
MBO_N_INIT = 96
MBO_BATCH = 32
MBO_PASSES = (13, 6, 6)
MBO_MEMBERS = 5
NOISE_TABLE = 1 << 20


def mbo_observations(seed: int, n_cand: Sequence[int], n_obs: int) -> tuple:
    """The measured sample of each partition: n_obs candidate indices drawn uniformly
    (repeats allowed) and a measurement-noise draw in [-1, 1) for the time and the energy
    of each.  Returns (obs_off int64[P+1], obs_idx int64 local indices, z [n][2])."""
    P = len(n_cand)
    u = splitmix64_uniform(seed, 0, 3 * P * n_obs).reshape(P * n_obs, 3)
    n = np.repeat(np.asarray(n_cand, dtype=np.int64), n_obs)
    idx = np.minimum((u[:, 0] * n).astype(np.int64), np.maximum(n - 1, 0))
    obs_off = np.arange(P + 1, dtype=np.int64) * n_obs
    return obs_off, idx, 2.0 * u[:, 1:] - 1.0


def noise_table(seed: int) -> np.ndarray:
    """NOISE_TABLE uniform draws in [-1, 1), indexed by noise_index."""
    return 2.0 * splitmix64_uniform(seed, 0, NOISE_TABLE) - 1.0


def noise_index(stream: int, x):
    """Table slot of draw `stream` for global candidate index x (numpy or torch int64)."""
    return (x * 0x9E3779B1 + (stream + 1) * 0x85EBCA77) & (NOISE_TABLE - 1)


def perturb(v, z, rel: float):
    """v * (1 + rel * z): a prediction or measurement off by up to rel (numpy or torch;
    one rounding per operation, so both give the same bits)."""
    return v * (1.0 + rel * z)


# ---- two-sequence launch-timing instances (Appendix B) ------------------------------
# A transformer block of one nanobatch: four computations, a collective, five
# computations, a collective; two nanobatches give the two sequences (Appendix B's
# 9 computations and the block's collectives per sequence).
DP_BLOCK = (0, 0, 0, 0, 1, 0, 0, 0, 0, 0, 1)
DP_KMAX = 9


def dp_instances(w: "Workload", parts: Sequence[int], block: Sequence[int] = DP_BLOCK) -> tuple:
    """Per (partition, frequency, SM choice) the ops of two nanobatches of `block`, read
    from a workload with two comm kernels: S1 takes computations 0, 1, ... and the comm
    kernels in order, S2 the next computations and the same comm kernels.  Computation
    o: (t alone, power alone, t shared, power shared) at SM state 0 and s + 1;
    communication m: (tc, pc) at SM choice s.  Returns (kind1, kind2, ops [n][I + J][4],
    index [n][3] of (partition, f, s)), instances in (partition, f, s) order."""
    sp = w.space
    parts = np.asarray(list(parts), dtype=np.int64)
    P, F, S = len(parts), sp.n_freq, sp.n_sm
    ncomp = sum(1 for k in block if k == 0)
    t, pw, tc, pc = w.t[parts], w.pw[parts], w.tc[parts], w.pc[parts]
    cols = []
    for seq in range(2):
        ci, cm = seq * ncomp, 0
        for k in block:
            op = np.zeros((P, F, S, 4))
            if k == 0:
                op[..., 0] = t[:, :, ci, 0][:, :, None]
                op[..., 1] = pw[:, :, ci, 0][:, :, None]
                op[..., 2] = t[:, :, ci, 1:S + 1]
                op[..., 3] = pw[:, :, ci, 1:S + 1]
                ci += 1
            else:
                op[..., 0] = tc[:, :, cm % sp.n_comm, :S]
                op[..., 1] = pc[:, :, cm % sp.n_comm, :S]
                cm += 1
            cols.append(op)
    ops = np.stack(cols, axis=3).reshape(P * F * S, len(cols), 4)
    pi, fi, si = np.meshgrid(parts, np.arange(F), np.arange(S), indexing="ij")
    index = np.stack([pi.ravel(), fi.ravel(), si.ravel()], axis=1).astype(np.int32)
    return list(block), list(block), np.ascontiguousarray(ops), index
