"""Problem builders: the five synthetic workloads, as host numpy arrays.

Every array is a simulator *input*; nothing here simulates.  The shapes follow
the paper's setups: models with a single-device latency and a weight size
(Table 1 ranges), devices split into equal groups that share one parallel
configuration (Sec. 4.2, Alg. 2's equal-size groups), Gamma arrivals per model
(Sec. 3.1, Sec. 6.2, Sec. 6.3), SLOs as multiples of the single-device latency
(Sec. 3.2, Sec. 6.2).  No public trace is reproduced; the synthetic Gamma
processes stand in for the paper's production traces.

Stage latency of model m under configuration (S pipeline stages, k-way
intra-op): total = d_m * (1 + 0.05 (S - 1)) * (1 + 0.1 (k - 1)), split evenly
over S stages, i.e. ((d*(1+0.05*(S-1)))*(1+0.1*(k-1)))/(S*k) evaluated left to
right in fp64.  With k = 1 this is the paper's alpha*L/n per-stage model
(Sec. 3.3) with alpha = 1 + 0.05 (S - 1); intra-op parallelism divides the
latency by k at a 10% communication cost per extra device.

Weights are integer MiB.  A group of D devices with per-device memory cap
holds models whose weights sum to at most D * cap (each device stores 1/D of
every hosted model).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

from . import gen

GIB_MIB = 1024


@dataclasses.dataclass
class Problem:
    name: str
    t: np.ndarray               # float64[N] arrival times (shared trace)
    model: np.ndarray           # int32[N] model ids
    d_single: np.ndarray        # float64[M] single-device latency (SLO base), seconds
    weight_mib: np.ndarray      # int64[M]
    cfg_stages: np.ndarray      # int32[C] pipeline depth S of each configuration
    cfg_k: np.ndarray           # int32[C] intra-op degree k
    stage_lat: np.ndarray       # float64[M, C, Smax] stage latencies (0 beyond S_c)
    group_cfg: np.ndarray       # int32[P, G] configuration of each group, -1 unused
    host_mask: np.ndarray       # uint64[P, M] bit g <=> group g hosts model m
    slo_scale: np.ndarray       # float64[K]
    finish_jobs: np.ndarray     # int32[F] jobs (p*K + k) whose per-request output is kept
    meta: dict = dataclasses.field(default_factory=dict)

    @property
    def n_jobs(self) -> int:
        return self.group_cfg.shape[0] * self.slo_scale.shape[0]

    @property
    def events(self) -> int:
        return self.n_jobs * self.t.shape[0]


def stage_latency(d: float, S: int, k: int) -> float:
    return ((d * (1.0 + 0.05 * (S - 1))) * (1.0 + 0.1 * (k - 1))) / (S * k)


def stage_table(d_single, cfgs, smax: Optional[int] = None) -> np.ndarray:
    """float64[M, C, Smax]: even split of the total latency over S stages."""
    smax = smax or max(S for S, _ in cfgs)
    M = len(d_single)
    L = np.zeros((M, len(cfgs), smax), dtype=np.float64)
    for m in range(M):
        for c, (S, k) in enumerate(cfgs):
            v = stage_latency(float(d_single[m]), S, k)
            L[m, c, :S] = v
    return L


def _uniform_range(seed, purpose, n, lo, hi):
    u = gen.uniforms(gen.key(seed, purpose, 0), n)
    return lo + (hi - lo) * u


def _weights_mib(seed, n, lo_gb, hi_gb):
    u = gen.uniforms(gen.key(seed, gen.PURPOSE_WEIGHT, 0), n)
    return np.floor((lo_gb + (hi_gb - lo_gb) * u) * GIB_MIB).astype(np.int64)


def c1_tiny(seed: int = 0, duration: float = 60.0) -> Problem:
    """4 models, 4 devices; every map of models onto the partitions 1+1+1+1
    (S=1), 2+2 (S=2), 4 (S=4), k=1: 4^4 + 2^4 + 1 = 273 placements.  Poisson
    5 req/s per model, SLO scale 5."""
    d = np.array([0.10, 0.15, 0.20, 0.25])
    M = 4
    cfgs = [(1, 1), (2, 1), (4, 1)]
    L = stage_table(d, cfgs)
    t, m = gen.trace(seed, [5.0] * M, 1.0, duration)
    gcfg, masks = [], []
    for c, n_groups in ((0, 4), (1, 2), (2, 1)):
        for assign in np.ndindex(*([n_groups] * M)):
            row = [c] * n_groups + [-1] * (4 - n_groups)
            gcfg.append(row)
            masks.append([1 << a for a in assign])
    return Problem("c1_tiny", t, m, d, np.zeros(M, np.int64), np.array([S for S, _ in cfgs], np.int32),
                   np.array([k for _, k in cfgs], np.int32), L, np.array(gcfg, np.int32),
                   np.array(masks, np.uint64), np.array([5.0]), np.array([0, 100, 256, 272], np.int32),
                   {"devices": 4})


C2_SCALES = [1.0, 1.5, 2.0, 3.0, 4.0, 5.0, 7.5, 10.0]


def c2_greedy_step(seed: int = 2, duration: float = 600.0) -> Problem:
    """16 models (d ~ U[0.1, 0.4] s, w ~ U[2, 6] GB), 16 x 16 GB devices in 4
    groups of 4 at S=4, k=1; Gamma 4 req/s per model, CV 3.  One greedy step
    from the empty selection: all 64 (model, group) additions x 8 SLO scales."""
    M, G = 16, 4
    d = _uniform_range(seed, gen.PURPOSE_LATENCY, M, 0.1, 0.4)
    w = _weights_mib(seed, M, 2.0, 6.0)
    cfgs = [(4, 1)]
    L = stage_table(d, cfgs)
    t, m = gen.trace(seed, [4.0] * M, 3.0, duration)
    gcfg, masks = [], []
    for mm in range(M):
        for g in range(G):
            gcfg.append([0] * G)
            row = [0] * M
            row[mm] = 1 << g
            masks.append(row)
    return Problem("c2_greedy_step", t, m, d, w, np.array([4], np.int32), np.array([1], np.int32), L,
                   np.array(gcfg, np.int32), np.array(masks, np.uint64), np.array(C2_SCALES),
                   np.array([0, 8 * 21 + 5, 8 * 42 + 7, 511], np.int32),
                   {"devices": 16, "device_mem_mib": 16 * GIB_MIB, "group_mem_mib": [4 * 16 * GIB_MIB] * G})


C3_PARTITIONS = [(1, 1, 1), (2, 2, 1), (2, 1, 2), (4, 4, 1), (4, 2, 2), (4, 1, 4),
                 (8, 8, 1), (8, 4, 2), (8, 2, 4), (8, 1, 8)]  # (group size, S, k)


@dataclasses.dataclass
class GreedyProblem:
    """Inputs of the greedy placement search (Alg. 1 / reduced Alg. 2)."""
    name: str
    t: np.ndarray
    model: np.ndarray
    d_single: np.ndarray
    weight_mib: np.ndarray
    cfg_stages: np.ndarray
    cfg_k: np.ndarray
    stage_lat: np.ndarray
    partitions: list            # [{"group_cfg": int32[G], "group_mem_mib": int64[G], "label": str}]
    slo_scale: float
    meta: dict = dataclasses.field(default_factory=dict)


def c3_greedy(seed: int = 3, duration: float = 1200.0, n_models: int = 32, n_devices: int = 64,
              device_mem_gb: int = 32, partitions=C3_PARTITIONS, rate: float = 4.0,
              cv: float = 2.0, slo_scale: float = 5.0) -> GreedyProblem:
    """32 models (d ~ U[0.05, 0.8] s, w ~ U[1, 13] GB), 64 x 32 GB devices,
    equal groups of size 1, 2, 4 or 8 with every (S, k), S*k = size (10
    partitions); Gamma 4 req/s per model, CV 2, 20 minutes, SLO scale 5."""
    M = n_models
    d = _uniform_range(seed, gen.PURPOSE_LATENCY, M, 0.05, 0.8)
    w = _weights_mib(seed, M, 1.0, 13.0)
    cfgs = [(S, k) for _, S, k in partitions]
    L = stage_table(d, cfgs)
    t, m = gen.trace(seed, [rate] * M, cv, duration)
    parts = []
    for c, (size, S, k) in enumerate(partitions):
        G = n_devices // size
        parts.append({"group_cfg": np.full(G, c, np.int32),
                      "group_mem_mib": np.full(G, size * device_mem_gb * GIB_MIB, np.int64),
                      "label": f"{G}x(S={S},k={k})"})
    return GreedyProblem("c3_greedy", t, m, d, w, np.array([S for S, _ in cfgs], np.int32),
                         np.array([k for _, k in cfgs], np.int32), L, parts, slo_scale,
                         {"devices": n_devices, "device_mem_mib": device_mem_gb * GIB_MIB})


def c4_rates(M: int = 64, total: float = 1000.0, exponent: float = 0.9) -> np.ndarray:
    w = np.array([(r + 1) ** (-exponent) for r in range(M)])
    return total * w / w.sum()


def c4_heavy(seed: int = 4, duration: float = 3600.0, n_placements: int = 8192,
             n_finish: int = 16) -> Problem:
    """64 models with power-law (exponent 0.9) rates summing to 1000 req/s,
    d ~ U[0.03, 0.11] s; 128 devices in 16 groups of 8 at S=4, k=2; Gamma CV 4,
    one hour.  Placement c gives model m r_m = clamp(round(48 lambda_m / 1000),
    1, 16) replicas on the first r_m groups of a seeded permutation of the 16
    groups (stream (seed, permute, c*64 + m)).  SLO scale 5."""
    M, G = 64, 16
    lam = c4_rates(M)
    d = _uniform_range(seed, gen.PURPOSE_LATENCY, M, 0.03, 0.11)
    cfgs = [(4, 2)]
    L = stage_table(d, cfgs)
    t, m = gen.trace(seed, lam, 4.0, duration)
    reps = np.clip(np.floor(48.0 * lam / 1000.0 + 0.5), 1, 16).astype(np.int64)
    perms = gen.permutations(seed, gen.PURPOSE_PERMUTE, 0, n_placements * M, G).reshape(n_placements, M, G)
    masks = np.zeros((n_placements, M), dtype=np.uint64)
    for mm in range(M):
        sel = perms[:, mm, : reps[mm]].astype(np.uint64)
        masks[:, mm] = np.bitwise_or.reduce(np.left_shift(np.uint64(1), sel), axis=1)
    step = max(1, n_placements // n_finish)
    fin = np.arange(0, n_placements, step, dtype=np.int32)[:n_finish]
    return Problem("c4_heavy", t, m, d, np.zeros(M, np.int64), np.array([4], np.int32),
                   np.array([2], np.int32), L, np.zeros((n_placements, G), np.int32), masks,
                   np.array([5.0]), fin, {"devices": 128, "replicas": reps.tolist(), "rates": lam.tolist()})


@dataclasses.dataclass
class SweepProblem:
    """One placement, many (trace segment, SLO scale) jobs (CSR traces)."""
    name: str
    t: np.ndarray               # float64[total] all segments back to back
    model: np.ndarray           # int32[total]
    seg_offsets: np.ndarray     # int64[S+1]
    d_single: np.ndarray
    cfg_stages: np.ndarray
    stage_lat: np.ndarray
    group_cfg: np.ndarray       # int32[1, G]
    host_mask: np.ndarray       # uint64[1, M]
    job_placement: np.ndarray   # int32[J]
    job_segment: np.ndarray     # int32[J]
    job_scale: np.ndarray       # float64[J]
    finish_jobs: np.ndarray     # int32[F]
    meta: dict = dataclasses.field(default_factory=dict)

    @property
    def events(self) -> int:
        lens = np.diff(self.seg_offsets)
        return int(lens[self.job_segment].sum())


def c5_grid_point(index: int, n: int = 16):
    i, rem = divmod(index, n * n)
    j, k = divmod(rem, n)
    rate_scale = 0.25 * 16.0 ** (i / (n - 1))
    cv = 8.0 ** (j / (n - 1))
    slo = 20.0 ** (k / (n - 1))
    return rate_scale, cv, slo


def c5_sweep(group_cfg, host_mask, base: Optional[GreedyProblem] = None, n: int = 16,
             duration: float = 600.0, seed0: int = 5000, points=None, threads=None) -> SweepProblem:
    """SLO-curve sweep: one fixed placement (the workload-3 search result) over
    an n x n x n grid of rate scale 0.25*16^(i/(n-1)), CV 8^(j/(n-1)) and SLO
    scale 20^(k/(n-1)); grid point (i*n + j)*n + k gets its own trace with
    4*rate_scale req/s per model for 10 minutes, seed 5000 + index.  Finish
    arrays are kept for the diagonal i = j = k.  `points` restricts the grid
    to a subset of indices (tests)."""
    base = base or c3_greedy()
    M = base.d_single.shape[0]
    idx = list(range(n ** 3)) if points is None else list(points)
    specs = []
    for p in idx:
        rs, cv, _ = c5_grid_point(p, n)
        specs.append((seed0 + p, [4.0 * rs] * M, cv, duration))
    segs = gen.traces(specs, threads=threads)
    lens = np.array([len(s[0]) for s in segs], dtype=np.int64)
    offs = np.zeros(len(segs) + 1, dtype=np.int64)
    np.cumsum(lens, out=offs[1:])
    t = np.concatenate([s[0] for s in segs]) if segs else np.zeros(0)
    mo = np.concatenate([s[1] for s in segs]) if segs else np.zeros(0, np.int32)
    scales = np.array([c5_grid_point(p, n)[2] for p in idx])
    diag = {(i * n + i) * n + i for i in range(n)}
    fin = np.array([q for q, p in enumerate(idx) if p in diag], dtype=np.int32)
    gcfg = np.asarray(group_cfg, np.int32).reshape(1, -1)
    hm = np.asarray(host_mask, np.uint64).reshape(1, -1)
    # keep only the configurations the placement uses (renumbered in order)
    used = sorted(set(int(c) for c in gcfg.ravel() if c >= 0))
    remap = {c: i for i, c in enumerate(used)}
    gcfg = np.array([[remap[int(c)] if c >= 0 else -1 for c in gcfg[0]]], np.int32)
    cfg_stages = base.cfg_stages[used]
    smax = int(cfg_stages.max())
    L = np.ascontiguousarray(base.stage_lat[:, used, :smax])
    return SweepProblem("c5_sweep", t, mo.astype(np.int32), offs, base.d_single, cfg_stages,
                        L, gcfg, hm, np.zeros(len(idx), np.int32),
                        np.arange(len(idx), dtype=np.int32), scales, fin,
                        {"grid": n, "points": idx, "configs": used})


def window_params(seed: int, base_rates, n_windows: int, sigma: float = 0.5,
                  cv_lo: float = 1.0, cv_hi: float = 4.0):
    """Per-window (rate, CV) of a non-stationary workload, a synthetic stand-in
    for windows fitted to a production trace: model m's log-rate follows a
    seeded random walk with N(0, sigma^2) steps, centred and clipped to
    +-2 around log(base_rates[m]); each window's CV is uniform in
    [cv_lo, cv_hi].  Draws: stream (seed, window-parameter, m), 2 * n_windows
    uniforms (normals by the inverse normal CDF).  Returns (rates, cvs), both
    [M][n_windows]."""
    from scipy.special import ndtri
    base = np.asarray(base_rates, dtype=np.float64)
    M = base.shape[0]
    rates = np.zeros((M, n_windows))
    cvs = np.zeros((M, n_windows))
    for m in range(M):
        u = gen.uniforms(gen.key(seed, gen.PURPOSE_WPARAM, m), 2 * n_windows)
        walk = np.cumsum(sigma * ndtri(u[:n_windows]))
        walk = np.clip(walk - walk.mean(), -2.0, 2.0)
        rates[m] = base[m] * np.exp(walk)
        cvs[m] = cv_lo + (cv_hi - cv_lo) * u[n_windows:]
    return rates, cvs


@dataclasses.dataclass
class RobustnessProblem:
    """One placement search on the assumed trace A, evaluated on trace B
    (Sec. 6.4: a placement chosen for one slice of traffic serves another)."""
    greedy: GreedyProblem       # trace A and the partitions to search
    t_b: np.ndarray
    model_b: np.ndarray
    windows: dict


def robustness(seed: int = 6, n_models: int = 16, n_devices: int = 16, device_mem_gb: int = 16,
               n_windows: int = 20, window: float = 60.0, total_rate: float = 64.0,
               exponent: float = 0.5, slo_scale: float = 5.0,
               partitions=((4, 4, 1), (4, 2, 2), (8, 8, 1), (16, 4, 4))) -> RobustnessProblem:
    """Models with d ~ U[0.1, 0.4] s and w ~ U[2, 6] GB; power-law (exponent
    0.5) base rates summing to total_rate; two non-stationary traces of
    n_windows windows of `window` seconds with independent window parameters
    (seeds seed and seed + 1000) -- trace A for the search, trace B for the
    evaluation."""
    M = n_models
    d = _uniform_range(seed, gen.PURPOSE_LATENCY, M, 0.1, 0.4)
    w = _weights_mib(seed, M, 2.0, 6.0)
    base = c4_rates(M, total_rate, exponent)
    ra, ca = window_params(seed, base, n_windows)
    rb, cb = window_params(seed + 1000, base, n_windows)
    ta, ma = gen.trace_windowed(seed, ra, ca, window)
    tb, mb = gen.trace_windowed(seed + 1000, rb, cb, window)
    cfgs = [(S, k) for _, S, k in partitions]
    L = stage_table(d, cfgs)
    parts = []
    for c, (size, S, k) in enumerate(partitions):
        G = n_devices // size
        parts.append({"group_cfg": np.full(G, c, np.int32),
                      "group_mem_mib": np.full(G, size * device_mem_gb * GIB_MIB, np.int64),
                      "label": f"{G}x(S={S},k={k})"})
    gp = GreedyProblem("robustness_a", ta, ma, d, w, np.array([S for S, _ in cfgs], np.int32),
                       np.array([k for _, k in cfgs], np.int32), L, parts, slo_scale,
                       {"devices": n_devices, "device_mem_mib": device_mem_gb * GIB_MIB})
    return RobustnessProblem(gp, tb, mb, {"a": (ra, ca), "b": (rb, cb), "window": window})


def batching(seed: int = 7, n_models: int = 32, n_groups: int = 16, group_size: int = 4,
             replicas: int = 4, n_placements: int = 256, duration: float = 600.0, rate: float = 4.0,
             cv: float = 4.0, scales=(1.0, 1.5, 2.0, 3.0, 5.0, 7.5, 10.0, 20.0)) -> Problem:
    """The shape of the batching experiment (Sec. 6.5): 32 instances of one
    model (151 ms single-device latency, 2.4 GB, like Table 1's BERT-1.3B),
    Gamma arrivals at 4 req/s per model with CV 4, ten minutes; 64 devices in
    16 groups of 4 at (S=4, k=1); each placement puts every model on
    `replicas` groups, the first of a seeded permutation of the groups (stream
    (seed, permute, p*M + m)); 8 SLO scales from 1 to 20."""
    M = n_models
    d = np.full(M, 0.151)
    w = np.full(M, int(2.4 * GIB_MIB), np.int64)
    cfgs = [(group_size, 1)]
    L = stage_table(d, cfgs)
    t, m = gen.trace(seed, [rate] * M, cv, duration)
    perms = gen.permutations(seed, gen.PURPOSE_PERMUTE, 0, n_placements * M, n_groups).reshape(
        n_placements, M, n_groups)
    hm = np.zeros((n_placements, M), np.uint64)
    for r in range(replicas):
        hm |= np.left_shift(np.uint64(1), perms[:, :, r].astype(np.uint64))
    return Problem("batching", t, m, d, w, np.array([group_size], np.int32), np.array([1], np.int32), L,
                   np.zeros((n_placements, n_groups), np.int32), hm, np.array(scales, np.float64),
                   np.array([0, 8 * 100 + 4], np.int32),
                   {"devices": n_groups * group_size})
