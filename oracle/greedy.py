"""Greedy placement search scored by the C oracle -- TEST INFRASTRUCTURE ONLY.

Alg. 1 of the paper (simulator-guided greedy model selection, Sec. 4.2) with
beam size 1, and the reduced form of Alg. 2 that enumerates a given list of
uniform group partitions and keeps the best Alg. 1 result.

Readings (listed in the design notes):
  - a candidate is a (model m, group g) pair with g not already hosting m;
    candidates are taken in (m, g) lexicographic order;
  - memory (Sec. 4.2 "in memory constraint"): every device of a group holds
    1/(S*k) of each hosted model, so a group fits iff the sum of hosted model
    weights is <= the group's total memory (per-device memory * S * k), in
    integer MiB;
  - each candidate is scored by its served-request count (attainment times the
    fixed trace length, an integer, so no rounding enters the comparison);
    the best candidate is the one with the most served requests, the lowest
    candidate index on ties;
  - the loop commits that candidate and repeats until no candidate fits; the
    returned selection is the best one seen, replaced only by a strictly
    better one (the empty selection scores 0).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np


def candidates(host_mask, used_mib, weight_mib, group_cfg, group_mem_mib):
    """Feasible (m, g) additions in lexicographic order."""
    M, G = len(weight_mib), len(group_cfg)
    out = []
    for m in range(M):
        for g in range(G):
            if group_cfg[g] < 0:
                continue
            if (int(host_mask[m]) >> g) & 1:
                continue
            if int(used_mib[g]) + int(weight_mib[m]) <= int(group_mem_mib[g]):
                out.append((m, g))
    return out


def greedy_selection(lib, t, model, d_single, weight_mib, cfg_stages, stage_lat, group_cfg,
                     group_mem_mib, slo_scale, threads=None, max_steps=None, on_step=None):
    """Alg. 1 with beam 1.  Returns dict(best_mask, best_served, steps=[(m, g, served)])."""
    group_cfg = np.asarray(group_cfg, dtype=np.int32)
    M = len(d_single)
    G = len(group_cfg)
    host_mask = np.zeros(M, dtype=np.uint64)
    used = np.zeros(G, dtype=np.int64)
    best_mask = host_mask.copy()
    best_served = 0
    steps = []
    nthreads = threads or min(8, os.cpu_count() or 1)
    with ThreadPoolExecutor(nthreads) as ex:
        while max_steps is None or len(steps) < max_steps:
            cands = candidates(host_mask, used, weight_mib, group_cfg, group_mem_mib)
            if not cands:
                break

            def score(mg):
                m, g = mg
                hm = host_mask.copy()
                hm[m] = np.uint64(int(hm[m]) | (1 << g))
                s, _, _ = lib.simulate_job(t, model, d_single, cfg_stages, stage_lat,
                                           group_cfg, hm, slo_scale)
                return s

            scores = list(ex.map(score, cands))
            bi = 0
            for i in range(1, len(scores)):
                if scores[i] > scores[bi]:
                    bi = i
            m, g = cands[bi]
            host_mask[m] = np.uint64(int(host_mask[m]) | (1 << g))
            used[g] += int(weight_mib[m])
            steps.append((m, g, scores[bi]))
            if on_step is not None:
                on_step(len(steps), m, g, scores[bi], len(cands))
            if scores[bi] > best_served:
                best_served = scores[bi]
                best_mask = host_mask.copy()
    return {"best_mask": best_mask, "best_served": best_served, "steps": steps}


def reduced_partition_search(lib, t, model, d_single, weight_mib, cfg_stages, stage_lat,
                             partitions, slo_scale, threads=None, on_step=None):
    """Reduced Alg. 2: run Alg. 1 on every partition (each a dict with
    group_cfg[G] and group_mem_mib[G]) and keep the strictly best result
    (first partition on ties)."""
    best = None
    results = []
    for pi, part in enumerate(partitions):
        cb = (lambda *a, _pi=pi: on_step(_pi, *a)) if on_step else None
        r = greedy_selection(lib, t, model, d_single, weight_mib, cfg_stages, stage_lat,
                             part["group_cfg"], part["group_mem_mib"], slo_scale,
                             threads=threads, on_step=cb)
        r["partition"] = pi
        results.append(r)
        if best is None or r["best_served"] > best["best_served"]:
            best = r
    return best, results
