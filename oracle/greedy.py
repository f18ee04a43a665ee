"""Greedy placement search scored by the C oracle -- TEST INFRASTRUCTURE ONLY.

Alg. 1 of the paper (simulator-guided greedy model selection, Sec. 4.2) with
beam size 1 and with a beam of any size, the fast heuristic that Sec. 4.2
proposes for very large workloads, and the reduced form of Alg. 2 that
enumerates a given list of uniform group partitions and keeps the best Alg. 1
result.

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


def candidates(host_mask, used_mib, weight_mib, group_cfg, group_mem_mib, models=None):
    """Feasible (m, g) additions in lexicographic order (models: the ids that
    may be placed, all by default)."""
    M, G = len(weight_mib), len(group_cfg)
    out = []
    for m in range(M):
        if models is not None and m not in models:
            continue
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


def beam_selection(lib, t, model, d_single, weight_mib, cfg_stages, stage_lat, group_cfg,
                   group_mem_mib, slo_scale, beam, models=None, threads=None, max_steps=None):
    """Alg. 1 with beam size `beam` (Sec. 4.2).

    Each step expands every selection of the beam, in beam order, by every
    feasible (m, g) addition in (m, g) order, simulates each new selection,
    keeps the `beam` best as the next beam and compares the best of them with
    the best selection seen so far (replaced only by a strictly better one).
    Readings: a selection is its set of (model, group) replicas, and a new
    selection equal to one produced earlier in the same step is dropped (two
    beam entries can reach the same set); the top-k order is by served count,
    the earlier candidate first on ties; `models` restricts the placeable
    models (a model bucket of Alg. 2).
    Returns dict(best_mask, best_served, steps=[(parent, m, g, served, n_candidates)])."""
    group_cfg = np.asarray(group_cfg, dtype=np.int32)
    M, G = len(d_single), len(group_cfg)
    mset = None if models is None else set(int(m) for m in models)
    beam_sels = [(np.zeros(M, dtype=np.uint64), np.zeros(G, dtype=np.int64))]
    best_mask, best_served = beam_sels[0][0].copy(), 0
    steps = []
    nthreads = threads or min(8, os.cpu_count() or 1)
    with ThreadPoolExecutor(nthreads) as ex:
        while max_steps is None or len(steps) < max_steps:
            new, seen = [], set()
            for b, (mask, used) in enumerate(beam_sels):
                for m, g in candidates(mask, used, weight_mib, group_cfg, group_mem_mib, mset):
                    nm = mask.copy()
                    nm[m] = np.uint64(int(nm[m]) | (1 << g))
                    key = nm.tobytes()
                    if key in seen:
                        continue
                    seen.add(key)
                    nu = used.copy()
                    nu[g] += int(weight_mib[m])
                    new.append((b, m, g, nm, nu))
            if not new:
                break

            def score(c):
                return lib.simulate_job(t, model, d_single, cfg_stages, stage_lat, group_cfg, c[3],
                                        slo_scale)[0]

            scores = list(ex.map(score, new))
            order = sorted(range(len(new)), key=lambda i: (-scores[i], i))[:beam]
            beam_sels = [(new[i][3], new[i][4]) for i in order]
            i0 = order[0]
            steps.append((new[i0][0], new[i0][1], new[i0][2], scores[i0], len(new)))
            if scores[i0] > best_served:
                best_served = scores[i0]
                best_mask = new[i0][3].copy()
    return {"best_mask": best_mask, "best_served": best_served, "steps": steps}


def fast_selection(lib, t, model, d_single, weight_mib, cfg_stages, stage_lat, group_cfg,
                   group_mem_mib, slo_scale, models=None, max_steps=None):
    """The fast heuristic of Sec. 4.2: simulate the current selection once,
    then place the model with the most unserved requests on the available
    group with the lowest utilization; repeat until no replica fits.

    Readings: a model is a choice if some feasible (m, g) addition exists for
    it; its unserved requests are its requests in the trace minus the ones the
    simulation served (ties to the lowest model id); a group is available for
    it if the addition is feasible; a group's utilization is its busy time in
    the simulation (the slowest-stage latency of every request it served,
    summed in trace order; all groups see the same trace span, so busy time
    orders them as utilization does; ties to the lowest group); every
    simulated selection, the last one included, competes for the result, which
    is replaced only by a strictly better one (the empty selection serves 0).
    Returns dict(best_mask, best_served, steps=[(m, g, served_before)])."""
    group_cfg = np.asarray(group_cfg, dtype=np.int32)
    M, G = len(d_single), len(group_cfg)
    mset = None if models is None else set(int(m) for m in models)
    n_req = np.bincount(np.asarray(model, dtype=np.int64), minlength=M)
    mask = np.zeros(M, dtype=np.uint64)
    used = np.zeros(G, dtype=np.int64)
    best_mask, best_served = mask.copy(), 0
    steps = []
    while True:
        served, _, ms, busy = lib.simulate_job_stats(t, model, d_single, cfg_stages, stage_lat,
                                                     group_cfg, mask, slo_scale)
        if served > best_served:
            best_served = served
            best_mask = mask.copy()
        if max_steps is not None and len(steps) >= max_steps:
            break
        cands = candidates(mask, used, weight_mib, group_cfg, group_mem_mib, mset)
        if not cands:
            break
        mstar = None
        for m in sorted(set(m for m, _ in cands)):
            if mstar is None or n_req[m] - ms[m] > n_req[mstar] - ms[mstar]:
                mstar = m
        gstar = None
        for m, g in cands:
            if m == mstar and (gstar is None or busy[g] < busy[gstar]):
                gstar = g
        mask[mstar] = np.uint64(int(mask[mstar]) | (1 << gstar))
        used[gstar] += int(weight_mib[mstar])
        steps.append((mstar, gstar, served))
    return {"best_mask": best_mask, "best_served": best_served, "steps": steps}
