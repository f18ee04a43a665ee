"""Pins of the oracle's greedy placement search (Alg. 1 with beam 1, reduced
Alg. 2).  The step logic is checked against a second, deliberately plain
implementation that re-scores every candidate with the event-driven brute
force, and against invariants of Alg. 1 (Sec. 4.2)."""
import numpy as np
import pytest

from oracle import brute, greedy


def plain_greedy(t, model, d_single, w, cfg_stages, L, group_cfg, group_mem, sigma):
    """Alg. 1 (beam 1) written out directly, every candidate scored by the
    brute-force simulator."""
    M, G = len(d_single), len(group_cfg)
    hosted = [[False] * G for _ in range(M)]
    used = [0] * G
    best = 0
    best_sel = None
    steps = []
    while True:
        cand = []
        for m in range(M):
            for g in range(G):
                if group_cfg[g] >= 0 and not hosted[m][g] and used[g] + w[m] <= group_mem[g]:
                    cand.append((m, g))
        if not cand:
            break
        scores = []
        for m, g in cand:
            mask = [sum(1 << gg for gg in range(G) if hosted[mm][gg] or (mm == m and gg == g))
                    for mm in range(M)]
            s, _ = brute.simulate(t, model, d_single, cfg_stages, L, group_cfg, np.array(mask, np.uint64), sigma)
            scores.append(s)
        top = max(scores)
        i = scores.index(top)  # first (lowest index) maximum
        m, g = cand[i]
        hosted[m][g] = True
        used[g] += w[m]
        steps.append((m, g, top))
        if top > best:
            best = top
            best_sel = [row[:] for row in hosted]
    return steps, best, best_sel


def test_greedy_matches_plain_bruteforce_greedy(olib):
    rng = np.random.default_rng(11)
    for case in range(25):
        M = int(rng.integers(1, 4))
        G = int(rng.integers(1, 4))
        n = int(rng.integers(3, 11))
        S = int(rng.integers(1, 3))
        C = G
        cfg_stages = rng.integers(1, S + 1, C).astype(np.int32)
        L = rng.uniform(0.1, 1.0, (M, C, S))
        t = np.cumsum(rng.exponential(0.3, n))
        model = rng.integers(0, M, n).astype(np.int32)
        d_single = L[:, 0, :].sum(axis=1)
        w = rng.integers(1, 5, M).astype(np.int64)
        group_cfg = rng.permutation(C)[:G].astype(np.int32)
        group_mem = rng.integers(1, 9, G).astype(np.int64)
        sigma = float(rng.choice([1.0, 2.0, 4.0]))
        r = greedy.greedy_selection(olib, t, model, d_single, w, cfg_stages, L, group_cfg, group_mem,
                                    sigma, threads=2)
        steps, best, best_sel = plain_greedy(t, model, d_single, w, cfg_stages, L, group_cfg, group_mem, sigma)
        assert [tuple(s) for s in r["steps"]] == steps, case
        assert r["best_served"] == best, case
        if best_sel is not None:
            want = [sum(1 << g for g in range(G) if best_sel[m][g]) for m in range(M)]
            assert [int(x) for x in r["best_mask"]] == want, case


def test_greedy_invariants_on_tiny_workload(olib):
    """Memory constraint respected at every step, loop ends only when nothing
    fits, best_served is the best step score, each step's chosen score is the
    maximum over all candidates of that step."""
    from paper_2302_11665_amd.workload import problems
    pb = problems.c2_greedy_step(duration=60.0)
    G = 4
    gcfg = np.zeros(G, np.int32)
    mem = np.full(G, 16 * 1024, np.int64)  # tighter than the workload's 64 GB groups
    r = greedy.greedy_selection(olib, pb.t, pb.model, pb.d_single, pb.weight_mib, pb.cfg_stages,
                                pb.stage_lat, gcfg, mem, 3.0)
    used = np.zeros(G, np.int64)
    hm = np.zeros(len(pb.d_single), np.uint64)
    for m, g, s in r["steps"]:
        used[g] += pb.weight_mib[m]
        assert used[g] <= mem[g]
        assert not (int(hm[m]) >> g) & 1
        hm[m] = np.uint64(int(hm[m]) | (1 << g))
    assert greedy.candidates(hm, used, pb.weight_mib, gcfg, mem) == []
    assert r["best_served"] == max(s for _, _, s in r["steps"])
    # re-score the first step exhaustively
    m0, g0, s0 = r["steps"][0]
    scores = []
    for m in range(len(pb.d_single)):
        for g in range(G):
            mask = np.zeros(len(pb.d_single), np.uint64)
            mask[m] = np.uint64(1 << g)
            scores.append(olib.simulate_job(pb.t, pb.model, pb.d_single, pb.cfg_stages, pb.stage_lat,
                                            gcfg, mask, 3.0)[0])
    assert s0 == max(scores) and (m0 * G + g0) == scores.index(max(scores))


def test_reduced_partition_search_picks_strict_best(olib):
    from paper_2302_11665_amd.workload import problems
    gp = problems.c3_greedy(duration=20.0, n_models=4, n_devices=8, partitions=[(2, 2, 1), (4, 4, 1), (4, 2, 2)])
    best, results = greedy.reduced_partition_search(olib, gp.t, gp.model, gp.d_single, gp.weight_mib,
                                                    gp.cfg_stages, gp.stage_lat, gp.partitions, gp.slo_scale)
    top = max(r["best_served"] for r in results)
    assert best["best_served"] == top
    assert best["partition"] == min(i for i, r in enumerate(results) if r["best_served"] == top)
