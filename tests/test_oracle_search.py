"""Pins of the oracle's beam search (Alg. 1 with beam k, Sec. 4.2), of its
per-job statistics and of the fast heuristic (Sec. 4.2), each against an
independent formulation:
  - beam 1 is the already-pinned greedy search;
  - a beam wide enough to keep every selection finds the best of ALL feasible
    selections, enumerated exhaustively and scored by the event-driven brute
    force;
  - per-model served counts and per-group busy times are recomputed from the
    brute force's per-request outcome and chosen group;
  - every heuristic step is re-derived from those recomputed statistics."""
import itertools

import numpy as np
import pytest

from oracle import brute, greedy


def _tiny(rng, M_hi=4, G_hi=3, n_lo=3, n_hi=11):
    M = int(rng.integers(1, M_hi))
    G = int(rng.integers(1, G_hi))
    n = int(rng.integers(n_lo, n_hi))
    S = int(rng.integers(1, 3))
    C = G
    cfg_stages = rng.integers(1, S + 1, C).astype(np.int32)
    L = rng.uniform(0.1, 1.0, (M, C, S))
    t = np.cumsum(rng.exponential(0.3, n))
    model = rng.integers(0, M, n).astype(np.int32)
    d_single = L[:, 0, :].sum(axis=1)
    w = rng.integers(1, 5, M).astype(np.int64)
    group_cfg = rng.permutation(C)[:G].astype(np.int32)
    group_mem = rng.integers(2, 10, G).astype(np.int64)
    sigma = float(rng.choice([1.0, 2.0, 4.0]))
    return dict(t=t, model=model, d_single=d_single, w=w, cfg_stages=cfg_stages, L=L,
                group_cfg=group_cfg, group_mem=group_mem, sigma=sigma, M=M, G=G)


def test_beam_one_is_the_greedy_search(olib):
    rng = np.random.default_rng(21)
    for _ in range(25):
        p = _tiny(rng)
        args = (olib, p["t"], p["model"], p["d_single"], p["w"], p["cfg_stages"], p["L"], p["group_cfg"],
                p["group_mem"], p["sigma"])
        g = greedy.greedy_selection(*args)
        b = greedy.beam_selection(*args, beam=1)
        assert [(m, gg, s) for (_, m, gg, s, _) in b["steps"]] == g["steps"]
        assert b["best_served"] == g["best_served"]
        assert b["best_mask"].tolist() == g["best_mask"].tolist()


def test_wide_beam_finds_the_best_feasible_selection(olib):
    """With a beam that never drops a selection, step s holds every feasible
    selection of s replicas (memory feasibility is closed under removing a
    replica), so the search's best equals the exhaustive maximum."""
    rng = np.random.default_rng(22)
    checked = 0
    for _ in range(40):
        p = _tiny(rng, M_hi=4, G_hi=3, n_hi=9)
        M, G = p["M"], p["G"]
        pairs = [(m, g) for m in range(M) for g in range(G)]
        best = 0
        for r in range(1, len(pairs) + 1):
            for sub in itertools.combinations(pairs, r):
                used = [0] * G
                for m, g in sub:
                    used[g] += int(p["w"][m])
                if any(used[g] > p["group_mem"][g] for g in range(G)):
                    continue
                mask = np.zeros(M, np.uint64)
                for m, g in sub:
                    mask[m] = np.uint64(int(mask[m]) | (1 << g))
                s, _ = brute.simulate(p["t"], p["model"], p["d_single"], p["cfg_stages"], p["L"],
                                      p["group_cfg"], mask, p["sigma"])
                best = max(best, s)
        b = greedy.beam_selection(olib, p["t"], p["model"], p["d_single"], p["w"], p["cfg_stages"], p["L"],
                                  p["group_cfg"], p["group_mem"], p["sigma"], beam=10 ** 6)
        assert b["best_served"] == best
        # the best mask really serves that many
        s, _ = brute.simulate(p["t"], p["model"], p["d_single"], p["cfg_stages"], p["L"], p["group_cfg"],
                              b["best_mask"], p["sigma"])
        assert s == best
        checked += 1
    assert checked == 40


def test_beam_steps_keep_distinct_top_candidates(olib):
    """Every step's candidate count is the number of DISTINCT feasible
    extensions of the previous beam, and its best is their maximum."""
    rng = np.random.default_rng(23)
    for _ in range(15):
        p = _tiny(rng, M_hi=4, G_hi=4)
        for k in (2, 3):
            b = greedy.beam_selection(olib, p["t"], p["model"], p["d_single"], p["w"], p["cfg_stages"], p["L"],
                                      p["group_cfg"], p["group_mem"], p["sigma"], beam=k)
            beam = [np.zeros(p["M"], np.uint64)]
            for (parent, m, g, served, ncand) in b["steps"]:
                ext = {}
                for base in beam:
                    used = np.zeros(p["G"], np.int64)
                    for mm in range(p["M"]):
                        for gg in range(p["G"]):
                            if (int(base[mm]) >> gg) & 1:
                                used[gg] += p["w"][mm]
                    for mm in range(p["M"]):
                        for gg in range(p["G"]):
                            if (int(base[mm]) >> gg) & 1 or used[gg] + p["w"][mm] > p["group_mem"][gg]:
                                continue
                            nm = base.copy()
                            nm[mm] = np.uint64(int(nm[mm]) | (1 << gg))
                            ext.setdefault(nm.tobytes(), nm)
                assert ncand == len(ext)
                sc = []
                for key, nm in ext.items():
                    s, _ = brute.simulate(p["t"], p["model"], p["d_single"], p["cfg_stages"], p["L"],
                                          p["group_cfg"], nm, p["sigma"])
                    sc.append((s, key, nm))
                assert served == max(s for s, _, _ in sc)
                # next beam: the k best (ties in production order, which the dict keeps)
                order = sorted(range(len(sc)), key=lambda i: (-sc[i][0], i))[:k]
                beam = [sc[i][2] for i in order]


def _brute_stats(p, mask):
    s, fin, grp = brute.simulate(p["t"], p["model"], p["d_single"], p["cfg_stages"], p["L"], p["group_cfg"],
                                 mask, p["sigma"], return_groups=True)
    ms = np.zeros(p["M"], np.int64)
    busy = np.zeros(len(p["group_cfg"]), np.float64)
    for i in range(len(fin)):
        if fin[i] >= 0:
            m, g = int(p["model"][i]), int(grp[i])
            ms[m] += 1
            c = int(p["group_cfg"][g])
            S = int(p["cfg_stages"][c])
            busy[g] += max(float(p["L"][m, c, s]) for s in range(S))
    return s, ms, busy


def test_stats_match_bruteforce(olib):
    rng = np.random.default_rng(24)
    for _ in range(60):
        p = _tiny(rng, M_hi=5, G_hi=4, n_hi=14)
        M, G = p["M"], p["G"]
        mask = rng.integers(0, 1 << G, M).astype(np.uint64)
        s, dg, ms, busy = olib.simulate_job_stats(p["t"], p["model"], p["d_single"], p["cfg_stages"], p["L"],
                                                  p["group_cfg"], mask, p["sigma"])
        s2, ms2, busy2 = _brute_stats(p, mask)
        assert s == s2 == int(ms.sum())
        assert ms.tolist() == ms2.tolist()
        assert busy.tobytes() == busy2.tobytes()
        s3, dg3, _ = olib.simulate_job(p["t"], p["model"], p["d_single"], p["cfg_stages"], p["L"],
                                       p["group_cfg"], mask, p["sigma"])
        assert (s3, dg3) == (s, dg)


def test_fast_heuristic_steps_follow_the_rule(olib):
    rng = np.random.default_rng(25)
    for _ in range(30):
        p = _tiny(rng, M_hi=5, G_hi=4, n_hi=14)
        M, G = p["M"], p["G"]
        r = greedy.fast_selection(olib, p["t"], p["model"], p["d_single"], p["w"], p["cfg_stages"], p["L"],
                                  p["group_cfg"], p["group_mem"], p["sigma"])
        n_req = np.bincount(p["model"], minlength=M)
        mask = np.zeros(M, np.uint64)
        used = np.zeros(G, np.int64)
        seen = []
        for (m, g, served) in r["steps"]:
            s, ms, busy = _brute_stats(p, mask)
            assert s == served
            seen.append(s)
            feas = [(mm, gg) for mm in range(M) for gg in range(G)
                    if not (int(mask[mm]) >> gg) & 1 and used[gg] + p["w"][mm] <= p["group_mem"][gg]]
            placeable = sorted(set(mm for mm, _ in feas))
            un = {mm: int(n_req[mm] - ms[mm]) for mm in placeable}
            assert un[m] == max(un.values()) and m == min(mm for mm in placeable if un[mm] == un[m])
            gs = [gg for mm, gg in feas if mm == m]
            assert g in gs
            assert busy[g] == min(busy[gg] for gg in gs) and g == min(gg for gg in gs if busy[gg] == busy[g])
            mask[m] = np.uint64(int(mask[m]) | (1 << g))
            used[g] += p["w"][m]
        # nothing fits at the end; the final selection is scored too
        assert not [(mm, gg) for mm in range(M) for gg in range(G)
                    if not (int(mask[mm]) >> gg) & 1 and used[gg] + p["w"][mm] <= p["group_mem"][gg]]
        s_final, _, _ = _brute_stats(p, mask)
        seen.append(s_final)
        assert r["best_served"] == max([0] + seen)
        s_best, _, _ = _brute_stats(p, r["best_mask"])
        assert s_best == r["best_served"]


@pytest.mark.parametrize("k", [1, 3])
def test_model_subset_is_respected(olib, k):
    rng = np.random.default_rng(26 + k)
    p = _tiny(rng, M_hi=5, G_hi=4)
    keep = {0} if p["M"] == 1 else {0, p["M"] - 1}
    for fn in ("beam", "fast"):
        if fn == "beam":
            r = greedy.beam_selection(olib, p["t"], p["model"], p["d_single"], p["w"], p["cfg_stages"], p["L"],
                                      p["group_cfg"], p["group_mem"], p["sigma"], beam=k, models=keep)
            placed = {m for (_, m, _, _, _) in r["steps"]}
        else:
            r = greedy.fast_selection(olib, p["t"], p["model"], p["d_single"], p["w"], p["cfg_stages"], p["L"],
                                      p["group_cfg"], p["group_mem"], p["sigma"], models=keep)
            placed = {m for (m, _, _) in r["steps"]}
        assert placed <= keep
        for m in range(p["M"]):
            if m not in keep:
                assert int(r["best_mask"][m]) == 0
