"""Pins of the oracle's Alg. 2 (Sec. 4.2): its enumerations against closed
forms and an independent brute-force enumeration, and the whole search
against what Alg. 2 promises -- the concatenated placement, simulated as ONE
placement by the event-driven brute force, serves exactly the sum of its
buckets, and a one-bucket, one-configuration search is Alg. 1."""
import itertools
from math import comb

import numpy as np
import pytest

from oracle import alg2, brute, greedy


def test_bucket_cuts_closed_forms():
    rng = np.random.default_rng(31)
    for M in range(1, 9):
        d = rng.uniform(0.05, 0.8, M)
        for K in range(1, 5):
            _, cuts = alg2.model_bucket_cuts(d, K, float("inf"))
            assert len(cuts) == sum(comb(M - 1, k - 1) for k in range(1, min(K, M) + 1))
            _, cuts0 = alg2.model_bucket_cuts(d, K, 0.0)  # distinct latencies: singletons only
            assert cuts0 == ([list(range(M))] if M <= K else [])


def test_bucket_cuts_match_bruteforce():
    """Every subset of cut points of the sorted list, filtered by run count and
    latency span, equals the enumeration (same order: by run count, then
    lexicographic starts)."""
    rng = np.random.default_rng(32)
    for _ in range(40):
        M = int(rng.integers(1, 8))
        d = np.round(rng.uniform(0.0, 1.0, M), 2)  # ties happen
        K = int(rng.integers(1, 5))
        th = float(rng.choice([0.0, 0.1, 0.3, 0.6, 2.0]))
        order, cuts = alg2.model_bucket_cuts(d, K, th)
        assert order == sorted(range(M), key=lambda m: (d[m], m))
        want = []
        for mask in range(1 << max(M - 1, 0)):
            starts = [0] + [i + 1 for i in range(M - 1) if (mask >> i) & 1]
            if len(starts) > K:
                continue
            ends = starts[1:] + [M]
            if all(d[order[e - 1]] - d[order[s]] <= th for s, e in zip(starts, ends)):
                want.append(starts)
        want.sort(key=lambda st: (len(st), st))
        assert cuts == want


def test_device_splits():
    for units in range(1, 10):
        for k in range(1, 5):
            sp = alg2.device_splits(units, k)
            assert len(sp) == (comb(units - 1, k - 1) if units >= k else 0)
            assert sp == sorted(sp) and len(set(map(tuple, sp))) == len(sp)
            assert all(sum(x) == units and min(x) >= 1 and len(x) == k for x in sp)


def test_bucket_options():
    # configurations: sizes 1, 2, 2, 4 with pipeline depths 1, 2, 1, 4
    cfg_devices = np.array([1, 2, 2, 4], np.int32)
    cfg_stages = np.array([1, 2, 1, 4], np.int32)
    opts = {c: (g.tolist(), m.tolist()) for c, g, m in alg2.bucket_options(7, cfg_devices, cfg_stages, 100)}
    assert opts[0] == ([0] * 7, [100] * 7)
    assert opts[1] == ([1, 1, 1, 0], [200, 200, 200, 100])
    assert opts[2] == ([2, 2, 2, 0], [200, 200, 200, 100])
    # 7 = 4 + 3: no configuration has 3 devices
    assert 3 not in opts
    opts6 = {c: g.tolist() for c, g, _ in alg2.bucket_options(6, cfg_devices, cfg_stages, 1)}
    assert opts6[3] == [3, 1]  # last group of 2: the deepest pipeline (S=2) not deeper than 4
    opts5 = {c: g.tolist() for c, g, _ in alg2.bucket_options(2, cfg_devices, cfg_stages, 1)}
    assert 3 not in opts5  # 4 devices do not fit in 2


def test_bucket_options_remainder_not_deeper_than_the_bucket_configuration():
    """Hand-derived: the last group of a bucket takes a configuration of the
    remaining device count whose pipeline is not deeper than the equal groups'
    one.  Sizes 1, 2, 2, 4, 4 with depths 1, 2, 1, 4, 1."""
    cfg_devices = np.array([1, 2, 2, 4, 4], np.int32)
    cfg_stages = np.array([1, 2, 1, 4, 1], np.int32)
    opts = {c: g.tolist() for c, g, _ in alg2.bucket_options(6, cfg_devices, cfg_stages, 1)}
    assert opts[4] == [4, 2]  # 4 + 2 at depth 1: the 2-device group is (S=1, k=2), not (S=2, k=1)
    assert opts[3] == [3, 1]  # 4 + 2 at depth 4: the deepest 2-device pipeline, S=2
    # depth 1 and no 2-device configuration of depth <= 1: skipped
    opts_b = {c: g.tolist() for c, g, _ in alg2.bucket_options(6, np.array([2, 4], np.int32),
                                                                np.array([2, 1], np.int32), 1)}
    assert 1 not in opts_b and opts_b[0] == [0, 0, 0]


def _balance_instance():
    """Two models of latency 0.5 s with three requests each: every bucket's
    load is 1.5 s of work divided by its devices (exact in binary)."""
    t = np.array([0.0, 0.0, 1.0, 1.0, 2.0, 2.0])
    model = np.array([0, 1, 0, 1, 0, 1], np.int32)
    d = np.array([0.5, 0.5])
    cfg_stages = np.array([1], np.int32)
    L = np.full((2, 1, 1), 0.5)
    return t, model, d, cfg_stages, L


@pytest.mark.parametrize("ratio,kept", [(1.0, 2), (2.0, 2), (2.999, 2), (3.0, 4), (float("inf"), 4)])
def test_balance_rule_keeps_the_splits_of_similar_load(olib, ratio, kept):
    """Sec. 4.2 drops device splits whose buckets would work at very different
    paces.  4 devices, buckets {0}, {1} (threshold 0 keeps equal latencies
    together or apart): the one-bucket cut has one split (always kept), the
    two-bucket cut has (1,3), (2,2), (3,1) with per-device loads 1.5 vs 0.5,
    0.75 vs 0.75 and 0.5 vs 1.5: largest/smallest 3, 1, 3.  Kept iff that
    ratio <= the balance ratio."""
    t, model, d, cs, L = _balance_instance()
    r = alg2.placement_search(olib, t, model, d, np.array([1, 1], np.int64), cs, L, np.array([1], np.int32), 4,
                              1, 4, 0.0, ratio, 2, 1, 10.0)
    assert r["n_bucket_configs"] == 2
    assert r["n_device_splits"] == 4
    assert r["n_kept_splits"] == kept
    if ratio < 3.0 and len(r["buckets"]) == 2:
        assert [b["devices"] for b in r["buckets"]] == [2, 2]


def _instance(seed, M, n_dev, duration=8.0):
    rng = np.random.default_rng(seed)
    d = rng.uniform(0.1, 0.5, M)
    cfgs = [(1, 1), (2, 1), (1, 2), (2, 2)]  # (S, k)
    cfg_stages = np.array([S for S, _ in cfgs], np.int32)
    cfg_devices = np.array([S * k for S, k in cfgs], np.int32)
    L = np.zeros((M, len(cfgs), 2))
    for c, (S, k) in enumerate(cfgs):
        for m in range(M):
            L[m, c, :S] = d[m] * (1 + 0.05 * (S - 1)) * (1 + 0.1 * (k - 1)) / (S * k)
    rate = rng.uniform(0.5, 2.0, M)
    ts, ms = [], []
    for m in range(M):
        x = np.cumsum(rng.exponential(1.0 / rate[m], 64))
        x = x[x < duration]
        ts.append(x)
        ms.append(np.full(len(x), m, np.int32))
    t = np.concatenate(ts)
    model = np.concatenate(ms)
    o = np.lexsort((model, t))
    w = rng.integers(1, 4, M).astype(np.int64)
    return dict(t=t[o], model=model[o], d_single=d, w=w, cfg_stages=cfg_stages, L=L, cfg_devices=cfg_devices,
                n_devices=n_dev, mem=4)


@pytest.mark.parametrize("beam", [1, 2, 0])
def test_concatenated_placement_serves_the_bucket_sum(olib, beam):
    for seed in range(3):
        p = _instance(40 + seed, M=4, n_dev=4)
        r = alg2.placement_search(olib, p["t"], p["model"], p["d_single"], p["w"], p["cfg_stages"], p["L"],
                                  p["cfg_devices"], p["n_devices"], 1, p["mem"], 0.25, 4.0, 3, beam, 3.0)
        assert r["n_kept_splits"] <= r["n_device_splits"]
        gcfg, masks = [], np.zeros(len(p["d_single"]), np.uint64)
        for b in r["buckets"]:
            off = len(gcfg)
            gcfg += b["group_cfg"].tolist()
            for m in range(len(masks)):
                masks[m] = np.uint64(int(masks[m]) | (int(b["mask"][m]) << off))
                if int(b["mask"][m]):
                    assert m in b["models"]
        if not gcfg:
            assert r["served"] == 0
            continue
        assert sum(b["devices"] for b in r["buckets"]) == p["n_devices"]
        s, _ = brute.simulate(p["t"], p["model"], p["d_single"], p["cfg_stages"], p["L"],
                              np.array(gcfg, np.int32), masks, 3.0)
        assert s == r["served"] == sum(b["served"] for b in r["buckets"])


def test_one_bucket_one_config_is_alg1(olib):
    p = _instance(50, M=4, n_dev=4)
    cd = p["cfg_devices"][:1]
    cs = p["cfg_stages"][:1]
    L = p["L"][:, :1, :1]
    r = alg2.placement_search(olib, p["t"], p["model"], p["d_single"], p["w"], cs, L, cd, 4, 1, p["mem"],
                              10.0, float("inf"), 1, 1, 3.0)
    g = greedy.greedy_selection(olib, p["t"], p["model"], p["d_single"], p["w"], cs, L,
                                np.zeros(4, np.int32), np.full(4, p["mem"], np.int64), 3.0)
    assert r["served"] == g["best_served"]
    if r["buckets"]:
        assert r["buckets"][0]["mask"].tolist() == g["best_mask"].tolist()


def test_search_keeps_the_best_split(olib):
    """Exhaustive re-scoring: every kept (cut, split) pair's bucket optima,
    recomputed independently, never beat the returned placement."""
    p = _instance(60, M=3, n_dev=4)
    args = (olib, p["t"], p["model"], p["d_single"], p["w"], p["cfg_stages"], p["L"], p["cfg_devices"], 4, 1,
            p["mem"])
    r = alg2.placement_search(*args, 1.0, float("inf"), 3, 1, 3.0)
    order, cuts = alg2.model_bucket_cuts(p["d_single"], 3, 1.0)
    best = 0
    for starts in cuts:
        k = len(starts)
        buckets = [order[starts[b]:(starts[b + 1] if b + 1 < k else 3)] for b in range(k)]
        for split in alg2.device_splits(4, k):
            tot = 0
            for b in range(k):
                top = 0
                for c, gc, gm in alg2.bucket_options(split[b], p["cfg_devices"], p["cfg_stages"], p["mem"]):
                    g = greedy.greedy_selection(olib, p["t"], p["model"], p["d_single"],
                                                np.where(np.isin(np.arange(3), buckets[b]), p["w"], 10 ** 9),
                                                p["cfg_stages"], p["L"], gc, gm, 3.0)
                    top = max(top, g["best_served"])
                tot += top
            best = max(best, tot)
    assert r["served"] == best
