"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each pin is a function of an OracleLib (the committed oracle or a mutated copy)
that raises AssertionError when the simulator disagrees with something other
than itself: a closed form, a hand-derived fixture, an invariant, or the
independent event-driven brute force (oracle/brute.py).  test_oracle_pins.py
runs them on the committed oracle; test_oracle_mutants.py checks that every
planted mistake in a copy of the oracle fails at least one of them.

Exact pins use dyadic rationals (multiples of 2^-k with small numerators), so
every fp64 sum is exact and the expected values are exact too.
"""
from __future__ import annotations

import json
import math
import os
import struct
from fractions import Fraction

import numpy as np

from oracle import brute

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
INF = float("inf")
HASH_K = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1


def single_group(lat_stages, M=1):
    """One group with one configuration of S = len(lat_stages) stages hosting
    models 0..M-1, every model with the same stage latencies."""
    S = len(lat_stages)
    L = np.zeros((M, 1, S))
    L[:, 0, :] = lat_stages
    return dict(d_single=np.full(M, float(sum(lat_stages))), cfg_stages=np.array([S], np.int32),
                stage_lat=L, group_cfg=np.array([0], np.int32),
                host_mask=np.full(M, 1, np.uint64))


def run(lib, t, model, prob, sigma, finish=True):
    return lib.simulate_job(np.asarray(t, np.float64), np.asarray(model, np.int32),
                            prob["d_single"], prob["cfg_stages"], prob["stage_lat"],
                            prob["group_cfg"], prob["host_mask"], sigma, want_finish=finish)


def digest_from_finish(finish):
    """Digest recomputed from the per-request output alone."""
    h = 0
    w = 0
    fs = 0
    n = len(finish)
    for i, f in enumerate(finish):
        if f >= 0:
            w |= 1 << (i & 63)
            fs = (fs + struct.unpack("<Q", struct.pack("<d", float(f)))[0]) & MASK64
        if (i & 63) == 63 or i == n - 1:
            h = ((h ^ w) * HASH_K) & MASK64
            w = 0
    return h, fs


# ---------------------------------------------------------------- exact pins

def pin_dd1(lib):
    """D/D/1: arrivals every tau, deterministic service d, no drops.
    d <= tau: no waiting, finish_i = a_i + d.  d > tau: the server never idles
    after the first arrival, finish_i = a_0 + (i + 1) d."""
    tau = 0.5
    a = [tau * (i + 1) for i in range(64)]
    for d in (0.25, 0.5):
        s, _, fin = run(lib, a, [0] * 64, single_group([d]), INF)
        assert s == 64
        assert list(fin) == [x + d for x in a], ("d<=tau", d)
    for d in (0.75, 1.25):
        s, _, fin = run(lib, a, [0] * 64, single_group([d]), INF)
        assert s == 64
        assert list(fin) == [a[0] + (i + 1) * d for i in range(64)], ("d>tau", d)


def _dyadic_arrivals(rng, n, denom=64, max_gap=64):
    gaps = rng.integers(0, max_gap, size=n)
    return [Fraction(int(x), denom) for x in np.cumsum(gaps)]


def pin_lindley(lib):
    """Single-stage FCFS on arbitrary arrivals: the wait obeys Lindley's
    recursion w_{i+1} = max(0, w_i + d - (a_{i+1} - a_i)), finish = a + w + d."""
    rng = np.random.default_rng(5)
    for d in (Fraction(37, 64), Fraction(3, 4)):
        a = _dyadic_arrivals(rng, 300)
        w = Fraction(0)
        want = []
        for i in range(len(a)):
            if i > 0:
                w = max(Fraction(0), w + d - (a[i] - a[i - 1]))
            want.append(float(a[i] + w + d))
        s, _, fin = run(lib, [float(x) for x in a], [0] * len(a), single_group([float(d)]), INF)
        assert s == len(a)
        assert list(fin) == want


def pin_boundary(lib):
    """Deadline boundary (a finish exactly at the deadline is on time): d = 2 tau,
    SLO = d.  Request 0 finishes at d = its deadline, request 1 would finish at
    2d > tau + d, request 2 starts at 2 tau = d and finishes at 2 tau + d, its
    deadline: every other request is served."""
    tau, d = 0.25, 0.5
    n = 41
    a = [tau * i for i in range(n)]
    s, _, fin = run(lib, a, [0] * n, single_group([d]), 1.0)
    assert s == (n + 1) // 2
    for i in range(n):
        assert fin[i] == (a[i] + d if i % 2 == 0 else -1.0), i


def pin_pipeline_identity(lib):
    """Deterministic FCFS tandem (one group, S stages, no drops): the departure
    from the last stage is c_i + sum(d) - max(d), where c is the single server
    with service max(d) (max-plus lattice-path argument; it is why the paper's
    pipeline wait only involves the largest stage, Sec. 3.4)."""
    rng = np.random.default_rng(7)
    stages = [Fraction(3, 16), Fraction(5, 16), Fraction(1, 16), Fraction(2, 16)]
    dmax, dsum = max(stages), sum(stages)
    for trial in range(3):
        a = _dyadic_arrivals(rng, 250, denom=32, max_gap=24)
        c = None
        want = []
        for x in a:
            c = (x if c is None else max(x, c)) + dmax
            want.append(float(c + dsum - dmax))
        s, _, fin = run(lib, [float(x) for x in a], [0] * len(a),
                        single_group([float(x) for x in stages]), INF)
        assert s == len(a)
        assert list(fin) == want, trial


def pin_special_cases(lib):
    """Infinite SLO serves every hosted request; SLO 0 serves none (stage
    latencies are positive); requests of an unhosted model are misses (-2)."""
    rng = np.random.default_rng(3)
    n = 200
    a = np.sort(rng.integers(0, 500, n)) / 8.0
    m = rng.integers(0, 3, n).astype(np.int32)
    prob = single_group([0.25, 0.125], M=3)
    prob["host_mask"] = np.array([1, 1, 0], np.uint64)
    s, _, fin = run(lib, a, m, prob, INF)
    assert s == int(np.sum(m != 2))
    assert np.all(fin[m == 2] == -2.0) and np.all(fin[m != 2] > 0)
    s, dg, fin = run(lib, a, m, prob, 0.0)
    assert s == 0 and dg[1] == 0
    assert np.all(fin[m != 2] == -1.0) and np.all(fin[m == 2] == -2.0)


def pin_fig1(lib):
    """Fig. 1 / Sec. 1 worked example: 4 simultaneous requests of one model with
    latency y = 1.  Dedicated device: finishes 1, 2, 3, 4 (mean 2.5y, as printed).
    Two-stage pipeline without overhead (stages 0.5y): 1, 1.5, 2, 2.5 (1.75y)."""
    s, _, fin = run(lib, [0.0] * 4, [0] * 4, single_group([1.0]), INF)
    assert list(fin) == [1.0, 2.0, 3.0, 4.0] and np.mean(fin) == 2.5
    s, _, fin = run(lib, [0.0] * 4, [0] * 4, single_group([0.5, 0.5]), INF)
    assert list(fin) == [1.0, 1.5, 2.0, 2.5] and np.mean(fin) == 1.75


def pin_dispatch_fixture(lib):
    """Hand-derived fixture (tests/golden/dispatch_rule.json)."""
    with open(os.path.join(GOLDEN, "dispatch_rule.json")) as f:
        g = json.load(f)
    prob = dict(d_single=np.array(g["d_single"]), cfg_stages=np.array(g["cfg_stages"], np.int32),
                stage_lat=np.array(g["stage_lat"]), group_cfg=np.array(g["group_cfg"], np.int32),
                host_mask=np.array(g["host_mask"], np.uint64))
    req = g["requests"]
    s, dg, fin = run(lib, [r[0] for r in req], [r[1] for r in req], prob, g["slo_scale"])
    for i, r in enumerate(req):
        assert fin[i] == r[2], (i, fin[i], r)
    assert s == g["served"]
    assert dg == digest_from_finish(fin)


# ------------------------------------------------------ randomized structure

def random_case(rng, n=None, G=None, S=None, M=None, dyadic=False, ties=True):
    """A random tiny problem: G groups with their own configurations (S stages
    each), M models with random hosting sets (some unhosted), random stage
    latencies, a trace with repeated timestamps, and an SLO scale."""
    G = G or int(rng.integers(1, 4))
    Smax = S or int(rng.integers(1, 4))
    M = M or int(rng.integers(1, 4))
    n = n or int(rng.integers(1, 13))
    C = G
    cfg_stages = rng.integers(1, Smax + 1, C).astype(np.int32)
    if dyadic:
        L = rng.integers(1, 16, (M, C, Smax)) / 16.0
        gaps = rng.integers(0, 12, n) / 8.0
    else:
        L = rng.uniform(0.05, 1.0, (M, C, Smax))
        gaps = rng.exponential(0.4, n)
    if ties:
        gaps[rng.random(n) < 0.3] = 0.0
    t = np.cumsum(gaps)
    group_cfg = rng.permutation(C)[:G].astype(np.int32)
    host_mask = rng.integers(0, 1 << G, M).astype(np.uint64)
    d_single = L[:, 0, :].sum(axis=1) / rng.uniform(0.5, 2.0, M)
    model = rng.integers(0, M, n).astype(np.int32)
    sigma = float(rng.choice([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 5.0, INF]))
    prob = dict(d_single=d_single, cfg_stages=cfg_stages, stage_lat=L, group_cfg=group_cfg,
                host_mask=host_mask)
    return t, model, prob, sigma


def pin_brute_force(lib, cases=300):
    """Whole simulator vs the event-driven brute force with explicit queues,
    identical fp64 bits on tiny random problems (random configs per group,
    replication, unhosted models, equal timestamps, finite/zero/infinite SLO)."""
    rng = np.random.default_rng(2024)
    for k in range(cases):
        t, model, prob, sigma = random_case(rng, dyadic=(k % 2 == 0))
        s, dg, fin = run(lib, t, model, prob, sigma)
        bs, bfin = brute.simulate(t, model, prob["d_single"], prob["cfg_stages"], prob["stage_lat"],
                                  prob["group_cfg"], prob["host_mask"], sigma)
        assert s == bs, (k, s, bs)
        assert fin.tobytes() == bfin.tobytes(), (k, fin, bfin)
        assert dg == digest_from_finish(fin), k


def pin_invariants(lib, cases=60):
    """Structural invariants on larger random problems: served counts the
    non-negative outputs; unhosted requests are exactly the -2s; an accepted
    request finishes no earlier than arrival + its stage-latency sum of some
    hosting group and no later than its deadline; single-group, single-model
    runs finish in strictly increasing order, spaced by at least the largest
    stage (throughput bound 1/max stage, Sec. 3.4); digest matches the
    per-request output."""
    rng = np.random.default_rng(77)
    for k in range(cases):
        t, model, prob, sigma = random_case(rng, n=int(rng.integers(50, 400)), G=int(rng.integers(1, 6)),
                                            S=int(rng.integers(1, 5)), M=int(rng.integers(1, 5)))
        s, dg, fin = run(lib, t, model, prob, sigma)
        assert s == int(np.sum(fin >= 0))
        unhosted = prob["host_mask"][model] == 0
        assert np.array_equal(fin == -2.0, unhosted)
        L, gc, cs = prob["stage_lat"], prob["group_cfg"], prob["cfg_stages"]
        for i in np.nonzero(fin >= 0)[0]:
            m = model[i]
            lo = min(sum(L[m, gc[g], : cs[gc[g]]]) for g in range(len(gc))
                     if (int(prob["host_mask"][m]) >> g) & 1)
            assert fin[i] >= t[i] + lo * (1 - 1e-12)
            assert fin[i] <= t[i] + sigma * prob["d_single"][m]
        assert dg == digest_from_finish(fin)
    for k in range(20):
        S = int(rng.integers(1, 5))
        stages = list(rng.uniform(0.05, 0.5, S))
        n = 300
        t = np.cumsum(rng.exponential(0.2, n))
        s, _, fin = run(lib, t, np.zeros(n, np.int32), single_group(stages), float(rng.choice([2.0, 5.0, INF])))
        f = fin[fin >= 0]
        assert np.all(np.diff(f) >= max(stages) * (1 - 1e-12))


EXACT_PINS = [pin_dd1, pin_lindley, pin_boundary, pin_pipeline_identity, pin_special_cases,
              pin_fig1, pin_dispatch_fixture]
RANDOM_PINS = [pin_brute_force, pin_invariants]
ALL_PINS = EXACT_PINS + RANDOM_PINS
