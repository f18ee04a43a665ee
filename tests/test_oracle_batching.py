"""Pins of the oracle's dynamic-batching simulation (Sec. 6.5):
  - with batches of one and a single group it is the FCFS single-server
    system, so it equals the already-pinned unbatched simulation bit for bit;
  - a burst of simultaneous requests has closed-form finish times for any
    maximum batch size and latency slope;
  - an event-driven formulation (explicit stage servers replayed per group,
    a global clock over arrival and idle events) gives identical bits;
  - invariants: served requests meet their deadlines, batches respect the
    maximum size and share one finish time and model, the digest is the
    order-free sum stated in the definition."""
import numpy as np
import pytest

from oracle import brute

INF = float("inf")


def _mix64(z):
    M64 = (1 << 64) - 1
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def _case(rng, G=None, M=None, n=None, S=None, dyadic=False):
    G = G or int(rng.integers(1, 4))
    M = M or int(rng.integers(1, 4))
    n = n or int(rng.integers(1, 14))
    Smax = S or int(rng.integers(1, 3))
    C = G
    cfg_stages = rng.integers(1, Smax + 1, C).astype(np.int32)
    if dyadic:
        L = rng.integers(1, 16, (M, C, Smax)) / 16.0
        gaps = rng.integers(0, 8, n) / 8.0
    else:
        L = rng.uniform(0.05, 1.0, (M, C, Smax))
        gaps = rng.exponential(0.3, n)
    gaps[rng.random(n) < 0.3] = 0.0
    t = np.cumsum(gaps)
    group_cfg = rng.permutation(C)[:G].astype(np.int32)
    host_mask = rng.integers(0, 1 << G, M).astype(np.uint64)
    d_single = L[:, 0, :].sum(axis=1) / rng.uniform(0.5, 2.0, M)
    model = rng.integers(0, M, n).astype(np.int32)
    sigma = float(rng.choice([0.5, 1.0, 2.0, 3.0, 5.0, INF]))
    return t, model, d_single, cfg_stages, L, group_cfg, host_mask, sigma


def test_batch_one_single_group_is_the_unbatched_simulation(olib):
    rng = np.random.default_rng(71)
    for k in range(200):
        t, model, d, cs, L, gc, hm, sigma = _case(rng, G=1, dyadic=k % 2 == 0)
        hm = np.where(rng.random(len(hm)) < 0.8, np.uint64(1), np.uint64(0)).astype(np.uint64)
        s, dg, fin = olib.simulate_job(t, model, d, cs, L, gc, hm, sigma, want_finish=True)
        sb, dgb, finb, bat = olib.simulate_job_batched(t, model, d, cs, L, gc, hm, sigma, 1, 0.7)
        assert sb == s and finb.tobytes() == fin.tobytes(), k
        assert dgb[1] == dg[1]
        assert set(bat.tolist()) <= {0, 1}


@pytest.mark.parametrize("B,beta", [(1, 1.0), (2, 1.0), (3, 0.5), (4, 0.25), (8, 0.0), (100, 0.5)])
def test_burst_closed_form(olib, B, beta):
    """n simultaneous requests, one single-stage group, latency 1, no SLO
    limit: the first runs alone on [0, 1]; the others wait and go in batches of
    min(B, rest), each lasting 1 + beta (b - 1)."""
    n = 11
    t = np.zeros(n)
    model = np.zeros(n, np.int32)
    L = np.ones((1, 1, 1))
    s, dg, fin, bat = olib.simulate_job_batched(t, model, np.ones(1), np.array([1], np.int32), L,
                                                np.array([0], np.int32), np.array([1], np.uint64), INF, B, beta)
    want, clock, rest, sizes = [1.0], 1.0, n - 1, [1]
    while rest > 0:
        b = min(B, rest)
        clock = clock + 1.0 * (1.0 + beta * (b - 1))
        want += [clock] * b
        sizes += [b] * b
        rest -= b
    assert s == n
    assert fin.tolist() == want
    assert bat.tolist() == sizes


def test_burst_with_tight_slo_drops_what_cannot_finish(olib):
    """Same burst, SLO 3 x latency, batches of up to 4 at slope 1: the first
    finishes at 1, a batch of 2 fits before 3 (finish 3), the rest expire."""
    n = 6
    s, _, fin, bat = olib.simulate_job_batched(np.zeros(n), np.zeros(n, np.int32), np.ones(1),
                                               np.array([1], np.int32), np.ones((1, 1, 1)),
                                               np.array([0], np.int32), np.array([1], np.uint64), 3.0, 4, 1.0)
    assert fin.tolist() == [1.0, 3.0, 3.0, -1.0, -1.0, -1.0]
    assert s == 3 and bat.tolist() == [1, 2, 2, 0, 0, 0]


def test_matches_event_driven_bruteforce(olib):
    rng = np.random.default_rng(72)
    for k in range(300):
        t, model, d, cs, L, gc, hm, sigma = _case(rng, dyadic=k % 2 == 0)
        B = int(rng.choice([1, 2, 3, 8]))
        beta = float(rng.choice([0.0, 0.25, 0.5, 1.0]))
        s, dg, fin, bat = olib.simulate_job_batched(t, model, d, cs, L, gc, hm, sigma, B, beta)
        bs, bfin, bbat, bdg = brute.simulate_batched(t, model, d, cs, L, gc, hm, sigma, B, beta)
        assert s == bs, k
        assert fin.tobytes() == bfin.tobytes(), (k, fin, bfin)
        assert bat.tolist() == bbat.tolist(), k
        assert dg == bdg, k


def test_invariants(olib):
    rng = np.random.default_rng(73)
    for k in range(60):
        t, model, d, cs, L, gc, hm, sigma = _case(rng, G=int(rng.integers(1, 6)), M=int(rng.integers(1, 6)),
                                                   n=int(rng.integers(50, 400)), S=int(rng.integers(1, 4)))
        B = int(rng.choice([1, 2, 4, 16]))
        beta = float(rng.choice([0.0, 0.5, 1.0]))
        s, (h, fs), fin, bat = olib.simulate_job_batched(t, model, d, cs, L, gc, hm, sigma, B, beta)
        served = bat > 0
        assert s == int(served.sum())
        assert ((fin >= 0) == served).all()
        unhosted = np.array([int(hm[m]) == 0 for m in model])
        assert (fin[unhosted] == -2.0).all() and not served[unhosted].any()
        dl = t + sigma * d[model]
        assert (fin[served] <= dl[served]).all()
        assert (fin[served] >= t[served]).all()
        assert bat.max(initial=0) <= B
        # requests of one batch share finish time and model; a batch of b has b members
        groups = {}
        for i in np.nonzero(served)[0]:
            groups.setdefault((float(fin[i]), int(model[i]), int(bat[i])), []).append(int(i))
        for (f, m, b), members in groups.items():
            assert len(members) % b == 0
        assert h == sum(_mix64(int(i)) for i in np.nonzero(served)[0]) % (1 << 64)
        assert fs == int(fin[served].view(np.uint64).astype(object).sum()) % (1 << 64)


def test_queue_is_a_run_of_its_models_arrivals():
    """A model's queue is always a run of its arrivals in trace order (the
    GPU kernel keeps queues as two positions in per-model arrival lists on
    this ground): a hosted arrival that runs or is dropped at once finds its
    model's queue empty, since the idle events before it let every group
    with queued work take it; and when request i joins the queue of model m,
    the queue holds exactly the arrivals of m from its head to i, since
    requests leave a queue only at its head."""
    rng = np.random.default_rng(91)
    long_runs = 0
    for k in range(400):
        t, model, d, cs, L, gc, hm, sigma = _case(rng, n=int(rng.integers(5, 40)), dyadic=k % 2 == 0)
        B = int(rng.choice([1, 2, 3, 8]))
        beta = float(rng.choice([0.0, 0.25, 1.0]))

        def check(m, q, i, at_once):
            nonlocal long_runs
            if at_once:
                assert q == (), (k, m, q, i)
            else:
                assert list(q) == [j for j in range(q[0], i + 1) if model[j] == m], (k, m, q, i)
                long_runs += len(q) >= 3

        brute.simulate_batched(t, model, d, cs, L, gc, hm, sigma, B, beta, on_queue=check)
    assert long_runs > 50  # queues of several requests were seen
