"""GPU parity of the per-job statistics kernel and of the native beam search
and fast heuristic (Sec. 4.2) against the oracle, bit-exact: served counts,
digests, per-model served counts, per-group busy times (fp64 bits), every
step of every search and the best selection."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_common import say  # noqa: E402

import oracle  # noqa: E402
from oracle import greedy as ogreedy  # noqa: E402

pytestmark = pytest.mark.gpu
INF = float("inf")


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2302_11665_amd import sim
    return sim


def _stats_case(rng, G, Smax, M, n):
    C = min(G, 6)
    cfg_stages = rng.integers(1, Smax + 1, C).astype(np.int32)
    cfg_stages[0] = Smax
    L = rng.uniform(0.02, 0.6, (M, C, Smax))
    gaps = rng.exponential(0.5 / max(G, 1), n)
    gaps[rng.random(n) < 0.2] = 0.0
    t = np.cumsum(gaps)
    model = rng.integers(0, M, n).astype(np.int32)
    d_single = L[:, 0, :].sum(axis=1) / rng.uniform(0.5, 2.0, M)
    P = 5
    group_cfg = rng.integers(-1, C, (P, G)).astype(np.int32)
    group_cfg[:, 0] = 0
    host_mask = np.zeros((P, M), np.uint64)
    for p in range(P):
        for m in range(M):
            bits = 0
            for g in range(G):
                if group_cfg[p, g] >= 0 and rng.random() < 0.35:
                    bits |= 1 << g
            host_mask[p, m] = np.uint64(bits)
    scales = np.array([2.5, INF, 0.0], np.float64)
    return t, model, d_single, cfg_stages, L, group_cfg, host_mask, scales


# one scale runs the shared-trace kernel's statistics mode, several scales the
# statistics kernel
@pytest.mark.parametrize("one_scale", [True, False])
@pytest.mark.parametrize("G,Smax", [(1, 1), (3, 2), (16, 4), (17, 3), (40, 8), (64, 1)])
def test_stats_kernel_matches_oracle(dev, G, Smax, one_scale):
    import torch
    rng = np.random.default_rng(100 + G * 10 + Smax)
    M = 7
    n = 2500 + 7 * G
    t, model, d_single, cfg_stages, L, gcfg, hm, scales = _stats_case(rng, G, Smax, M, n)
    if one_scale:
        scales = scales[:1]
    say("stats", G, Smax, n)
    d = dev.to_device
    P, K = gcfg.shape[0], scales.shape[0]
    J = P * K
    served = torch.empty(J, dtype=torch.int64, device="cuda")
    digest = torch.empty((J, 2), dtype=torch.int64, device="cuda")
    ms = torch.empty((J, M), dtype=torch.int64, device="cuda")
    busy = torch.empty((J, G), dtype=torch.float64, device="cuda")
    dev.as_simulate_stats(d(t), d(model), d(d_single), cfg_stages, d(L), d(gcfg), d(hm), d(scales),
                          served, digest, ms, busy)
    served, digest = served.cpu().numpy(), dev.u64(digest)
    ms, busy = ms.cpu().numpy(), busy.cpu().numpy()
    lib = oracle.lib()
    for j in range(J):
        p, k = divmod(j, K)
        s, dg, oms, obusy = lib.simulate_job_stats(t, model, d_single, cfg_stages, L, gcfg[p], hm[p], scales[k])
        assert int(served[j]) == s, (j, served[j], s)
        assert tuple(int(x) for x in digest[j]) == dg, j
        assert ms[j].tolist() == oms.tolist(), j
        assert busy[j].tobytes() == obusy.tobytes(), (j, busy[j], obusy)


def test_stats_empty_trace(dev):
    import torch
    rng = np.random.default_rng(5)
    t, model, d_single, cfg_stages, L, gcfg, hm, scales = _stats_case(rng, 4, 2, 3, 10)
    d = dev.to_device
    J = gcfg.shape[0] * scales.shape[0]
    served = torch.full((J,), -7, dtype=torch.int64, device="cuda")
    ms = torch.full((J, 3), -7, dtype=torch.int64, device="cuda")
    busy = torch.full((J, 4), -7.0, dtype=torch.float64, device="cuda")
    dev.as_simulate_stats(d(t[:0]), d(model[:0]), d(d_single), cfg_stages, d(L), d(gcfg), d(hm), d(scales),
                          served, None, ms, busy)
    assert served.cpu().numpy().tolist() == [0] * J
    assert (ms.cpu().numpy() == 0).all() and (busy.cpu().numpy() == 0.0).all()


def _upload(sim, gp):
    d = sim.to_device
    return d(gp.t), d(gp.model), d(gp.d_single), d(gp.stage_lat)


@pytest.mark.parametrize("beam", [2, 4])
def test_beam_search_matches_oracle(dev, beam):
    from paper_2302_11665_amd.workload import problems
    gp = problems.c3_greedy(duration=30.0, n_models=8, n_devices=16,
                            partitions=[(2, 2, 1), (4, 4, 1), (4, 2, 2)])
    t, m, d, L = _upload(dev, gp)
    lib = oracle.lib()
    for part in gp.partitions:
        say("beam", beam, part["label"])
        r = dev.as_beam_placement(t, m, d, gp.cfg_stages, L, gp.weight_mib, part["group_cfg"],
                                  part["group_mem_mib"], gp.slo_scale, beam)
        o = ogreedy.beam_selection(lib, gp.t, gp.model, gp.d_single, gp.weight_mib, gp.cfg_stages,
                                   gp.stage_lat, part["group_cfg"], part["group_mem_mib"], gp.slo_scale,
                                   beam=beam)
        assert r["n_steps"] == len(o["steps"])
        assert r["steps"] == [(int(mm), int(g), int(s)) for (_, mm, g, s, _) in o["steps"]]
        assert r["best_served"] == o["best_served"]
        assert [int(x) for x in r["best_mask"]] == [int(x) for x in o["best_mask"]]


def test_beam_one_equals_greedy(dev):
    from paper_2302_11665_amd.workload import problems
    gp = problems.c3_greedy(duration=30.0, n_models=8, n_devices=16, partitions=[(4, 4, 1)])
    t, m, d, L = _upload(dev, gp)
    part = gp.partitions[0]
    a = dev.as_beam_placement(t, m, d, gp.cfg_stages, L, gp.weight_mib, part["group_cfg"],
                              part["group_mem_mib"], gp.slo_scale, 1)
    b = dev.as_greedy_placement(t, m, d, gp.cfg_stages, L, gp.weight_mib, part["group_cfg"],
                                part["group_mem_mib"], gp.slo_scale)
    assert a["steps"] == b["steps"] and a["n_steps"] == b["n_steps"]
    assert a["best_served"] == b["best_served"]
    assert a["best_mask"].tolist() == b["best_mask"].tolist()


def test_fast_heuristic_matches_oracle(dev):
    from paper_2302_11665_amd.workload import problems
    gp = problems.c3_greedy(duration=60.0, n_models=12, n_devices=32,
                            partitions=[(1, 1, 1), (4, 4, 1), (4, 2, 2), (8, 8, 1)])
    t, m, d, L = _upload(dev, gp)
    lib = oracle.lib()
    for part in gp.partitions:
        say("fast", part["label"])
        r = dev.as_fast_placement(t, m, d, gp.cfg_stages, L, gp.weight_mib, part["group_cfg"],
                                  part["group_mem_mib"], gp.slo_scale)
        o = ogreedy.fast_selection(lib, gp.t, gp.model, gp.d_single, gp.weight_mib, gp.cfg_stages,
                                   gp.stage_lat, part["group_cfg"], part["group_mem_mib"], gp.slo_scale)
        assert r["n_steps"] == len(o["steps"])
        assert r["steps"] == [tuple(int(x) for x in s) for s in o["steps"]]
        assert r["best_served"] == o["best_served"]
        assert [int(x) for x in r["best_mask"]] == [int(x) for x in o["best_mask"]]
