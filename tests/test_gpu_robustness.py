"""Placements chosen on one non-stationary trace and served on another
(Sec. 6.4's robustness setting, on synthetic windowed Gamma traces in place of
two slices of a production trace): the native partition search on trace A
equals the oracle's, and every partition's chosen placement simulated on
trace B equals the oracle bit for bit."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_common import compare, oracle_problem, say  # noqa: E402

import oracle  # noqa: E402
from oracle import greedy as ogreedy  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2302_11665_amd import sim
    return sim


def test_search_on_trace_a_served_on_trace_b(dev):
    from paper_2302_11665_amd import api
    from paper_2302_11665_amd.workload import problems
    rp = problems.robustness(n_windows=10)
    gp = rp.greedy
    say("robustness", len(gp.t), "requests on A,", len(rp.t_b), "on B")
    d = dev.to_device
    r = dev.as_partition_search(d(gp.t), d(gp.model), d(gp.d_single), gp.cfg_stages, d(gp.stage_lat),
                                gp.weight_mib, gp.partitions, gp.slo_scale)
    best, results = ogreedy.reduced_partition_search(oracle.lib(), gp.t, gp.model, gp.d_single,
                                                     gp.weight_mib, gp.cfg_stages, gp.stage_lat,
                                                     gp.partitions, gp.slo_scale)
    assert r["part_served"] == [x["best_served"] for x in results]
    assert r["best_partition"] == best["partition"]
    assert [int(x) for x in r["best_mask"]] == [int(x) for x in best["best_mask"]]
    # every partition's chosen selection, served on trace B
    G = max(len(p["group_cfg"]) for p in gp.partitions)
    gcfg = np.full((len(results), G), -1, np.int32)
    masks = np.zeros((len(results), len(gp.d_single)), np.uint64)
    for i, (p, x) in enumerate(zip(gp.partitions, results)):
        gcfg[i, : len(p["group_cfg"])] = p["group_cfg"]
        masks[i] = np.asarray(x["best_mask"], np.uint64)
    pb = problems.Problem("robustness_b", rp.t_b, rp.model_b, gp.d_single, gp.weight_mib, gp.cfg_stages,
                          gp.cfg_k, gp.stage_lat, gcfg, masks, np.array([gp.slo_scale]),
                          np.array([best["partition"]], np.int32))
    res = api.simulate_problem(pb)
    compare(res, oracle_problem(pb, finish_jobs=pb.finish_jobs), len(pb.t), "robustness B")
    att_a = [x["best_served"] / len(gp.t) for x in results]
    say("attainment on A", [round(a, 4) for a in att_a], "on B", [round(float(a), 4) for a in res["attain"]])
