"""GPU test of the speculative kernels' fallback: when their workspace cannot
be had (forced here with ALPASERVE_SPEC_MAX_WORKSPACE, which makes a larger
workspace fail as a failed allocation does), as_simulate_placements must
still succeed, on the shared-trace kernels, with the same results bit for
bit (served counts, attainment, digests, output rows) as the speculative
kernels give, and those must equal the oracle's on sampled jobs."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_common import say  # noqa: E402

import oracle  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sim():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2302_11665_amd import sim as s
    return s


def _run(sim, pb):
    import torch
    d = sim.to_device
    J, N = pb.n_jobs, len(pb.t)
    served = torch.full((J,), -7, dtype=torch.int64, device="cuda")
    attain = torch.full((J,), float("nan"), dtype=torch.float64, device="cuda")
    digest = torch.full((J, 2), -7, dtype=torch.int64, device="cuda")
    fj = np.ascontiguousarray(pb.finish_jobs, np.int32)
    fin = torch.full((len(fj), N), float("nan"), dtype=torch.float64, device="cuda")
    sim.as_simulate_placements(d(pb.t), d(pb.model), d(pb.d_single), pb.cfg_stages, d(pb.stage_lat),
                               d(pb.group_cfg), d(pb.host_mask), d(pb.slo_scale), served, attain, digest, fj, fin)
    torch.cuda.synchronize()
    return served.cpu().numpy(), attain.cpu().numpy(), sim.u64(digest), fin.cpu().numpy()


def test_workspace_failure_falls_back(sim, monkeypatch):
    from paper_2302_11665_amd.workload import problems
    pb = problems.c4_heavy(duration=300.0, n_placements=256, n_finish=4)
    monkeypatch.setenv("ALPASERVE_PATH", "spec")
    monkeypatch.setenv("ALPASERVE_SPEC_SEGMENTS", "7")
    monkeypatch.delenv("ALPASERVE_SPEC_MAX_WORKSPACE", raising=False)
    say("spec fallback: speculative kernels", pb.n_jobs, "jobs", len(pb.t), "requests")
    spec = _run(sim, pb)
    monkeypatch.setenv("ALPASERVE_SPEC_MAX_WORKSPACE", "1")
    say("spec fallback: workspace refused")
    fell = _run(sim, pb)
    for a, b in zip(spec, fell):
        assert np.asarray(a).tobytes() == np.asarray(b).tobytes()
    served, attain, digest, fin = spec
    assert (served >= 0).all() and not np.isnan(fin).any()
    lib = oracle.lib()
    K = pb.slo_scale.shape[0]
    rows = {int(j): f for f, j in enumerate(pb.finish_jobs)}
    for j in sorted(set([0, pb.n_jobs - 1] + [int(x) for x in pb.finish_jobs[:2]])):
        p, k = divmod(j, K)
        s, dg, f = lib.simulate_job(pb.t, pb.model, pb.d_single, pb.cfg_stages, pb.stage_lat, pb.group_cfg[p],
                                    pb.host_mask[p], pb.slo_scale[k], want_finish=j in rows)
        assert int(served[j]) == s and tuple(int(x) for x in digest[j]) == dg, j
        if j in rows:
            assert fin[rows[j]].tobytes() == f.tobytes(), j
