"""GPU test of as_simulate_placements_noalloc, called through the C-ABI: its
outputs equal those of as_simulate_placements bit for bit (served counts,
attainment, digests, every per-request output row) on calls in a row whose
inputs shrink, so that the shared scratch array carries the previous call's
contents into the next; on the speculative kernels (forced, with several
segments), on the default path choice, and on re-runs that give up; and a
call whose workspace would exceed the scratch is refused with AS_E_LIMITS
before anything is launched."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_common import say  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sim():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2302_11665_amd import sim as s
    return s


def _run(sim, pb, noalloc):
    """One call of either entry point on freshly uploaded inputs; outputs
    start as NaN / -7 so that anything left unwritten shows."""
    import torch
    d = sim.to_device
    J, N = pb.n_jobs, len(pb.t)
    served = torch.full((J,), -7, dtype=torch.int64, device="cuda")
    attain = torch.full((J,), float("nan"), dtype=torch.float64, device="cuda")
    digest = torch.full((J, 2), -7, dtype=torch.int64, device="cuda")
    fj = np.ascontiguousarray(pb.finish_jobs, np.int32)
    fin = torch.full((len(fj), N), float("nan"), dtype=torch.float64, device="cuda")
    fn = sim.as_simulate_placements_noalloc if noalloc else sim.as_simulate_placements
    fn(d(pb.t), d(pb.model), d(pb.d_single), pb.cfg_stages, d(pb.stage_lat), d(pb.group_cfg), d(pb.host_mask),
       d(pb.slo_scale), served, attain, digest, fj, fin)
    torch.cuda.synchronize()
    return served.cpu().numpy(), attain.cpu().numpy(), sim.u64(digest), fin.cpu().numpy()


def _same(a, b, label):
    s1, a1, d1, f1 = a
    s2, a2, d2, f2 = b
    assert np.array_equal(s1, s2), label
    assert a1.tobytes() == a2.tobytes(), label
    assert np.array_equal(d1, d2), label
    assert f1.tobytes() == f2.tobytes(), label
    assert not np.isnan(f1).any() and (s1 >= 0).all(), label


def _problems():
    from paper_2302_11665_amd.workload import problems
    # heavy-trace shape (16 groups of S=4, power-law rates, Gamma CV 4, SLO
    # scale 5), shrinking from one call to the next
    return [problems.c4_heavy(duration=900.0, n_placements=1024),
            problems.c4_heavy(duration=600.0, n_placements=512),
            problems.c4_heavy(duration=300.0, n_placements=200)]


def test_noalloc_equals_allocating_entry_point_forced_spec(sim, monkeypatch):
    monkeypatch.setenv("ALPASERVE_PATH", "spec")
    monkeypatch.setenv("ALPASERVE_SPEC_SEGMENTS", "7")
    for k, pb in enumerate(_problems()):
        say(f"noalloc forced spec: call {k}, {pb.n_jobs} jobs x {len(pb.t)} requests")
        _same(_run(sim, pb, True), _run(sim, pb, False), f"forced spec call {k}")


def test_noalloc_equals_allocating_entry_point_default_path(sim, monkeypatch):
    for v in ("ALPASERVE_PATH", "ALPASERVE_SPEC_SEGMENTS", "ALPASERVE_SPEC_WARMUP", "ALPASERVE_SPEC_CAP"):
        monkeypatch.delenv(v, raising=False)
    for k, pb in enumerate(_problems()[:2]):
        say(f"noalloc default path: call {k}, {pb.n_jobs} jobs x {len(pb.t)} requests")
        _same(_run(sim, pb, True), _run(sim, pb, False), f"default path call {k}")


def test_noalloc_equals_allocating_entry_point_give_up(sim, monkeypatch):
    """Re-runs that give up after 64 requests: the gated shared-trace kernels
    read the give-up flag from the scratch array and produce the results."""
    monkeypatch.setenv("ALPASERVE_PATH", "spec")
    monkeypatch.setenv("ALPASERVE_SPEC_SEGMENTS", "5")
    monkeypatch.setenv("ALPASERVE_SPEC_WARMUP", "0")
    monkeypatch.setenv("ALPASERVE_SPEC_CAP", "64")
    for k, pb in enumerate(_problems()[1:]):
        say(f"noalloc give-up: call {k}, {pb.n_jobs} jobs x {len(pb.t)} requests")
        _same(_run(sim, pb, True), _run(sim, pb, False), f"give-up call {k}")


def test_noalloc_refuses_a_workspace_beyond_the_scratch(sim, monkeypatch):
    """8192 jobs x 1.8 M requests need about 2.8 GB of speculative workspace,
    more than the 256 MiB scratch: AS_E_LIMITS, outputs untouched."""
    import torch
    from paper_2302_11665_amd.workload import problems
    monkeypatch.setenv("ALPASERVE_PATH", "spec")
    pb = problems.c4_heavy(duration=1800.0, n_placements=8192)
    say(f"noalloc refusal: {pb.n_jobs} jobs x {len(pb.t)} requests")
    d = sim.to_device
    served = torch.full((pb.n_jobs,), -7, dtype=torch.int64, device="cuda")
    with pytest.raises(sim.SimError) as ei:
        sim.as_simulate_placements_noalloc(d(pb.t), d(pb.model), d(pb.d_single), pb.cfg_stages,
                                           d(pb.stage_lat), d(pb.group_cfg), d(pb.host_mask),
                                           d(pb.slo_scale), served)
    assert ei.value.code == sim.AS_E_LIMITS
    assert "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert (served.cpu().numpy() == -7).all()
