"""GPU parity of the segmented entry point (as_simulate_jobs): jobs that each
bring their own trace segment and SLO scale, against the oracle job by job,
bit-exact.  Covers both kernels behind it (up to 32 groups: the general
kernel; more: one job per wavefront), empty segments, job records naming a
missing placement or segment (empty jobs), scales 0 and +inf, and output rows
whose stride is shorter or longer than the segments."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
from gpu_common import say  # noqa: E402

import oracle  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2302_11665_amd import sim
    return sim


def _segments(rng, n_seg, M, max_len):
    ts, ms, offs = [], [], [0]
    for s in range(n_seg):
        n = int(rng.choice([0, 1, 31, 64, 65, 200, max_len]))
        gaps = rng.exponential(0.02, n)
        gaps[rng.random(n) < 0.2] = 0.0
        ts.append(np.cumsum(gaps))
        ms.append(rng.integers(0, M, n).astype(np.int32))
        offs.append(offs[-1] + n)
    return (np.concatenate(ts) if ts else np.zeros(0), np.concatenate(ms).astype(np.int32) if ms else np.zeros(0, np.int32),
            np.array(offs, np.int64))


def _case(rng, G, S):
    M = int(rng.integers(2, 9))
    C = int(rng.integers(1, 4))
    cfg_stages = rng.integers(1, S + 1, C).astype(np.int32)
    cfg_stages[0] = S
    L = rng.uniform(0.01, 0.3, (M, C, S))
    d = L[:, 0, :].sum(axis=1) * rng.uniform(0.5, 1.5, M)
    P = int(rng.integers(1, 6))
    gcfg = rng.integers(0, C, (P, G)).astype(np.int32)
    if rng.random() < 0.5:
        gcfg[:] = gcfg[:, :1]  # one configuration per placement
    gcfg[rng.random((P, G)) < 0.05] = -1
    gcfg[:, 0] = np.maximum(gcfg[:, 0], 0)
    masks = np.zeros((P, M), np.uint64)
    for p in range(P):
        valid = [g for g in range(G) if gcfg[p, g] >= 0]
        for m in range(M):
            if rng.random() < 0.1:
                continue
            k = int(rng.integers(1, min(len(valid), 6) + 1))
            for g in rng.choice(valid, size=k, replace=False):
                masks[p, m] = np.uint64(int(masks[p, m]) | (1 << int(g)))
    n_seg = int(rng.integers(1, 8))
    t, model, offs = _segments(rng, n_seg, M, 3000)
    if len(t) == 0:  # keep the concatenated trace non-empty (device pointers)
        t, model, offs = np.array([0.5]), np.zeros(1, np.int32), np.concatenate([offs[:-1], [1]]).astype(np.int64)
        offs[-1] = 1
    J = int(rng.integers(1, 40))
    jp = rng.integers(0, P, J).astype(np.int32)
    js = rng.integers(0, n_seg, J).astype(np.int32)
    jsc = rng.choice([0.0, 0.5, 1.0, 2.0, 5.0, np.inf], J)
    # a few invalid records: they make empty jobs
    if J > 3:
        jp[1] = P + 3
        js[2] = n_seg + 1
    return dict(M=M, C=C, cfg_stages=cfg_stages, L=L, d=d, gcfg=gcfg, masks=masks, t=t, model=model,
                offs=offs, jp=jp, js=js, jsc=jsc)


def _run(sim, c, finish, stride):
    import torch
    d = sim.to_device
    J = len(c["jp"])
    jobs = sim.jobs_to_bytes(c["jp"], c["js"], c["jsc"])
    served = torch.empty(J, dtype=torch.int64, device="cuda")
    attain = torch.empty(J, dtype=torch.float64, device="cuda")
    digest = torch.empty((J, 2), dtype=torch.int64, device="cuda")
    fin = torch.full((len(finish), max(stride, 1)), float("nan"), dtype=torch.float64, device="cuda") \
        if len(finish) else None
    sim.as_simulate_jobs(d(c["t"]), d(c["model"]), d(c["offs"]), d(c["d"]), c["cfg_stages"], d(c["L"]),
                         d(c["gcfg"]), d(c["masks"]), d(jobs), served, attain, digest,
                         np.array(finish, np.int32) if len(finish) else None, fin, stride)
    return (served.cpu().numpy(), attain.cpu().numpy(), sim.u64(digest),
            fin.cpu().numpy() if fin is not None else None)


def _check(c, res, finish, stride):
    lib = oracle.lib()
    served, attain, digest, fin = res
    P = c["gcfg"].shape[0]
    n_seg = len(c["offs"]) - 1
    for j in range(len(c["jp"])):
        p, sg = int(c["jp"][j]), int(c["js"][j])
        if not (0 <= p < P and 0 <= sg < n_seg):
            assert served[j] == 0 and attain[j] == 0.0 and tuple(digest[j]) == (0, 0), j
            continue
        a, b = int(c["offs"][sg]), int(c["offs"][sg + 1])
        want_f = j in finish
        s, dg, f = lib.simulate_job(c["t"][a:b], c["model"][a:b], c["d"], c["cfg_stages"], c["L"], c["gcfg"][p],
                                    c["masks"][p], float(c["jsc"][j]), want_finish=want_f)
        assert int(served[j]) == s, j
        assert tuple(int(x) for x in digest[j]) == dg, j
        assert attain[j] == (s / (b - a) if b > a else 0.0), j
        if want_f:
            row = fin[finish.index(j)]
            k = min(b - a, stride)
            assert row[:k].tobytes() == f[:k].tobytes(), j
            assert np.all(np.isnan(row[k:stride])), j  # past the segment: untouched


@pytest.mark.parametrize("G", [8, 17, 33, 64])
def test_random_segmented_jobs(dev, G):
    rng = np.random.default_rng(700 + G)
    for S in (1, 2, 4, 8):
        c = _case(rng, G, S)
        J = len(c["jp"])
        finish = sorted(set(rng.choice(J, size=min(3, J), replace=False).tolist()))
        stride = int(rng.choice([50, 4000]))
        say("segmented", G, S, "jobs", J, "requests", len(c["t"]), "stride", stride)
        _check(c, _run(dev, c, finish, stride), finish, stride)


def _permuted(c, perm):
    return dict(c, jp=c["jp"][perm], js=c["js"][perm], jsc=c["jsc"][perm])


@pytest.mark.parametrize("J", [2, 300, 4096, 4100])
def test_launch_order_does_not_change_results(dev, J):
    """With more than 32 groups the jobs run one per wavefront, launched
    longest and shortest segment alternating (sorted on the device for up
    to 4096 jobs, in the given order beyond): the results, indexed by job,
    are the same for any order of the job records."""
    rng = np.random.default_rng(900 + J)
    c = _case(rng, 64, 2)
    n_seg = len(c["offs"]) - 1
    # many jobs over segments of very different lengths (several ties)
    c = dict(c, jp=rng.integers(0, c["gcfg"].shape[0], J).astype(np.int32),
             js=rng.integers(0, n_seg, J).astype(np.int32), jsc=rng.choice([0.5, 2.0, 5.0, np.inf], J))
    say("launch order", J, "jobs", n_seg, "segments")
    ref = _run(dev, c, [], 0)
    perm = rng.permutation(J)
    got = _run(dev, _permuted(c, perm), [], 0)
    for a, b in zip(ref[:3], got[:3]):
        assert np.array_equal(np.asarray(a)[perm], np.asarray(b))
    sample = sorted(set(rng.choice(J, size=min(J, 24), replace=False).tolist()))
    sub = dict(c, jp=c["jp"][sample], js=c["js"][sample], jsc=c["jsc"][sample])
    _check(sub, tuple(np.asarray(x)[sample] for x in ref[:3]) + (None,), [], 0)


@pytest.mark.parametrize("J,blocks", [(13, 3), (300, 1), (1000, 3), (4096, 7)])
def test_job_queue_matches_one_job_per_wavefront(dev, monkeypatch, J, blocks):
    """With more jobs than the wavefronts launched, the wavefronts take the
    jobs in turn, longest segment first, from a counter (ALPASERVE_SEG_BLOCKS
    forces that with a few workgroups, so that each wavefront runs many jobs
    one after the other in its own LDS records): every output, output rows
    included, equals the one-job-per-wavefront launch's, and a sample equals
    the oracle's."""
    rng = np.random.default_rng(1300 + J)
    c = _case(rng, 64, 4)
    n_seg = len(c["offs"]) - 1
    c = dict(c, jp=rng.integers(0, c["gcfg"].shape[0], J).astype(np.int32),
             js=rng.integers(0, n_seg, J).astype(np.int32), jsc=rng.choice([0.5, 2.0, 5.0, np.inf], J))
    finish = sorted(set(rng.choice(J, size=min(J, 5), replace=False).tolist()))
    stride = 2000
    monkeypatch.delenv("ALPASERVE_SEG_BLOCKS", raising=False)
    monkeypatch.setenv("ALPASERVE_SEG_WAVES", "4")  # one job per wavefront for up to 4096 jobs on 256 CUs
    say("job queue reference", J, "jobs")
    ref = _run(dev, c, finish, stride)
    monkeypatch.setenv("ALPASERVE_SEG_BLOCKS", str(blocks))
    say("job queue", J, "jobs,", blocks, "workgroups")
    got = _run(dev, c, finish, stride)
    for a, b in zip(ref[:3], got[:3]):
        assert np.array_equal(np.asarray(a), np.asarray(b))
    assert ref[3].tobytes() == got[3].tobytes()
    sample = sorted(set(rng.choice(J, size=min(J, 16), replace=False).tolist()) | set(finish))
    sub = dict(c, jp=c["jp"][sample], js=c["js"][sample], jsc=c["jsc"][sample])
    fin_sub = [sample.index(j) for j in finish]
    _check(sub, tuple(np.asarray(x)[sample] for x in got[:3]) + (got[3],), fin_sub, stride)
