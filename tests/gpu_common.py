"""Shared helpers of the GPU parity tests: run a workload through the HIP
library and through the oracle on the same seeded inputs and compare
element by element (bit-exact: served counts, digests, attain = served / n,
per-request finish times)."""
from __future__ import annotations

import os
import sys

import numpy as np

import oracle


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def host_threads():
    """Oracle worker threads: this process's CPUs, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def oracle_problem(pb, jobs=None, finish_jobs=()):
    """Oracle results for the selected jobs (all when jobs is None) of a
    shared-trace Problem: dict job -> (served, digest, finish or None)."""
    lib = oracle.lib()
    K = pb.slo_scale.shape[0]
    J = pb.group_cfg.shape[0] * K
    jobs = range(J) if jobs is None else jobs
    want = set(int(j) for j in finish_jobs)
    out = {}
    from concurrent.futures import ThreadPoolExecutor

    def one(j):
        p, k = divmod(int(j), K)
        return int(j), lib.simulate_job(pb.t, pb.model, pb.d_single, pb.cfg_stages, pb.stage_lat,
                                        pb.group_cfg[p], pb.host_mask[p], pb.slo_scale[k],
                                        want_finish=int(j) in want)

    with ThreadPoolExecutor(host_threads()) as ex:
        for j, r in ex.map(one, list(jobs)):
            out[j] = r
    return out


def compare(gpu, ora, n, label):
    """gpu: dict from api.results; ora: dict job -> (served, digest, finish)."""
    bad = []
    for j, (s, dg, fin) in ora.items():
        if int(gpu["served"][j]) != s:
            bad.append((j, "served", int(gpu["served"][j]), s))
            continue
        if tuple(int(x) for x in gpu["digest"][j]) != dg:
            bad.append((j, "digest", tuple(int(x) for x in gpu["digest"][j]), dg))
        want_att = (s / n) if n > 0 else 0.0
        if gpu["attain"][j] != want_att:
            bad.append((j, "attain", gpu["attain"][j], want_att))
        if fin is not None:
            g = gpu["finish"][j]
            if g.tobytes() != fin.tobytes():
                i = int(np.nonzero(g.view(np.uint64) != fin.view(np.uint64))[0][0])
                bad.append((j, "finish", i, g[i], fin[i]))
    assert not bad, f"{label}: {len(bad)} mismatches, first {bad[:5]}"
