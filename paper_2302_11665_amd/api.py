"""Convenience layer over the binding: upload a workload once, run it many times.

Marshalling only (device copies via torch, output allocation, one C-ABI call
per run); the simulation itself is the HIP library's."""
from __future__ import annotations

import dataclasses

import numpy as np

from . import sim


@dataclasses.dataclass
class DeviceProblem:
    """Device-resident inputs and outputs of one batched call."""
    t: object
    model: object
    d_single: object
    cfg_stages: np.ndarray
    stage_lat: object
    group_cfg: object
    host_mask: object
    slo_scale: object
    finish_jobs: np.ndarray
    out_served: object
    out_attain: object
    out_digest: object
    out_finish: object
    n_jobs: int
    n: int


def upload(pb, device="cuda", finish=True) -> DeviceProblem:
    import torch
    d = lambda a: sim.to_device(a, device)  # noqa: E731
    J = pb.group_cfg.shape[0] * pb.slo_scale.shape[0]
    fj = np.ascontiguousarray(pb.finish_jobs if finish else np.zeros(0), dtype=np.int32)
    n = int(pb.t.shape[0])
    return DeviceProblem(
        t=d(pb.t), model=d(pb.model), d_single=d(pb.d_single),
        cfg_stages=np.ascontiguousarray(pb.cfg_stages, np.int32), stage_lat=d(pb.stage_lat),
        group_cfg=d(pb.group_cfg), host_mask=d(pb.host_mask), slo_scale=d(pb.slo_scale),
        finish_jobs=fj,
        out_served=torch.empty(J, dtype=torch.int64, device=device),
        out_attain=torch.empty(J, dtype=torch.float64, device=device),
        out_digest=torch.empty((J, 2), dtype=torch.int64, device=device),
        out_finish=torch.empty((len(fj), n), dtype=torch.float64, device=device) if len(fj) else None,
        n_jobs=J, n=n)


def run(dp: DeviceProblem, stream=None) -> None:
    """One batched call (asynchronous on the stream)."""
    sim.as_simulate_placements(dp.t, dp.model, dp.d_single, dp.cfg_stages, dp.stage_lat, dp.group_cfg,
                               dp.host_mask, dp.slo_scale, dp.out_served, dp.out_attain, dp.out_digest,
                               dp.finish_jobs if len(dp.finish_jobs) else None, dp.out_finish,
                               stream=stream)


def results(dp: DeviceProblem) -> dict:
    """Copy outputs to host numpy (synchronises)."""
    out = {"served": dp.out_served.cpu().numpy(), "attain": dp.out_attain.cpu().numpy(),
           "digest": sim.u64(dp.out_digest)}
    if dp.out_finish is not None:
        fin = dp.out_finish.cpu().numpy()
        out["finish"] = {int(j): fin[f] for f, j in enumerate(dp.finish_jobs)}
    else:
        out["finish"] = {}
    return out


def simulate_problem(pb, device="cuda", finish=True) -> dict:
    dp = upload(pb, device, finish)
    run(dp)
    return results(dp)


@dataclasses.dataclass
class DeviceSweep:
    t: object
    model: object
    seg_offsets: object
    d_single: object
    cfg_stages: np.ndarray
    stage_lat: object
    group_cfg: object
    host_mask: object
    jobs: object
    finish_jobs: np.ndarray
    finish_stride: int
    out_served: object
    out_attain: object
    out_digest: object
    out_finish: object
    n_jobs: int


def upload_sweep(sp, device="cuda", finish=True) -> DeviceSweep:
    import torch
    d = lambda a: sim.to_device(a, device)  # noqa: E731
    J = int(sp.job_segment.shape[0])
    fj = np.ascontiguousarray(sp.finish_jobs if finish else np.zeros(0), dtype=np.int32)
    lens = np.diff(sp.seg_offsets)
    stride = int(lens[sp.job_segment[fj]].max()) if len(fj) else 0
    jobs = sim.jobs_to_bytes(sp.job_placement, sp.job_segment, sp.job_scale)
    return DeviceSweep(
        t=d(sp.t), model=d(sp.model), seg_offsets=d(sp.seg_offsets), d_single=d(sp.d_single),
        cfg_stages=np.ascontiguousarray(sp.cfg_stages, np.int32), stage_lat=d(sp.stage_lat),
        group_cfg=d(sp.group_cfg), host_mask=d(sp.host_mask), jobs=d(jobs), finish_jobs=fj,
        finish_stride=stride,
        out_served=torch.empty(J, dtype=torch.int64, device=device),
        out_attain=torch.empty(J, dtype=torch.float64, device=device),
        out_digest=torch.empty((J, 2), dtype=torch.int64, device=device),
        out_finish=(torch.full((len(fj), stride), float("nan"), dtype=torch.float64, device=device)
                    if len(fj) else None),
        n_jobs=J)


def run_sweep(ds: DeviceSweep, stream=None) -> None:
    sim.as_simulate_jobs(ds.t, ds.model, ds.seg_offsets, ds.d_single, ds.cfg_stages, ds.stage_lat,
                         ds.group_cfg, ds.host_mask, ds.jobs, ds.out_served, ds.out_attain, ds.out_digest,
                         ds.finish_jobs if len(ds.finish_jobs) else None, ds.out_finish,
                         ds.finish_stride, stream=stream)


def sweep_results(ds: DeviceSweep) -> dict:
    out = {"served": ds.out_served.cpu().numpy(), "attain": ds.out_attain.cpu().numpy(),
           "digest": sim.u64(ds.out_digest)}
    out["finish"] = {}
    if ds.out_finish is not None:
        fin = ds.out_finish.cpu().numpy()
        out["finish"] = {int(j): fin[f] for f, j in enumerate(ds.finish_jobs)}
    return out
