"""Thin ctypes binding of libalpaserve_sim.so (see include/alpaserve_sim.h).

Argument marshalling only: device arrays are torch CUDA tensors (PyTorch is
used for device memory and streams), host arrays are numpy, calls go to the
C-ABI unchanged and run on torch's current stream.  Every step of the
simulation runs in the library's HIP kernels; if the library is not built this
module raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

AS_OK = 0
AS_E_INVALID_ARG = -1
AS_E_LIMITS = -2
AS_E_HIP = -3
AS_E_NOMEM = -4
AS_E_INVALID_DATA = -5
AS_MAX_FINISH = 256

_P = ctypes.c_void_p


class as_trace_t(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("t", _P), ("model", _P)]


class as_models_t(ctypes.Structure):
    _fields_ = [("n_models", ctypes.c_int32), ("n_configs", ctypes.c_int32),
                ("max_stages", ctypes.c_int32), ("d_single", _P), ("cfg_stages", _P),
                ("stage_lat", _P)]


class as_placements_t(ctypes.Structure):
    _fields_ = [("n_placements", ctypes.c_int32), ("max_groups", ctypes.c_int32),
                ("group_cfg", _P), ("host_mask", _P)]


class as_job_t(ctypes.Structure):
    _fields_ = [("placement", ctypes.c_int32), ("segment", ctypes.c_int32),
                ("slo_scale", ctypes.c_double)]


AS_MAX_MODELS = 64
AS_MAX_GROUPS = 64
AS_MAX_BUCKETS = 8


class as_search_opts_t(ctypes.Structure):
    _fields_ = [("n_devices", ctypes.c_int32), ("device_unit", ctypes.c_int32),
                ("device_mem_mib", ctypes.c_int64), ("cfg_devices", _P),
                ("bucket_threshold", ctypes.c_double), ("balance_ratio", ctypes.c_double),
                ("slo_scale", ctypes.c_double), ("max_buckets", ctypes.c_int32), ("beam", ctypes.c_int32)]


class as_search_result_t(ctypes.Structure):
    _fields_ = [("served", ctypes.c_int64), ("n_buckets", ctypes.c_int32),
                ("n_bucket_configs", ctypes.c_int32), ("n_device_splits", ctypes.c_int32),
                ("n_kept_splits", ctypes.c_int32), ("n_problems", ctypes.c_int32),
                ("launches", ctypes.c_int64), ("jobs_simulated", ctypes.c_int64),
                ("model_bucket", ctypes.c_int32 * AS_MAX_MODELS),
                ("bucket_devices", ctypes.c_int32 * AS_MAX_BUCKETS),
                ("bucket_cfg", ctypes.c_int32 * AS_MAX_BUCKETS),
                ("bucket_groups", ctypes.c_int32 * AS_MAX_BUCKETS),
                ("bucket_group_cfg", (ctypes.c_int32 * AS_MAX_GROUPS) * AS_MAX_BUCKETS),
                ("bucket_served", ctypes.c_int64 * AS_MAX_BUCKETS),
                ("bucket_mask", (ctypes.c_uint64 * AS_MAX_MODELS) * AS_MAX_BUCKETS)]


AS_JOB_DTYPE = np.dtype([("placement", np.int32), ("segment", np.int32), ("slo_scale", np.float64)])
assert AS_JOB_DTYPE.itemsize == ctypes.sizeof(as_job_t) == 16


class SimError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"[{code}] {msg}")
        self.code = code


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.SIM_LIB):
            raise RuntimeError(f"{_build.SIM_LIB} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(_build.SIM_LIB)
        L.as_simulate_placements.argtypes = [ctypes.POINTER(as_trace_t), ctypes.POINTER(as_models_t),
                                             ctypes.POINTER(as_placements_t), _P, ctypes.c_int32,
                                             _P, _P, _P, _P, ctypes.c_int32, _P, _P]
        L.as_simulate_placements.restype = ctypes.c_int
        L.as_simulate_placements_noalloc.argtypes = L.as_simulate_placements.argtypes
        L.as_simulate_placements_noalloc.restype = ctypes.c_int
        L.as_simulate_jobs.argtypes = [_P, _P, _P, ctypes.c_int32, ctypes.POINTER(as_models_t),
                                       ctypes.POINTER(as_placements_t), _P, ctypes.c_int32, _P, _P, _P,
                                       _P, ctypes.c_int32, _P, ctypes.c_int64, _P]
        L.as_simulate_jobs.restype = ctypes.c_int
        L.as_validate.argtypes = [ctypes.POINTER(as_trace_t), ctypes.POINTER(as_models_t),
                                  ctypes.POINTER(as_placements_t), _P, ctypes.c_int32, _P]
        L.as_validate.restype = ctypes.c_int
        L.as_greedy_placement.argtypes = [ctypes.POINTER(as_trace_t), ctypes.POINTER(as_models_t), _P,
                                          ctypes.c_int32, _P, _P, ctypes.c_double, _P, _P, _P, _P, _P,
                                          ctypes.c_int32, _P, _P]
        L.as_greedy_placement.restype = ctypes.c_int
        L.as_partition_search.argtypes = [ctypes.POINTER(as_trace_t), ctypes.POINTER(as_models_t), _P,
                                          ctypes.c_int32, _P, _P, _P, ctypes.c_double, _P, _P, _P, _P, _P]
        L.as_partition_search.restype = ctypes.c_int
        L.as_beam_placement.argtypes = [ctypes.POINTER(as_trace_t), ctypes.POINTER(as_models_t), _P,
                                        ctypes.c_int32, _P, _P, ctypes.c_double, ctypes.c_int32, _P, _P,
                                        _P, _P, _P, ctypes.c_int32, _P, _P]
        L.as_beam_placement.restype = ctypes.c_int
        L.as_fast_placement.argtypes = L.as_greedy_placement.argtypes
        L.as_fast_placement.restype = ctypes.c_int
        L.as_simulate_stats.argtypes = [ctypes.POINTER(as_trace_t), ctypes.POINTER(as_models_t),
                                        ctypes.POINTER(as_placements_t), _P, ctypes.c_int32, _P, _P, _P,
                                        _P, _P]
        L.as_simulate_stats.restype = ctypes.c_int
        L.as_placement_search.argtypes = [ctypes.POINTER(as_trace_t), ctypes.POINTER(as_models_t), _P,
                                          ctypes.POINTER(as_search_opts_t), ctypes.POINTER(as_search_result_t),
                                          _P]
        L.as_placement_search.restype = ctypes.c_int
        L.as_simulate_batched.argtypes = [ctypes.POINTER(as_trace_t), ctypes.POINTER(as_models_t),
                                          ctypes.POINTER(as_placements_t), _P, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_double, ctypes.c_int32, _P, _P, _P, ctypes.c_int32, _P, _P]
        L.as_simulate_batched.restype = ctypes.c_int
        L.as_last_error.argtypes = []
        L.as_last_error.restype = ctypes.c_char_p
        L.as_version.argtypes = []
        L.as_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def as_last_error() -> str:
    return lib().as_last_error().decode()


def as_version() -> str:
    return lib().as_version().decode()


def _ptr(x):
    """Device pointer of a torch tensor, host pointer of a numpy array, or NULL."""
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _check(rc):
    if rc != AS_OK:
        raise SimError(rc, as_last_error())


def _stream(stream):
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def make_models(d_single, cfg_stages: np.ndarray, stage_lat):
    """as_models_t over device tensors d_single[M], stage_lat[M, C, Smax] and the
    host array cfg_stages[C] (kept alive by the returned tuple)."""
    cfg = np.ascontiguousarray(cfg_stages, dtype=np.int32)
    M, C, S = stage_lat.shape
    m = as_models_t(M, C, S, _ptr(d_single), cfg.ctypes.data, _ptr(stage_lat))
    return m, cfg


def make_placements(group_cfg, host_mask):
    P, G = group_cfg.shape
    return as_placements_t(P, G, _ptr(group_cfg), _ptr(host_mask))


def as_simulate_placements_noalloc(t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask,
                                   slo_scale, out_served, out_attain=None, out_digest=None,
                                   finish_jobs=None, out_finish=None, stream=None):
    """Marshal to as_simulate_placements_noalloc (arguments as for
    as_simulate_placements; the library allocates nothing)."""
    return as_simulate_placements(t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask, slo_scale,
                                  out_served, out_attain, out_digest, finish_jobs, out_finish, stream,
                                  _fn=lib().as_simulate_placements_noalloc)


def as_simulate_placements(t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask,
                           slo_scale, out_served, out_attain=None, out_digest=None,
                           finish_jobs=None, out_finish=None, stream=None, _fn=None):
    """Marshal to as_simulate_placements.  Device tensors: t[N] f64, model[N] i32,
    d_single[M] f64, stage_lat[M,C,Smax] f64, group_cfg[P,G] i32, host_mask[P,M]
    (int64 storage of the uint64 bitmaps), slo_scale[K] f64, out_served[P*K] i64,
    out_attain[P*K] f64, out_digest[P*K,2] (int64 storage), out_finish[F,N] f64.
    Host: cfg_stages[C] i32, finish_jobs[F] i32."""
    tr = as_trace_t(int(t.shape[0]), _ptr(t), _ptr(model))
    md, _keep = make_models(d_single, cfg_stages, stage_lat)
    pl = make_placements(group_cfg, host_mask)
    fj = None if finish_jobs is None else np.ascontiguousarray(finish_jobs, dtype=np.int32)
    nf = 0 if fj is None else int(fj.shape[0])
    fn = _fn if _fn is not None else lib().as_simulate_placements
    rc = fn(ctypes.byref(tr), ctypes.byref(md), ctypes.byref(pl),
                                      _ptr(slo_scale), int(slo_scale.shape[0]), _ptr(out_served),
                                      _ptr(out_attain), _ptr(out_digest), _ptr(fj), nf,
                                      _ptr(out_finish), _stream(stream))
    _check(rc)


def as_simulate_jobs(t, model, seg_offsets, d_single, cfg_stages, stage_lat, group_cfg, host_mask,
                     jobs, out_served, out_attain=None, out_digest=None, finish_jobs=None,
                     out_finish=None, finish_stride=0, stream=None):
    """Marshal to as_simulate_jobs.  jobs: device tensor of as_job_t records
    (uint8 storage, 16 bytes each) -- see jobs_to_bytes()."""
    md, _keep = make_models(d_single, cfg_stages, stage_lat)
    pl = make_placements(group_cfg, host_mask)
    fj = None if finish_jobs is None else np.ascontiguousarray(finish_jobs, dtype=np.int32)
    nf = 0 if fj is None else int(fj.shape[0])
    n_jobs = int(jobs.numel() // AS_JOB_DTYPE.itemsize)
    rc = lib().as_simulate_jobs(_ptr(t), _ptr(model), _ptr(seg_offsets), int(seg_offsets.shape[0] - 1),
                                ctypes.byref(md), ctypes.byref(pl), _ptr(jobs), n_jobs,
                                _ptr(out_served), _ptr(out_attain), _ptr(out_digest), _ptr(fj), nf,
                                _ptr(out_finish), int(finish_stride), _stream(stream))
    _check(rc)


def as_validate(t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask, slo_scale,
                stream=None):
    tr = as_trace_t(int(t.shape[0]), _ptr(t), _ptr(model))
    md, _keep = make_models(d_single, cfg_stages, stage_lat)
    pl = make_placements(group_cfg, host_mask)
    rc = lib().as_validate(ctypes.byref(tr), ctypes.byref(md), ctypes.byref(pl), _ptr(slo_scale),
                           int(slo_scale.shape[0]), _stream(stream))
    _check(rc)


def jobs_to_bytes(placement, segment, slo_scale) -> np.ndarray:
    """Pack job records into the as_job_t byte layout (host uint8 array)."""
    n = len(placement)
    rec = np.zeros(n, dtype=AS_JOB_DTYPE)
    rec["placement"] = placement
    rec["segment"] = segment
    rec["slo_scale"] = slo_scale
    return rec.view(np.uint8)


# ------------------------------------------------------------------ helpers

def to_device(a, device="cuda"):
    """numpy -> torch device tensor (uint64 bitmaps travel as int64 storage)."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(a).to(device)


def u64(x) -> np.ndarray:
    """int64 storage (torch tensor or numpy) back to uint64 numpy."""
    if not isinstance(x, np.ndarray):
        x = x.cpu().numpy()
    return x.view(np.uint64)


def as_greedy_placement(t, model, d_single, cfg_stages, stage_lat, weight_mib, group_cfg, group_mem_mib,
                        slo_scale, max_steps=4096, stream=None):
    """Marshal to as_greedy_placement (device trace/model tables, host
    partition).  Returns dict(best_mask uint64[M], best_served, steps=[(m, g, served)])."""
    return _search_call(lib().as_greedy_placement, (), t, model, d_single, cfg_stages, stage_lat,
                        weight_mib, group_cfg, group_mem_mib, slo_scale, max_steps, stream)


def _search_call(fn, extra, t, model, d_single, cfg_stages, stage_lat, weight_mib, group_cfg,
                 group_mem_mib, slo_scale, max_steps, stream):
    tr = as_trace_t(int(t.shape[0]), _ptr(t), _ptr(model))
    md, _keep = make_models(d_single, cfg_stages, stage_lat)
    M = md.n_models
    w = np.ascontiguousarray(weight_mib, dtype=np.int64)
    gc = np.ascontiguousarray(group_cfg, dtype=np.int32)
    gm = np.ascontiguousarray(group_mem_mib, dtype=np.int64)
    best = np.zeros(M, dtype=np.uint64)
    best_s = np.zeros(1, dtype=np.int64)
    sm = np.zeros(max_steps, dtype=np.int32)
    sg = np.zeros(max_steps, dtype=np.int32)
    ss = np.zeros(max_steps, dtype=np.int64)
    n = np.zeros(1, dtype=np.int32)
    rc = fn(ctypes.byref(tr), ctypes.byref(md), w.ctypes.data, int(gc.shape[0]), gc.ctypes.data,
            gm.ctypes.data, float(slo_scale), *extra, best.ctypes.data, best_s.ctypes.data, sm.ctypes.data,
            sg.ctypes.data, ss.ctypes.data, max_steps, n.ctypes.data, _stream(stream))
    _check(rc)
    k = min(int(n[0]), max_steps)
    return {"best_mask": best, "best_served": int(best_s[0]), "n_steps": int(n[0]),
            "steps": [(int(sm[i]), int(sg[i]), int(ss[i])) for i in range(k)]}


def as_beam_placement(t, model, d_single, cfg_stages, stage_lat, weight_mib, group_cfg, group_mem_mib,
                      slo_scale, beam, max_steps=4096, stream=None):
    """Marshal to as_beam_placement.  Returns dict(best_mask, best_served, n_steps,
    steps=[(m, g, served)] of each step's best selection)."""
    return _search_call(lib().as_beam_placement, (int(beam),), t, model, d_single, cfg_stages, stage_lat,
                        weight_mib, group_cfg, group_mem_mib, slo_scale, max_steps, stream)


def as_fast_placement(t, model, d_single, cfg_stages, stage_lat, weight_mib, group_cfg, group_mem_mib,
                      slo_scale, max_steps=4096, stream=None):
    """Marshal to as_fast_placement.  Returns dict(best_mask, best_served, n_steps,
    steps=[(m, g, served before the addition)])."""
    return _search_call(lib().as_fast_placement, (), t, model, d_single, cfg_stages, stage_lat,
                        weight_mib, group_cfg, group_mem_mib, slo_scale, max_steps, stream)


def as_simulate_stats(t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask, slo_scale,
                      out_served, out_digest=None, out_model_served=None, out_group_busy=None,
                      stream=None):
    """Marshal to as_simulate_stats (device tensors as for as_simulate_placements;
    out_model_served[P*K, M] i64, out_group_busy[P*K, G] f64)."""
    tr = as_trace_t(int(t.shape[0]), _ptr(t), _ptr(model))
    md, _keep = make_models(d_single, cfg_stages, stage_lat)
    pl = make_placements(group_cfg, host_mask)
    rc = lib().as_simulate_stats(ctypes.byref(tr), ctypes.byref(md), ctypes.byref(pl), _ptr(slo_scale),
                                 int(slo_scale.shape[0]), _ptr(out_served), _ptr(out_digest),
                                 _ptr(out_model_served), _ptr(out_group_busy), _stream(stream))
    _check(rc)


def as_partition_search(t, model, d_single, cfg_stages, stage_lat, weight_mib, partitions, slo_scale,
                        stream=None):
    """Marshal to as_partition_search.  partitions: list of dicts with host
    arrays group_cfg[G], group_mem_mib[G]."""
    tr = as_trace_t(int(t.shape[0]), _ptr(t), _ptr(model))
    md, _keep = make_models(d_single, cfg_stages, stage_lat)
    M = md.n_models
    w = np.ascontiguousarray(weight_mib, dtype=np.int64)
    pg = np.array([len(p["group_cfg"]) for p in partitions], dtype=np.int32)
    pc = np.ascontiguousarray(np.concatenate([p["group_cfg"] for p in partitions]), dtype=np.int32)
    pm = np.ascontiguousarray(np.concatenate([p["group_mem_mib"] for p in partitions]), dtype=np.int64)
    bp = np.zeros(1, dtype=np.int32)
    best = np.zeros(M, dtype=np.uint64)
    bs = np.zeros(1, dtype=np.int64)
    ps = np.zeros(len(partitions), dtype=np.int64)
    rc = lib().as_partition_search(ctypes.byref(tr), ctypes.byref(md), w.ctypes.data, len(partitions),
                                   pg.ctypes.data, pc.ctypes.data, pm.ctypes.data, float(slo_scale),
                                   bp.ctypes.data, best.ctypes.data, bs.ctypes.data, ps.ctypes.data,
                                   _stream(stream))
    _check(rc)
    return {"best_partition": int(bp[0]), "best_mask": best, "best_served": int(bs[0]),
            "part_served": ps.tolist()}


def as_placement_search(t, model, d_single, cfg_stages, stage_lat, weight_mib, cfg_devices, n_devices,
                        device_unit, device_mem_mib, bucket_threshold, balance_ratio, max_buckets, beam,
                        slo_scale, stream=None):
    """Marshal to as_placement_search (Alg. 2).  Returns dict(served, buckets=[dict(models,
    devices, cfg, group_cfg, mask, served)], n_bucket_configs, n_device_splits,
    n_kept_splits, n_problems)."""
    tr = as_trace_t(int(t.shape[0]), _ptr(t), _ptr(model))
    md, _keep = make_models(d_single, cfg_stages, stage_lat)
    M = md.n_models
    w = np.ascontiguousarray(weight_mib, dtype=np.int64)
    cd = np.ascontiguousarray(cfg_devices, dtype=np.int32)
    o = as_search_opts_t(int(n_devices), int(device_unit), int(device_mem_mib), cd.ctypes.data,
                         float(bucket_threshold), float(balance_ratio), float(slo_scale), int(max_buckets),
                         int(beam))
    r = as_search_result_t()
    rc = lib().as_placement_search(ctypes.byref(tr), ctypes.byref(md), w.ctypes.data, ctypes.byref(o),
                                   ctypes.byref(r), _stream(stream))
    _check(rc)
    buckets = []
    for b in range(r.n_buckets):
        G = r.bucket_groups[b]
        buckets.append({"models": [m for m in range(M) if r.model_bucket[m] == b],
                        "devices": int(r.bucket_devices[b]), "cfg": int(r.bucket_cfg[b]),
                        "group_cfg": np.array([r.bucket_group_cfg[b][g] for g in range(G)], np.int32),
                        "mask": np.array([r.bucket_mask[b][m] for m in range(M)], np.uint64),
                        "served": int(r.bucket_served[b])})
    return {"served": int(r.served), "buckets": buckets, "n_bucket_configs": int(r.n_bucket_configs),
            "n_device_splits": int(r.n_device_splits), "n_kept_splits": int(r.n_kept_splits),
            "n_problems": int(r.n_problems), "launches": int(r.launches),
            "jobs_simulated": int(r.jobs_simulated)}


def as_simulate_batched(t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask, slo_scale,
                        max_batch, beta, out_served, out_digest=None, finish_jobs=None, out_finish=None,
                        queue_cap=1024, stream=None):
    """Marshal to as_simulate_batched (dynamic batching, Sec. 6.5); device
    tensors as for as_simulate_placements."""
    tr = as_trace_t(int(t.shape[0]), _ptr(t), _ptr(model))
    md, _keep = make_models(d_single, cfg_stages, stage_lat)
    pl = make_placements(group_cfg, host_mask)
    fj = None if finish_jobs is None else np.ascontiguousarray(finish_jobs, dtype=np.int32)
    nf = 0 if fj is None else int(fj.shape[0])
    rc = lib().as_simulate_batched(ctypes.byref(tr), ctypes.byref(md), ctypes.byref(pl), _ptr(slo_scale),
                                   int(slo_scale.shape[0]), int(max_batch), float(beta), int(queue_cap),
                                   _ptr(out_served), _ptr(out_digest), _ptr(fj), nf, _ptr(out_finish),
                                   _stream(stream))
    _check(rc)
