"""C-ABI checks that need no GPU: the library loads, exports every function the
headers declare, and rejects bad scalar / host arguments with the documented
codes before touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2302_11665_amd import build, sim

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared(header):
    with open(os.path.join(ROOT, "include", header)) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(as_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(build.SIM_LIB):
        pytest.skip("HIP library not built")
    return sim.lib()


def test_sim_exports_every_declared_function(L):
    names = _declared("alpaserve_sim.h")
    assert {"as_simulate_placements", "as_simulate_jobs", "as_validate", "as_last_error"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_gen_exports_every_declared_function():
    lib = ctypes.CDLL(build.GEN_LIB)
    for n in _declared("alpaserve_gen.h"):
        assert hasattr(lib, n), n


def _models(M=2, C=1, S=1, cfg=None):
    cfg = np.array(cfg if cfg is not None else [S] * C, np.int32)
    return sim.as_models_t(M, C, S, 0x1000, cfg.ctypes.data, 0x2000), cfg


def _call(trace, models, plc, scales_ptr=0x3000, K=1, served=0x4000, fj=None, nf=0, fin=None):
    return sim.lib().as_simulate_placements(
        ctypes.byref(trace) if trace is not None else None,
        ctypes.byref(models) if models is not None else None,
        ctypes.byref(plc) if plc is not None else None,
        scales_ptr, K, served, None, None, fj, nf, fin, None)


def test_argument_errors_without_device(L):
    tr = sim.as_trace_t(10, 0x10, 0x20)
    md, _k = _models()
    pl = sim.as_placements_t(3, 4, 0x30, 0x40)
    assert _call(None, md, pl) == sim.AS_E_INVALID_ARG
    assert "trace" in sim.as_last_error()
    assert _call(sim.as_trace_t(-1, 0x10, 0x20), md, pl) == sim.AS_E_INVALID_ARG
    assert _call(sim.as_trace_t(5, None, 0x20), md, pl) == sim.AS_E_INVALID_ARG
    assert _call(tr, None, pl) == sim.AS_E_INVALID_ARG
    md65, _k2 = _models(M=65)
    assert _call(tr, md65, pl) == sim.AS_E_LIMITS
    md0, _k3 = _models(M=0)
    assert _call(tr, md0, pl) == sim.AS_E_INVALID_ARG
    mds, _k4 = _models(S=9, cfg=[9])
    assert _call(tr, mds, pl) == sim.AS_E_LIMITS
    mdb, _k5 = _models(S=2, cfg=[3])
    assert _call(tr, mdb, pl) == sim.AS_E_INVALID_ARG  # S_c > max_stages
    assert _call(tr, md, sim.as_placements_t(3, 65, 0x30, 0x40)) == sim.AS_E_LIMITS
    assert _call(tr, md, sim.as_placements_t(3, 0, 0x30, 0x40)) == sim.AS_E_INVALID_ARG
    assert _call(tr, md, sim.as_placements_t(-1, 4, 0x30, 0x40)) == sim.AS_E_INVALID_ARG
    assert _call(tr, md, pl, K=-1) == sim.AS_E_INVALID_ARG
    assert _call(tr, md, pl, served=None) == sim.AS_E_INVALID_ARG
    fj = np.array([0, 0], np.int32)
    assert _call(tr, md, pl, fj=fj.ctypes.data, nf=2, fin=0x50) == sim.AS_E_INVALID_ARG  # repeated job
    fj = np.array([3], np.int32)
    assert _call(tr, md, pl, fj=fj.ctypes.data, nf=1, fin=0x50) == sim.AS_E_INVALID_ARG  # job >= P*K
    assert _call(tr, md, pl, fj=fj.ctypes.data, nf=1, fin=None) == sim.AS_E_INVALID_ARG
    assert _call(tr, md, pl, nf=sim.AS_MAX_FINISH + 1, fj=np.zeros(300, np.int32).ctypes.data,
                 fin=0x50) == sim.AS_E_LIMITS
    # zero jobs is a successful no-op that touches nothing
    assert _call(tr, md, sim.as_placements_t(0, 4, None, None)) == sim.AS_OK
    assert sim.as_last_error() == ""


def test_jobs_entry_argument_errors(L):
    md, _k = _models()
    pl = sim.as_placements_t(3, 4, 0x30, 0x40)
    f = L.as_simulate_jobs
    assert f(0x10, 0x20, 0x30, -1, ctypes.byref(md), ctypes.byref(pl), 0x60, 1, 0x70, None, None,
             None, 0, None, 0, None) == sim.AS_E_INVALID_ARG
    assert f(None, 0x20, 0x30, 1, ctypes.byref(md), ctypes.byref(pl), 0x60, 1, 0x70, None, None,
             None, 0, None, 0, None) == sim.AS_E_INVALID_ARG
    assert f(0x10, 0x20, 0x30, 1, ctypes.byref(md), ctypes.byref(pl), 0x60, 1, 0x70, None, None,
             None, 0, None, -5, None) == sim.AS_E_INVALID_ARG
    assert f(0x10, 0x20, 0x30, 1, ctypes.byref(md), ctypes.byref(pl), None, 0, None, None, None,
             None, 0, None, 0, None) == sim.AS_OK


def test_validate_argument_errors(L):
    md, _k = _models()
    pl = sim.as_placements_t(3, 4, 0x30, 0x40)
    assert L.as_validate(None, ctypes.byref(md), ctypes.byref(pl), 0x1, 1, None) == sim.AS_E_INVALID_ARG
    tr = sim.as_trace_t(4, 0x10, 0x20)
    assert L.as_validate(ctypes.byref(tr), ctypes.byref(md), ctypes.byref(pl), None, 1, None) == sim.AS_E_INVALID_ARG


def test_struct_layouts_match_header():
    assert ctypes.sizeof(sim.as_trace_t) == 24
    assert ctypes.sizeof(sim.as_models_t) == 40
    assert ctypes.sizeof(sim.as_placements_t) == 24
    assert ctypes.sizeof(sim.as_job_t) == 16


def test_search_and_stats_argument_errors(L):
    """Beam search, fast heuristic and statistics reject bad arguments before
    any device work."""
    md, _k = _models(M=2)
    tr = sim.as_trace_t(4, 0x10, 0x20)
    w = np.array([1, 2], np.int64)
    gc = np.array([0, 0], np.int32)
    gm = np.array([10, 10], np.int64)
    best = np.zeros(2, np.uint64)
    bs = np.zeros(1, np.int64)
    n = np.zeros(1, np.int32)

    def beam(k, trace=tr, G=2, scale=1.0, weights=w):
        return L.as_beam_placement(ctypes.byref(trace) if trace is not None else None, ctypes.byref(md),
                                   weights.ctypes.data, G, gc.ctypes.data, gm.ctypes.data, scale, k,
                                   best.ctypes.data, bs.ctypes.data, None, None, None, 0, n.ctypes.data, None)

    def fast(trace=tr, G=2, scale=1.0):
        return L.as_fast_placement(ctypes.byref(trace) if trace is not None else None, ctypes.byref(md),
                                   w.ctypes.data, G, gc.ctypes.data, gm.ctypes.data, scale,
                                   best.ctypes.data, bs.ctypes.data, None, None, None, 0, n.ctypes.data, None)

    assert beam(0) == sim.AS_E_INVALID_ARG
    assert "beam" in sim.as_last_error()
    assert beam(2, trace=None) == sim.AS_E_INVALID_ARG
    assert beam(2, G=0) == sim.AS_E_LIMITS
    assert beam(2, G=65) == sim.AS_E_LIMITS
    assert beam(2, scale=float("nan")) == sim.AS_E_INVALID_ARG
    assert beam(2, weights=np.array([1, -1], np.int64)) == sim.AS_E_INVALID_ARG
    assert fast(trace=None) == sim.AS_E_INVALID_ARG
    assert fast(G=0) == sim.AS_E_LIMITS
    assert fast(scale=-1.0) == sim.AS_E_INVALID_ARG
    pl = sim.as_placements_t(3, 4, 0x30, 0x40)
    st = L.as_simulate_stats
    assert st(None, ctypes.byref(md), ctypes.byref(pl), 0x50, 1, 0x60, None, None, None, None) == sim.AS_E_INVALID_ARG
    assert st(ctypes.byref(tr), ctypes.byref(md), ctypes.byref(pl), None, 1, 0x60, None, None, None,
              None) == sim.AS_E_INVALID_ARG
    assert st(ctypes.byref(tr), ctypes.byref(md), ctypes.byref(pl), 0x50, -1, 0x60, None, None, None,
              None) == sim.AS_E_INVALID_ARG
    assert st(ctypes.byref(tr), ctypes.byref(md), ctypes.byref(sim.as_placements_t(0, 4, None, None)), 0x50, 1,
              None, None, None, None, None) == sim.AS_OK


def test_batched_argument_errors(L):
    md, _k = _models(M=2)
    tr = sim.as_trace_t(4, 0x10, 0x20)
    pl = sim.as_placements_t(3, 4, 0x30, 0x40)
    f = L.as_simulate_batched

    def call(trace=tr, K=1, B=2, beta=1.0, qcap=64, served=0x60, placements=pl):
        return f(ctypes.byref(trace) if trace is not None else None, ctypes.byref(md), ctypes.byref(placements),
                 0x50, K, B, beta, qcap, served, None, None, 0, None, None)

    assert call(trace=None) == sim.AS_E_INVALID_ARG
    assert call(B=0) == sim.AS_E_INVALID_ARG
    assert call(beta=-1.0) == sim.AS_E_INVALID_ARG
    assert call(beta=float("nan")) == sim.AS_E_INVALID_ARG
    assert call(qcap=48) == sim.AS_E_INVALID_ARG  # not a power of two
    assert call(qcap=0) == sim.AS_E_INVALID_ARG
    assert call(K=-1) == sim.AS_E_INVALID_ARG
    assert call(served=None) == sim.AS_E_INVALID_ARG
    # the queues take no memory: the largest capacity is accepted (no
    # placements, so nothing reaches the device)
    assert call(qcap=1 << 20, placements=sim.as_placements_t(0, 4, None, None)) == sim.AS_OK
    assert call(placements=sim.as_placements_t(0, 4, None, None)) == sim.AS_OK
