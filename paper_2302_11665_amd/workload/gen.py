"""ctypes wrapper of libas_gen.so (seeded arrival traces and keyed uniforms).

Marshalling only; every draw is made by the C generator (gen.c)."""
from __future__ import annotations

import ctypes
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .. import build as _build

PURPOSE_ARRIVAL = 1
PURPOSE_LATENCY = 2
PURPOSE_WEIGHT = 3
PURPOSE_PERMUTE = 4
PURPOSE_WINDOW = 5
PURPOSE_WPARAM = 6

_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.GEN_LIB):
            raise RuntimeError(f"{_build.GEN_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(_build.GEN_LIB)
        lib.as_gen_key.argtypes = [ctypes.c_uint64] * 3
        lib.as_gen_key.restype = ctypes.c_uint64
        lib.as_gen_uniforms.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p]
        lib.as_gen_uniforms.restype = ctypes.c_int
        lib.as_gen_gamma.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double,
                                     ctypes.c_void_p]
        lib.as_gen_gamma.restype = ctypes.c_double
        lib.as_gen_trace.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_double, ctypes.c_double, ctypes.c_int64,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        lib.as_gen_trace.restype = ctypes.c_int
        lib.as_gen_trace_windowed.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                              ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_void_p]
        lib.as_gen_trace_windowed.restype = ctypes.c_int
        _lib = lib
    return _lib


def key(seed: int, purpose: int, index: int) -> int:
    return int(_load().as_gen_key(seed, purpose, index))


def uniforms(k: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    rc = _load().as_gen_uniforms(k, n, out.ctypes.data)
    if rc != 0:
        raise ValueError(f"as_gen_uniforms rc={rc}")
    return out


def gammas(k: int, shape: float, n: int) -> np.ndarray:
    """n consecutive Gamma(shape, 1) draws from stream k (counters threaded)."""
    lib = _load()
    out = np.empty(n, dtype=np.float64)
    ctr = ctypes.c_uint64(0)
    for i in range(n):
        out[i] = lib.as_gen_gamma(k, ctr.value, shape, ctypes.byref(ctr))
    return out


def trace(seed: int, rates, cv: float, duration: float):
    """Merged Gamma arrival trace.  Returns (t float64[n], model int32[n])."""
    lib = _load()
    rates = np.ascontiguousarray(rates, dtype=np.float64)
    lam_t = float(rates.sum()) * duration
    cap = int(lam_t + 12.0 * max(cv, 1.0) * math.sqrt(lam_t + 1.0) + 1024)
    n = ctypes.c_int64(0)
    for _ in range(3):
        t = np.empty(cap, dtype=np.float64)
        m = np.empty(cap, dtype=np.int32)
        rc = lib.as_gen_trace(seed, rates.shape[0], rates.ctypes.data, cv, duration, cap,
                              t.ctypes.data, m.ctypes.data, ctypes.byref(n))
        if rc == 0:
            return t[: n.value].copy(), m[: n.value].copy()
        if rc != -2:
            raise ValueError(f"as_gen_trace rc={rc}")
        cap = n.value
    raise RuntimeError("as_gen_trace: capacity retry failed")


def trace_windowed(seed: int, rates, cvs, window: float):
    """Non-stationary trace: rates[m][w], cvs[m][w] per window of `window`
    seconds.  Returns (t float64[n], model int32[n])."""
    lib = _load()
    rates = np.ascontiguousarray(rates, dtype=np.float64)
    cvs = np.ascontiguousarray(cvs, dtype=np.float64)
    if rates.ndim != 2 or rates.shape != cvs.shape:
        raise ValueError("rates and cvs must be [n_models][n_windows] arrays of one shape")
    if not (np.isfinite(rates).all() and np.isfinite(cvs).all() and math.isfinite(window)):
        raise ValueError("rates, cvs and window must be finite")
    M, Wn = rates.shape
    lam_t = float(rates.sum()) * window
    cap = int(lam_t + 12.0 * max(float(cvs.max(initial=1.0)), 1.0) * math.sqrt(lam_t + 1.0) + 1024)
    n = ctypes.c_int64(0)
    for _ in range(3):
        t = np.empty(cap, dtype=np.float64)
        m = np.empty(cap, dtype=np.int32)
        rc = lib.as_gen_trace_windowed(seed, M, Wn, float(window), rates.ctypes.data, cvs.ctypes.data,
                                       cap, t.ctypes.data, m.ctypes.data, ctypes.byref(n))
        if rc == 0:
            return t[: n.value].copy(), m[: n.value].copy()
        if rc != -2:
            raise ValueError(f"as_gen_trace_windowed rc={rc}")
        cap = n.value
    raise RuntimeError("as_gen_trace_windowed: capacity retry failed")


def traces(specs, threads=None):
    """Many independent traces in parallel (ctypes releases the GIL).
    specs: iterable of (seed, rates, cv, duration).  Returns a list of (t, model)."""
    specs = list(specs)
    nthreads = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(nthreads) as ex:
        return list(ex.map(lambda s: trace(*s), specs))


def permutations(seed: int, purpose: int, first_index: int, count: int, n: int) -> np.ndarray:
    lib = _load()
    lib.as_gen_permutations.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                        ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p]
    lib.as_gen_permutations.restype = ctypes.c_int
    out = np.empty((count, n), dtype=np.int32)
    rc = lib.as_gen_permutations(seed, purpose, first_index, count, n, out.ctypes.data)
    if rc != 0:
        raise ValueError(f"as_gen_permutations rc={rc}")
    return out
