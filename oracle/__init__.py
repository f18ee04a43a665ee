"""Oracle for the batched serving simulator -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or runs anything here, and this
package imports nothing from the product; the two share only the seeded input
generator module, which holds no simulator arithmetic.

Contents:
  sim_oracle.c   plain sequential C simulator (one job at a time)
  brute.py       event-driven simulator with explicit per-stage FIFO queues,
                 for tiny traces (an independent formulation of the same model)
  greedy.py      the paper's Alg. 1 (simulator-guided greedy selection, beam 1)
                 and the reduced Alg. 2 over a list of uniform partitions, both
                 scoring candidates with the C oracle
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_BUILD = os.path.join(_HERE, "_build")
LIB_PATH = os.path.join(_BUILD, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "sim_oracle.c")

CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-Wall", "-Wextra",
          "-shared", "-fPIC"]


def build(src: str = SRC_PATH, out: str = LIB_PATH) -> str:
    """Compile the C oracle with gcc (no FMA contraction, no fast-math)."""
    os.makedirs(os.path.dirname(out), exist_ok=True)
    tmp = out + ".tmp"
    subprocess.run(["gcc", *CFLAGS, "-o", tmp, src], check=True)
    os.replace(tmp, out)
    return out


class OracleLib:
    """ctypes handle on a compiled oracle library (the committed one, or a
    mutated copy compiled by a test)."""

    def __init__(self, path: str = LIB_PATH):
        if not os.path.exists(path):
            raise FileNotFoundError(f"oracle library {path} is not built; run oracle.build()")
        self.path = path
        self._lib = ctypes.CDLL(path)
        f = self._lib.oracle_simulate_job
        P = ctypes.c_void_p
        f.argtypes = [ctypes.c_int64, P, P, ctypes.c_int32, P, ctypes.c_int32, P,
                      ctypes.c_int32, P, ctypes.c_int32, P, P, ctypes.c_double, P, P, P]
        f.restype = ctypes.c_int
        self._fn = f
        g = getattr(self._lib, "oracle_simulate_job_stats", None)
        if g is not None:
            g.argtypes = f.argtypes + [P, P]
            g.restype = ctypes.c_int
        self._fn_stats = g
        h = getattr(self._lib, "oracle_simulate_job_batched", None)
        if h is not None:
            h.argtypes = f.argtypes[:13] + [ctypes.c_int32, ctypes.c_double, P, P, P, P]
            h.restype = ctypes.c_int
        self._fn_batched = h

    def simulate_job(self, t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask,
                     slo_scale, want_finish=False):
        """Simulate one job.  Returns (served, (h, fin_sum), finish or None).

        t: float64[n]; model: int32[n]; d_single: float64[M]; cfg_stages: int32[C];
        stage_lat: float64[M, C, Smax]; group_cfg: int32[G]; host_mask: uint64[M].
        """
        t = np.ascontiguousarray(t, dtype=np.float64)
        model = np.ascontiguousarray(model, dtype=np.int32)
        d_single = np.ascontiguousarray(d_single, dtype=np.float64)
        cfg_stages = np.ascontiguousarray(cfg_stages, dtype=np.int32)
        stage_lat = np.ascontiguousarray(stage_lat, dtype=np.float64)
        group_cfg = np.ascontiguousarray(group_cfg, dtype=np.int32)
        host_mask = np.ascontiguousarray(host_mask, dtype=np.uint64)
        n = t.shape[0]
        M, C, S = stage_lat.shape
        assert model.shape == (n,) and d_single.shape == (M,) and cfg_stages.shape == (C,)
        assert host_mask.shape == (M,)
        served = np.zeros(1, dtype=np.int64)
        digest = np.zeros(2, dtype=np.uint64)
        finish = np.empty(n, dtype=np.float64) if want_finish else None
        rc = self._fn(n, t.ctypes.data, model.ctypes.data, M, d_single.ctypes.data, C,
                      cfg_stages.ctypes.data, S, stage_lat.ctypes.data, group_cfg.shape[0],
                      group_cfg.ctypes.data, host_mask.ctypes.data, float(slo_scale),
                      served.ctypes.data, digest.ctypes.data,
                      finish.ctypes.data if finish is not None else None)
        if rc != 0:
            raise ValueError(f"oracle_simulate_job rejected its arguments (rc={rc})")
        return int(served[0]), (int(digest[0]), int(digest[1])), finish

    def simulate_job_stats(self, t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask,
                           slo_scale):
        """simulate_job plus the fast heuristic's statistics.  Returns (served,
        (h, fin_sum), model_served int64[M], group_busy float64[G])."""
        t = np.ascontiguousarray(t, dtype=np.float64)
        model = np.ascontiguousarray(model, dtype=np.int32)
        d_single = np.ascontiguousarray(d_single, dtype=np.float64)
        cfg_stages = np.ascontiguousarray(cfg_stages, dtype=np.int32)
        stage_lat = np.ascontiguousarray(stage_lat, dtype=np.float64)
        group_cfg = np.ascontiguousarray(group_cfg, dtype=np.int32)
        host_mask = np.ascontiguousarray(host_mask, dtype=np.uint64)
        n = t.shape[0]
        M, C, S = stage_lat.shape
        G = group_cfg.shape[0]
        served = np.zeros(1, dtype=np.int64)
        digest = np.zeros(2, dtype=np.uint64)
        ms = np.zeros(M, dtype=np.int64)
        busy = np.zeros(G, dtype=np.float64)
        rc = self._fn_stats(n, t.ctypes.data, model.ctypes.data, M, d_single.ctypes.data, C,
                            cfg_stages.ctypes.data, S, stage_lat.ctypes.data, G,
                            group_cfg.ctypes.data, host_mask.ctypes.data, float(slo_scale),
                            served.ctypes.data, digest.ctypes.data, None, ms.ctypes.data,
                            busy.ctypes.data)
        if rc != 0:
            raise ValueError(f"oracle_simulate_job_stats rejected its arguments (rc={rc})")
        return int(served[0]), (int(digest[0]), int(digest[1])), ms, busy

    def simulate_job_batched(self, t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask,
                             slo_scale, max_batch, beta):
        """Dynamic batching (Sec. 6.5).  Returns (served, (h, fin_sum), finish
        float64[n], batch int32[n]) -- h is the order-free digest of the batched
        variant (sum of mix(i) over served requests)."""
        t = np.ascontiguousarray(t, dtype=np.float64)
        model = np.ascontiguousarray(model, dtype=np.int32)
        d_single = np.ascontiguousarray(d_single, dtype=np.float64)
        cfg_stages = np.ascontiguousarray(cfg_stages, dtype=np.int32)
        stage_lat = np.ascontiguousarray(stage_lat, dtype=np.float64)
        group_cfg = np.ascontiguousarray(group_cfg, dtype=np.int32)
        host_mask = np.ascontiguousarray(host_mask, dtype=np.uint64)
        n = t.shape[0]
        M, C, S = stage_lat.shape
        served = np.zeros(1, dtype=np.int64)
        digest = np.zeros(2, dtype=np.uint64)
        finish = np.empty(n, dtype=np.float64)
        batch = np.empty(n, dtype=np.int32)
        rc = self._fn_batched(n, t.ctypes.data, model.ctypes.data, M, d_single.ctypes.data, C,
                              cfg_stages.ctypes.data, S, stage_lat.ctypes.data, group_cfg.shape[0],
                              group_cfg.ctypes.data, host_mask.ctypes.data, float(slo_scale), int(max_batch),
                              float(beta), served.ctypes.data, digest.ctypes.data, finish.ctypes.data,
                              batch.ctypes.data)
        if rc != 0:
            raise ValueError(f"oracle_simulate_job_batched rejected its arguments (rc={rc})")
        return int(served[0]), (int(digest[0]), int(digest[1])), finish, batch

    def simulate_placements(self, t, model, d_single, cfg_stages, stage_lat, group_cfg,
                            host_mask, slo_scale, finish_jobs=(), threads=None):
        """Every placement x every scale (job = p * K + k), like the product's
        batched call.  Returns served[P*K], digest[P*K, 2], {job: finish}.

        Jobs are independent; they run on a thread pool (ctypes releases the
        GIL), each job exactly as simulate_job runs it."""
        group_cfg = np.asarray(group_cfg, dtype=np.int32)
        host_mask = np.asarray(host_mask, dtype=np.uint64)
        scales = np.atleast_1d(np.asarray(slo_scale, dtype=np.float64))
        P, K = group_cfg.shape[0], scales.shape[0]
        want = set(int(j) for j in finish_jobs)
        served = np.zeros(P * K, dtype=np.int64)
        digest = np.zeros((P * K, 2), dtype=np.uint64)
        fins = {}

        def one(j):
            p, k = divmod(j, K)
            s, d, fin = self.simulate_job(t, model, d_single, cfg_stages, stage_lat,
                                          group_cfg[p], host_mask[p], scales[k],
                                          want_finish=j in want)
            return j, s, d, fin

        nthreads = threads or min(8, os.cpu_count() or 1)
        with ThreadPoolExecutor(nthreads) as ex:
            for j, s, d, fin in ex.map(one, range(P * K)):
                served[j] = s
                digest[j] = d
                if fin is not None:
                    fins[j] = fin
        return served, digest, fins


_default = None


def lib() -> OracleLib:
    """The committed oracle, compiled by build()."""
    global _default
    if _default is None:
        _default = OracleLib(LIB_PATH)
    return _default
