"""In-tree builds of the package's native libraries.

  libas_gen.so         workload generator (gcc, plain C, host only)
  libalpaserve_sim.so  HIP kernels for gfx950 + C-ABI (hipcc)
  libas_probe.so       fp64 VALU and device-memory read probes (hipcc; bench.py only)

Both land in paper_2302_11665_amd/_build/.  Every call recompiles.
"""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
BUILD = os.path.join(PKG, "_build")
INCLUDE = os.path.join(ROOT, "include")

GEN_SRC = os.path.join(PKG, "workload", "gen.c")
GEN_LIB = os.path.join(BUILD, "libas_gen.so")

CSRC = os.path.join(PKG, "csrc")
SIM_API_SRC = os.path.join(CSRC, "sim_api.hip")
SIM_LAUNCH_SRC = os.path.join(CSRC, "sim_launch.hip")
SIM_SEARCH_SRC = os.path.join(CSRC, "sim_search.hip")
SIM_STATS_SRC = os.path.join(CSRC, "sim_stats.hip")
SIM_MULTI_SRC = os.path.join(CSRC, "sim_multi.hip")
SIM_ALG2_SRC = os.path.join(CSRC, "sim_alg2.hip")
SIM_BATCH_SRC = os.path.join(CSRC, "sim_batch.hip")
SIM_SPEC_SRC = os.path.join(CSRC, "sim_spec.hip")
LANE_WIDTHS = (1, 2, 4, 8, 16, 32, 64)  # one launcher translation unit per width
SIM_LIB = os.path.join(BUILD, "libalpaserve_sim.so")
PROBE_SRC = os.path.join(CSRC, "peak_probe.hip")
PROBE_LIB = os.path.join(BUILD, "libas_probe.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# -ffp-contract=off: no FMA contraction (the deadline t + scale*d and the stage
# chain must round exactly like the separate IEEE operations they are).
# -packed-fp32-ops off: the compiler may not form v_pk_*_f32 on its own.
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fPIC", "-shared", "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument",
]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build_gen() -> str:
    os.makedirs(BUILD, exist_ok=True)
    tmp = GEN_LIB + ".tmp"
    _run(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-Wall", "-Wextra",
          "-shared", "-fPIC", "-I", INCLUDE, "-o", tmp, GEN_SRC, "-lm"])
    os.replace(tmp, GEN_LIB)
    return GEN_LIB


def build_sim(extra_flags=(), jobs=None) -> str:
    """Compile the launcher units (one per lane width) and the API unit in
    parallel, then link the shared library."""
    from concurrent.futures import ThreadPoolExecutor
    obj_dir = os.path.join(BUILD, "obj")
    os.makedirs(obj_dir, exist_ok=True)
    compile_flags = [f for f in HIP_FLAGS if f != "-shared"]
    units = [(SIM_API_SRC, os.path.join(obj_dir, "sim_api.o"), []),
             (SIM_SEARCH_SRC, os.path.join(obj_dir, "sim_search.o"), []),
             (SIM_STATS_SRC, os.path.join(obj_dir, "sim_stats.o"), []),
             (SIM_ALG2_SRC, os.path.join(obj_dir, "sim_alg2.o"), []),
             (SIM_BATCH_SRC, os.path.join(obj_dir, "sim_batch.o"), []),
             (SIM_SPEC_SRC, os.path.join(obj_dir, "sim_spec.o"), []),
             (SIM_MULTI_SRC, os.path.join(obj_dir, "sim_multi.o"), [])]
    for w in LANE_WIDTHS:
        units.append((SIM_LAUNCH_SRC, os.path.join(obj_dir, f"sim_launch_w{w}.o"), [f"-DAS_W={w}"]))

    def compile_one(u):
        src, obj, defs = u
        _run([HIPCC, *compile_flags, *extra_flags, *defs, "-I", INCLUDE, "-I", CSRC, "-c", "-o", obj, src])
        return obj

    n = jobs or min(len(units), os.cpu_count() or 1)
    with ThreadPoolExecutor(n) as ex:
        objs = list(ex.map(compile_one, units))
    tmp = SIM_LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, SIM_LIB)
    return SIM_LIB


def build_probe() -> str:
    """The peak probes: a stand-alone library that bench.py loads."""
    os.makedirs(BUILD, exist_ok=True)
    tmp = PROBE_LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-o", tmp, PROBE_SRC])
    os.replace(tmp, PROBE_LIB)
    return PROBE_LIB


def build_all() -> None:
    build_gen()
    build_sim()
    build_probe()
