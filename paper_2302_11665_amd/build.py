"""In-tree builds of the package's native libraries.

  libas_gen.so         workload generator (gcc, plain C, host only)
  libalpaserve_sim.so  HIP kernels for gfx950 + C-ABI (hipcc)

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

SIM_SRCS = [os.path.join(PKG, "csrc", "sim_api.hip")]
SIM_LIB = os.path.join(BUILD, "libalpaserve_sim.so")

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


def build_sim(extra_flags=()) -> str:
    os.makedirs(BUILD, exist_ok=True)
    tmp = SIM_LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, *extra_flags, "-I", INCLUDE, "-o", tmp, *SIM_SRCS])
    os.replace(tmp, SIM_LIB)
    return SIM_LIB


def build_all() -> None:
    build_gen()
    build_sim()
