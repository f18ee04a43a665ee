"""MI355X-native batched serving simulator for AlpaServe-style placement search.

Subpackages and modules:
  workload/   seeded synthetic inputs: Gamma arrival traces (C library
              libas_gen.so) and the problem builders for the five workloads
  csrc/       HIP kernels for gfx950 and the C-ABI library libalpaserve_sim.so
  sim.py      thin ctypes binding of the C-ABI (argument marshalling only)
  build.py    compiles the two native libraries in-tree

Importing this package loads nothing native; sim.py loads the HIP library on
first use and raises if it is not built.
"""
