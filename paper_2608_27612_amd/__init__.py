"""MI355X (gfx950) eager multi-resolution substrate discovery (EMR-HyperNEAT, Phase 1).

Submodules:
  emr        ctypes binding of include/emr.h (the HIP library libemr.so)
  workloads  seeded synthetic genomes and substrate layouts
  build      in-tree build of libemr.so with hipcc
"""
