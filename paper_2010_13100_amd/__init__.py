"""Tensor Casting sparse-embedding training step on AMD MI355X (gfx950).

Modules:
  tc         -- binding of libtc (include/tc.h): forward gather-reduce, Tensor
                Casting, casted backward gather-reduce, sparse SGD/Adagrad update
  workload   -- seeded synthetic inputs (host, numpy)
  device_fill-- device-side table fill (include/tc_workload.h)
  build      -- compiles the HIP libraries in-tree
"""
