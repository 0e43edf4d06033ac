"""Sequence-bucketed LSTM/GRU training hot path for AMD Instinct MI355X (gfx950).

Khomenko et al., "Accelerating Recurrent Neural Network Training using
Sequence Bucketing and Multi-GPU Data Parallelization" (arXiv 1708.05604).

Submodules:
  synth  -- seeded synthetic workloads (lengths, features, labels, parameters,
            shuffle keys); holds none of the method's arithmetic.
  lib    -- ctypes binding of the C-ABI library ``librnnbkt.so`` (the product
            path; every step runs in HIP kernels or the library's host code).
  build  -- compiles the library with hipcc for gfx950.

Importing the package itself loads nothing; ``lib`` loads the shared library
on first use and raises if it is missing.
"""
__version__ = "0.1.0"
