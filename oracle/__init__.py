"""Test infrastructure: plain, slow, fp64 CPU oracle for the TSP per-rank layer forward.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The product path (the HIP library and its Python binding) never calls
it, and it shares no code with that path: it reads bf16 values that the seeded input
generator produced and computes everything in float64 with NumPy.

Modules:
  tsp_oracle  -- O1 unsharded layer (the definition), O2 folded per-rank schedule
                 (Algorithms 1 and 2 of the paper, step by step), and the sampled-rows
                 form of attention used to check full-size runs.
  brute       -- O3 scalar-loop brute force for micro shapes (no matrix library).
"""
from . import brute, tsp_oracle  # noqa: F401
