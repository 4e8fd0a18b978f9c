"""MI355X-native per-rank forward of folded Tensor-and-Sequence Parallelism (TSP).

One rank of a TSP group holds S/D tokens of the sequence and visits all D weight
shards of a transformer layer: the attention schedule of the paper's Algorithm 1
(broadcast parameter shards, sequence-wise K/V exchange) and the gated ring MLP of
Algorithm 2 (shards circulate, partial outputs accumulate locally).

Importing this package loads nothing native.  The compute entry points live in
:mod:`paper_2604_26294_amd.tsp`, a thin ctypes binding over ``libtsp.so`` (the
hand-written HIP kernels for gfx950); that module raises if the library is missing.
"""

__all__ = ["inputs", "workloads", "flops", "costmodel"]
