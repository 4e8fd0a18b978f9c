"""Helpers for the GPU parity tests: seeded inputs, oracle runs, tolerance checks.

The tolerance is the one the build targets for bf16 operands with fp32
accumulation, applied per output tensor:
    max |gpu - ref| / max |ref| <= 2e-2   and   cosine(gpu, ref) >= 0.9999.
"""
from __future__ import annotations

import numpy as np

from oracle import tsp_oracle as O
from paper_2604_26294_amd import inputs as I
from paper_2604_26294_amd.workloads import Workload

MAX_REL = 2e-2
MIN_COS = 0.9999

# Small workloads the oracle finishes in seconds; each spans several GEMM and
# attention tiles and has ragged tails (S/D vs the 128-query tile and 256-row
# GEMM tile; F/D vs the 128-column tile and the 64-wide contraction step).
MID_GQA64 = Workload("mid-gqa-d64", 2, 768, 512, 1376, 8, 4, 64, 4, 0, w_std=0.05)
MID_MHA128 = Workload("mid-mha-d128", 1, 1280, 1024, 2768, 8, 8, 128, 2, 1, w_std=0.03)
MID_GQA8 = Workload("mid-gqa8-d128", 1, 512, 2048, 5504, 16, 2, 128, 2, 1, w_std=0.02)
SINGLE = Workload("single-rank-d1", 1, 320, 512, 1024, 4, 2, 128, 1, 0, w_std=0.04)
# An odd degree: grouped two steps at a time, the last step forms a group on its own.
ODD3 = Workload("odd-degree-d3", 1, 768, 384, 1152, 6, 3, 64, 3, 2, w_std=0.05)
# More shards than one grouped launch holds: the default grouping makes two groups of 8.
DEG16 = Workload("degree-d16", 1, 1024, 1024, 2048, 16, 16, 64, 16, 13, w_std=0.04)
# Many attention work items per shard (5 query tiles x 2 heads x 10 batch entries): the
# launch plan pairs query tiles (5 tiles: pairs (0, 4), (1, 3) and tile 2 alone; in the
# zigzag layout 6 tiles, pairs across the two segments); GQA g = 2.
SUBL = Workload("sub-launch-b10", 10, 5120, 512, 1024, 8, 4, 64, 4, 2, w_std=0.05)
# the gate+up product of a group of 8 shards in 256 x 128 tiles (at least 4 rounds on 256
# CUs: 16 x 8 x 8 = 1024 tiles) with a ragged F/D = 1000
MLP_BIG = Workload("mlp-big-fd1000", 1, 32768, 512, 8000, 8, 8, 64, 8, 7, w_std=0.04)


def metrics(got, ref):
    g = np.asarray(got, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    max_rel = float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-300))
    cos = float(g @ r / max(np.linalg.norm(g) * np.linalg.norm(r), 1e-300))
    return max_rel, cos


def assert_close(got, ref, what="", max_rel=MAX_REL, min_cos=MIN_COS):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    mr, cos = metrics(got, ref)
    assert mr <= max_rel and cos >= min_cos, f"{what}: max_rel={mr:.3e} cos={cos:.6f}"
    return mr, cos


def gen(wl: Workload):
    return I.make_x_full(wl), I.make_weights(wl)


RISING_ROWS = 128  # the first key tile of the attention kernel


def stress_inputs(wl: Workload, kind: str):
    """Seeded inputs of wl; kind "peaky" multiplies W_Q by 8 (exact in bf16), which makes
    the softmax rows peaky (the attention stress input); "rising" also divides the
    token rows at sequence positions below RISING_ROWS by 16 (exact), so that the logits
    of the first keys are small and a row's maximum grows by tens of log2 units after
    its first key tile."""
    x_bits, w_bits = gen(wl)
    if kind in ("peaky", "rising"):
        w_bits = dict(w_bits)
        w_bits["wq"] = I.round_to_bf16_bits(I.bf16_bits_to_f32(w_bits["wq"]) * np.float32(8.0))
    if kind == "rising":
        x_bits = x_bits.copy()
        x_bits[:, :RISING_ROWS] = I.round_to_bf16_bits(
            I.bf16_bits_to_f32(x_bits[:, :RISING_ROWS]) * np.float32(0.0625))
    return x_bits, w_bits


def f64(bits):
    return I.bf16_bits_to_f64(bits)


def oracle_blocks(wl: Workload, x_bits, w_bits, p, blocks=("mlp", "attn", "layer"),
                  scale=None):
    """fp64 outputs of rank p: the MLP and attention blocks on x, and the layer
    (``scale``: softmax scale, None = 1/sqrt(d))."""
    x = f64(x_bits)
    w = {k: f64(v) for k, v in w_bits.items()}
    D = wl.degree
    hs, ks, d = wl.n_heads // D, wl.n_kv_heads // D, wl.head_dim
    zz = wl.layout == 1
    if zz:
        chunks = [x[:, O.zigzag_positions(wl.seq, D, q)] for q in range(D)]
    else:
        chunks = [I.local_chunk(x, q, D) for q in range(D)]
    attn_sh = [I.attn_shard_packed(w, r, D, wl.n_heads, wl.n_kv_heads, d) for r in range(D)]
    mlp_sh = [I.mlp_shard(w, j, D) for j in range(D)]
    w1s, w3s, w2s = [m[0] for m in mlp_sh], [m[1] for m in mlp_sh], [m[2] for m in mlp_sh]
    out = {}
    if "mlp" in blocks:
        out["mlp"] = O.mlp_rank(chunks[p], w1s, w3s, w2s, p)
    if "attn" in blocks:
        if zz:
            kv = [O.gather_kv_zigzag(chunks, attn_sh[r], hs, ks, d) for r in range(D)]
            out["attn"] = O.attn_rank_zigzag(chunks[p], attn_sh, kv, p, wl.n_heads,
                                             wl.n_kv_heads, d, scale)
        else:
            kv = [O.gather_kv(chunks, attn_sh[r], hs, ks, d) for r in range(D)]
            out["attn"] = O.attn_rank(chunks[p], attn_sh, kv, p, wl.n_heads, wl.n_kv_heads, d,
                                      scale)
    if "layer" in blocks:
        fn = O.layer_rank_zigzag if zz else O.layer_rank
        out["layer"] = fn(chunks, attn_sh, w1s, w3s, w2s, p, wl.n_heads, wl.n_kv_heads, d,
                          scale)["y"]
    return out
