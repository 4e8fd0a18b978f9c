"""Algorithmic FLOP and byte counts of one rank's TSP layer forward.

The paper's FLOP model (Section 4, "FLOPs") counts the dense products of a layer and
ignores softmax, masking and other pointwise work:
    F_attn ~ 4 (1 + 1/g) B S h^2 + 4 B S^2 h,   F_mlp ~ 6 F B S h^2,
with F the FFN expansion factor (so F h is the MLP width).  Per rank this module
counts the same products for the S/D local tokens, and restricts the attention core
to the query/key pairs a causal chunk actually needs: with contiguous chunks rank
p's queries see p S_loc earlier keys plus a causal triangle of its own, p S_loc^2 +
S_loc (S_loc + 1) / 2 pairs per head; a zigzag shard (Algorithm 1) has
(2D-1) S_c^2 + S_c (S_c + 1) for every rank, S_c = S_loc / 2.  Summed over all ranks this is the causal
half (with diagonal) of the paper's 4 B S^2 h term.
"""
from __future__ import annotations

from dataclasses import dataclass

from .workloads import Workload


@dataclass(frozen=True)
class RankFlops:
    mlp: float
    proj: float
    attn_core: float

    @property
    def attn(self) -> float:
        return self.proj + self.attn_core

    @property
    def total(self) -> float:
        return self.mlp + self.proj + self.attn_core


def causal_pairs(s_loc: int, p: int) -> int:
    """Unmasked (query, key) pairs per head for rank p's contiguous chunk."""
    return p * s_loc * s_loc + s_loc * (s_loc + 1) // 2


def causal_pairs_zigzag(s_loc: int, degree: int) -> int:
    """Unmasked pairs per head for a zigzag shard (chunks p and 2D-1-p of S/(2D) tokens):
    (2D-1) S_c^2 + S_c (S_c + 1) with S_c = S_loc / 2, the same for every rank."""
    s_c = s_loc // 2
    return (2 * degree - 1) * s_c * s_c + s_c * (s_c + 1)


def rank_pairs(wl: Workload, p: int) -> int:
    if wl.layout == 1:
        return causal_pairs_zigzag(wl.s_loc, wl.degree)
    return causal_pairs(wl.s_loc, p)


def rank_flops(wl: Workload, p: int | None = None) -> RankFlops:
    p = wl.rank if p is None else p
    b, s_loc, h = wl.batch, wl.s_loc, wl.hidden
    qd = wl.n_heads * wl.head_dim
    kvd = wl.n_kv_heads * wl.head_dim
    mlp = 6.0 * b * s_loc * h * wl.ffn
    proj = 2.0 * b * s_loc * h * (qd + 2 * kvd) + 2.0 * b * s_loc * qd * h
    core = 4.0 * b * wl.n_heads * wl.head_dim * rank_pairs(wl, p)
    return RankFlops(mlp, proj, core)


def step_attn_core_flops(wl: Workload, p: int | None = None) -> float:
    """Attention-core FLOPs of one shard step (H_s = n_h / D heads)."""
    p = wl.rank if p is None else p
    return 4.0 * wl.batch * (wl.n_heads // wl.degree) * wl.head_dim * rank_pairs(wl, p)


def paper_layer_flops(wl: Workload) -> float:
    """The paper's leading-order F_layer (Section 4, equation for F_layer), non-causal."""
    g = wl.n_heads / wl.n_kv_heads
    f = wl.ffn / wl.hidden
    b, s, h = wl.batch, wl.seq, wl.hidden
    return (4 * (1 + 1 / g) + 6 * f) * b * s * h * h + 4 * b * s * s * h


def params_per_layer(hidden: int, ffn_factor: float, gqa: float) -> float:
    """P_L = (2 (1 + 1/g) + 3 F) h^2 (Section 4, parameter count)."""
    return (2 * (1 + 1 / gqa) + 3 * ffn_factor) * hidden * hidden


def rank_weight_bytes(wl: Workload) -> int:
    """bf16 bytes of all D weight shards a rank streams once per layer."""
    h = wl.hidden
    qd = wl.n_heads * wl.head_dim
    kvd = wl.n_kv_heads * wl.head_dim
    return 2 * (2 * qd * h + 2 * kvd * h + 3 * wl.ffn * h)


def rank_algorithmic_bytes(wl: Workload, p: int | None = None) -> int:
    """HBM bytes one rank's layer forward must move at least once: every weight shard
    (bf16), the K/V prefix of keys [0, (p + 1) S_loc) for all kv heads (bf16, read once),
    the local input x (bf16, read) and the fp32 output Y (written)."""
    p = wl.rank if p is None else p
    kv = 2 * wl.batch * (p + 1) * wl.s_loc * wl.n_kv_heads * wl.head_dim * 2
    xy = wl.batch * wl.s_loc * wl.hidden * (2 + 4)
    return rank_weight_bytes(wl) + kv + xy
