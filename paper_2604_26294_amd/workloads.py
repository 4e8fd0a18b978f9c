"""Named TSP workloads: the shapes one rank sees, with the synthetic-value recipe.

Symbols follow the paper's notation table (Section 4): B micro-batch, S sequence,
h hidden, n_h / n_kv query and key/value heads, d head dim, D parallel degree,
p rank.  ``ffn`` is the MLP intermediate width itself (the paper's F*h).
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int          # B
    seq: int            # S (full sequence; each rank holds S/D tokens)
    hidden: int         # h = n_h * d
    ffn: int            # MLP intermediate width (paper F*h)
    n_heads: int        # n_h
    n_kv_heads: int     # n_kv  (GQA ratio g = n_h / n_kv)
    head_dim: int       # d
    degree: int         # D
    rank: int           # p
    w_std: float = 0.02
    x_std: float = 1.0
    seed: int = 0
    layout: int = 0     # 0 contiguous chunks, 1 zigzag (two chunks of S/(2D) per rank)

    @property
    def s_loc(self) -> int:
        return self.seq // self.degree

    @property
    def layout_name(self) -> str:
        return ("contiguous", "zigzag")[self.layout]

    def with_layout(self, layout: int) -> "Workload":
        return replace(self, layout=layout)

    @property
    def gqa(self) -> int:
        return self.n_heads // self.n_kv_heads

    def at_rank(self, p: int) -> "Workload":
        return replace(self, rank=p)


# The five layer shapes of the study (contiguous sequence chunks; the last rank
# carries the heaviest causal chunk).
TINY = Workload("tiny-h256-S256-D2", 1, 256, 256, 688, 4, 4, 64, 2, 1)
L7B_8K = Workload("7b-h4096-S8192-D8", 1, 8192, 4096, 11008, 32, 32, 128, 8, 7)
L7B_64K = Workload("7b-h4096-S65536-D8", 1, 65536, 4096, 11008, 32, 32, 128, 8, 7)
L70B_GQA = Workload("70b-gqa-h8192-S32768-D8", 1, 32768, 8192, 28672, 64, 8, 128, 8, 7,
                    w_std=0.015)
L13B_B4 = Workload("13b-h5120-S16384-D4-B4", 4, 16384, 5120, 13824, 40, 40, 128, 4, 0)

ALL = (TINY, L7B_8K, L7B_64K, L70B_GQA, L13B_B4)
BY_NAME = {w.name: w for w in ALL}
