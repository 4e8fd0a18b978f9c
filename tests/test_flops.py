"""FLOP accounting of one rank's layer forward against the paper's closed forms
(Section 4, FLOPs and parameter count; Appendix C reference model)."""
import json
import os

import pytest

from paper_2604_26294_amd import flops as F
from paper_2604_26294_amd.workloads import ALL, L7B_64K, Workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")


def test_reference_7b_parameter_count():
    ref = json.load(open(GOLDEN))["reference_7b_model"]
    g = ref["n_heads"] / ref["n_kv_heads"]
    total = ref["layers"] * F.params_per_layer(ref["hidden"], ref["ffn_factor"], g)
    assert abs(total - ref["total_params_approx"]) <= ref["rounding"]
    # P_attn + P_mlp with MHA is (4 + 3F) h^2 as the appendix states
    assert F.params_per_layer(4096, 4, 1.0) == (4 + 3 * 4) * 4096 ** 2


@pytest.mark.parametrize("wl", ALL, ids=lambda w: w.name)
def test_rank_sum_reproduces_paper_layer_flops(wl):
    """Summed over ranks: MLP + projections equal (4(1+1/g) + 6F) B S h^2 exactly, and
    the attention core equals the causal half (with diagonal) of 4 B S^2 h."""
    per = [F.rank_flops(wl, p) for p in range(wl.degree)]
    g = wl.n_heads / wl.n_kv_heads
    f = wl.ffn / wl.hidden
    b, s, h = wl.batch, wl.seq, wl.hidden
    dense = sum(r.mlp + r.proj for r in per)
    assert dense == pytest.approx((4 * (1 + 1 / g) + 6 * f) * b * s * h * h, rel=1e-12)
    core = sum(r.attn_core for r in per)
    assert core == pytest.approx(4 * b * h * s * (s + 1) / 2, rel=1e-12)
    # the paper's non-causal F_layer counts the full S^2 square
    full_sq = F.paper_layer_flops(wl) - (4 * (1 + 1 / g) + 6 * f) * b * s * h * h
    assert full_sq == pytest.approx(4 * b * s * s * h, rel=1e-12)


def test_rank_imbalance_and_target_config():
    per = [F.rank_flops(L7B_64K, p).total for p in range(8)]
    assert all(a < b for a, b in zip(per, per[1:]))          # later ranks see longer prefixes
    r7 = F.rank_flops(L7B_64K, 7)
    assert r7.total == pytest.approx(11562.1e9, rel=1e-4)
    assert r7.attn_core / r7.total == pytest.approx(0.713, abs=0.002)
    assert F.step_attn_core_flops(L7B_64K) * 8 == pytest.approx(r7.attn_core, rel=1e-12)


def test_causal_pairs_brute_force():
    for s_loc in (1, 3, 8):
        for p in range(4):
            brute = sum(1 for i in range(s_loc) for j in range((p + 1) * s_loc)
                        if j <= p * s_loc + i)
            assert F.causal_pairs(s_loc, p) == brute


def test_algorithmic_bytes_closed_form():
    """Weights of all D shards once, (2 h n_h d + 2 h n_kv d + 3 h F) x 2 B; the K/V prefix
    once, 2 B (p+1) S_loc n_kv d x 2 B; x (bf16) and Y (fp32)."""
    from paper_2604_26294_amd.workloads import L7B_8K
    for wl, kv_mb in ((L7B_8K, 134.2), (L7B_64K, 1073.7)):
        total = F.rank_algorithmic_bytes(wl)
        weights = 2 * (2 * 4096 * 4096 + 2 * 4096 * 4096 + 3 * 4096 * 11008)
        assert F.rank_weight_bytes(wl) == weights
        assert weights / 1e6 == pytest.approx(404.8, abs=0.05)
        kv = 2 * wl.batch * (wl.rank + 1) * wl.s_loc * wl.n_kv_heads * wl.head_dim * 2
        assert kv / 1e6 == pytest.approx(kv_mb, abs=0.05)
        assert total == weights + kv + wl.s_loc * 4096 * 6


def test_zigzag_pairs_brute_force_and_balance():
    """A zigzag shard's pair count, by brute force over its positions, equals the closed
    form for every rank, and summed over ranks gives the causal half of the square."""
    from paper_2604_26294_amd.workloads import TINY
    for degree, s_c in ((1, 3), (2, 4), (4, 2)):
        seq = 2 * degree * s_c
        total = 0
        for p in range(degree):
            pos = [p * s_c + i for i in range(s_c)] + \
                  [(2 * degree - 1 - p) * s_c + i for i in range(s_c)]
            brute = sum(1 for t in pos for j in range(seq) if j <= t)
            assert F.causal_pairs_zigzag(2 * s_c, degree) == brute
            total += brute
        assert total == seq * (seq + 1) // 2
    zz = TINY.with_layout(1)
    assert F.rank_flops(zz, 0).total == F.rank_flops(zz, 1).total


@pytest.mark.parametrize("wl", ALL, ids=lambda w: w.name)
def test_bench_kernel_classes_sum_to_rank_flops(wl):
    """The benchmark's per-kernel-class FLOPs over one layer call (whatever the number of
    launches that carry them) add up to the rank's algorithmic count."""
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import bench
    kf = bench.kernel_flops(wl)
    rf = F.rank_flops(wl)
    assert kf["gate_up"] + kf["down"] == pytest.approx(rf.mlp, rel=1e-12)
    assert kf["qkv"] + kf["oproj"] + kf["attn"] == pytest.approx(rf.attn, rel=1e-12)
