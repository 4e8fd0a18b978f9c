"""Pins of the Section 4 cost model (paper_2604_26294_amd.costmodel) against what the
paper prints and against counts taken by other routes: parameter and FLOP counts
from the layer's weight and product shapes, collective volumes from a byte-counting
simulation of ring collectives, and TSP's forward traffic from a simulation of the
Algorithm 1 (broadcast + K/V all-gather) and Algorithm 2 (weight ring) schedules."""
import json
import math
import os

import numpy as np
import pytest

from paper_2604_26294_amd import costmodel as C
from paper_2604_26294_amd import flops
from paper_2604_26294_amd.workloads import ALL

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "paper_constants.json")))
REF = C.reference_7b()
GQA = C.ModelConfig(hidden=1024, layers=4, n_heads=16, n_kv_heads=4, head_dim=64,
                    ffn_factor=3.5, beta_p=2, beta_g=4, n_opt=2, beta_o=4)


# ---- counts from shapes ------------------------------------------------------------

def _weight_shapes(c):
    """(rows, cols) of every weight matrix of one layer, from the model's dimensions."""
    h, qd, kvd = c.hidden, c.n_heads * c.head_dim, c.n_kv_heads * c.head_dim
    fh = int(round(c.ffn_factor * h))
    return [(h, qd), (h, kvd), (h, kvd), (qd, h), (h, fh), (h, fh), (fh, h)]


def _products(c, b, s):
    """(M, N, K) of every dense product of one layer's forward over B S tokens,
    the attention core taken without the causal mask, one pair of products per head."""
    h, d = c.hidden, c.head_dim
    m = b * s
    out = [(m, n, k) for (k, n) in _weight_shapes(c)]
    out += [(s, s, d)] * (b * c.n_heads)        # Q K^T
    out += [(s, d, s)] * (b * c.n_heads)        # P V
    return out


@pytest.mark.parametrize("c", [REF, GQA], ids=["ref7b", "gqa"])
def test_parameter_count_from_weight_shapes(c):
    assert c.n_heads * c.head_dim == c.hidden
    assert C.params_layer(c) == pytest.approx(sum(r * k for r, k in _weight_shapes(c)))
    assert C.params_attn(c) == pytest.approx(sum(r * k for r, k in _weight_shapes(c)[:4]))


def test_reference_model_is_8p6_billion():
    g = GOLDEN["reference_7b_model"]
    assert (REF.hidden, REF.layers, REF.n_heads, REF.n_kv_heads, REF.head_dim, REF.ffn_factor) == \
        (g["hidden"], g["layers"], g["n_heads"], g["n_kv_heads"], g["head_dim"], g["ffn_factor"])
    assert abs(C.params_total(REF) - g["total_params_approx"]) <= g["rounding"]
    # the appendix's own form of the count, L (4 + 3F) h^2 for MHA
    assert C.params_total(REF) == REF.layers * (4 + 3 * REF.ffn_factor) * REF.hidden ** 2


@pytest.mark.parametrize("c,b,s", [(REF, 1, 4096), (GQA, 3, 2048)], ids=["ref7b", "gqa"])
def test_layer_flops_from_product_shapes(c, b, s):
    assert C.layer_flops(c, b, s) == pytest.approx(sum(2 * m * n * k for m, n, k in
                                                       _products(c, b, s)), rel=1e-12)


@pytest.mark.parametrize("wl", ALL, ids=lambda w: w.name)
def test_layer_flops_agree_with_per_rank_accounting(wl):
    c = C.from_workload(wl)
    assert C.layer_flops(c, wl.batch, wl.seq) == pytest.approx(flops.paper_layer_flops(wl))
    # the dense projections and MLP of all D ranks add up to the layer's
    per_rank = [flops.rank_flops(wl, p) for p in range(wl.degree)]
    dense = sum(r.mlp + r.proj for r in per_rank)
    h = wl.hidden
    assert dense == pytest.approx((4 * (1 + 1 / c.g) + 6 * c.ffn_factor) * wl.batch * wl.seq * h * h)


# ---- collectives by simulation -----------------------------------------------------

def _ring_allreduce(bufs):
    """Ring reduce-scatter then all-gather over len(bufs) devices on float arrays split
    into D chunks; returns (results, bytes sent per device)."""
    d = len(bufs)
    chunks = [np.array_split(b.copy(), d) for b in bufs]
    sent = [0] * d
    for step in range(d - 1):                    # reduce-scatter
        msgs = [(r, (r - step) % d, chunks[r][(r - step) % d].copy()) for r in range(d)]
        for r, k, data in msgs:
            chunks[(r + 1) % d][k] += data
            sent[r] += data.nbytes
    for step in range(d - 1):                    # all-gather of the reduced chunks
        msgs = [(r, (r + 1 - step) % d, chunks[r][(r + 1 - step) % d].copy()) for r in range(d)]
        for r, k, data in msgs:
            chunks[(r + 1) % d][k] = data
            sent[r] += data.nbytes
    return [np.concatenate(c) for c in chunks], sent


def _ring_allgather(parts):
    d = len(parts)
    have = [{r: parts[r]} for r in range(d)]
    sent = [0] * d
    for step in range(d - 1):
        msgs = [(r, (r - step) % d) for r in range(d)]
        for r, k in msgs:
            have[(r + 1) % d][k] = have[r][k]
            sent[r] += have[r][k].nbytes
    return have, sent


@pytest.mark.parametrize("d", [2, 3, 4, 8])
def test_ring_collective_volumes(d):
    rng = np.random.default_rng(d)
    n = 96 * d                                    # elements, divisible by d
    bufs = [rng.standard_normal(n) for _ in range(d)]
    out, sent = _ring_allreduce(bufs)
    for o in out:
        np.testing.assert_allclose(o, sum(bufs), rtol=1e-12, atol=1e-12)
    nbytes = bufs[0].nbytes
    assert all(v == pytest.approx(C.allreduce_bytes(nbytes, d)) for v in sent)
    parts = [rng.standard_normal(n // d) for _ in range(d)]
    have, sent = _ring_allgather(parts)
    assert all(sorted(h) == list(range(d)) for h in have)
    assert all(v == pytest.approx(C.allgather_bytes(nbytes, d)) for v in sent)
    assert C.broadcast_bytes(nbytes, d) == nbytes


def _tsp_forward_traffic(c, b, s, d):
    """Bytes each rank moves in one TSP layer forward, counted from the schedules:
    attention iteration j broadcasts rank j's packed [W_Q; W_K; W_V; W_O^T] shard
    (every rank moves the whole shard) and all-gathers the local K and V of head group
    j; the MLP ring hands each rank its predecessor's shard at each of D - 1 steps."""
    beta = c.beta_p
    h, qd, kvd = c.hidden, c.n_heads * c.head_dim, c.n_kv_heads * c.head_dim
    attn_shard = (2 * qd * h + 2 * kvd * h) / d * beta
    mlp_shard = 3 * c.ffn_factor * h * h / d * beta
    kv_local = 2 * b * (s // d) * (kvd // d) * beta       # one rank's K and V of a group
    moved = np.zeros(d)
    kv = np.zeros(d)
    for j in range(d):                                    # Algorithm 1 iterations
        moved += attn_shard
        _, sent = _ring_allgather([np.zeros(int(kv_local // 8)) for _ in range(d)])
        kv += np.array(sent, dtype=float)
    held = list(range(d))                                 # Algorithm 2: rank p holds shard p
    seen = [{p} for p in range(d)]
    for t in range(1, d):
        held = [held[(p - 1) % d] for p in range(d)]      # receive from the predecessor
        for p in range(d):
            assert held[p] == (p - t) % d
            seen[p].add(held[p])
        moved += mlp_shard
    assert all(len(x) == d for x in seen)
    return kv, moved


@pytest.mark.parametrize("c,b,s,d", [(REF, 1, 16384, 8), (GQA, 2, 4096, 4)],
                         ids=["ref7b", "gqa"])
def test_tsp_forward_terms_from_schedule(c, b, s, d):
    kv, weights = _tsp_forward_traffic(c, b, s, d)
    act, w = C.comm_terms_fwd("TSP", c, b, s, d)
    assert np.allclose(kv, act, rtol=1e-12)
    assert np.allclose(weights, w, rtol=1e-12)
    assert C.comm_bytes("TSP", "fwd", c, b, s, d) == pytest.approx(act + w)


# ---- relations the section states --------------------------------------------------

CASES = [(REF, 1, 16384, 8), (REF, 4, 4096, 4), (GQA, 2, 8192, 8)]


@pytest.mark.parametrize("c,b,s,d", CASES)
def test_tp_sp_mesh_reduces_to_tp_and_sp(c, b, s, d):
    for ph in C.PHASES:
        assert C.comm_bytes("TP+SP", ph, c, b, s, d, t=d, sigma=1) == \
            pytest.approx(C.comm_bytes("TP", ph, c, b, s, d))
        assert C.comm_bytes("TP+SP", ph, c, b, s, d, t=1, sigma=d) == \
            pytest.approx(C.comm_bytes("SP", ph, c, b, s, d))
    for rc in C.RECOMPUTE:
        assert C.memory_bytes("TP+SP", c, b, s, d, rc, t=d, sigma=1) == \
            pytest.approx(C.memory_bytes("TP", c, b, s, d, rc))
        assert C.memory_bytes("TP+SP", c, b, s, d, rc, t=1, sigma=d) == \
            pytest.approx(C.memory_bytes("SP", c, b, s, d, rc))


@pytest.mark.parametrize("c,b,s,d", CASES)
def test_table_relations(c, b, s, d):
    # DP's forward is free; TSP shares SP's activation term
    assert C.comm_bytes("DP", "fwd", c, b, s, d) == 0
    assert C.comm_terms_fwd("TSP", c, b, s, d)[0] == pytest.approx(
        C.comm_terms_fwd("SP", c, b, s, d)[0])
    # TP's activation term is 4 B S h beta (D-1)/D, twice SP's for MHA
    bsh = b * s * c.hidden * c.beta_p
    assert C.comm_bytes("TP", "fwd", c, b, s, d) == pytest.approx(4 * bsh * (d - 1) / d)
    # recomputation: TP grows by half, DP not at all
    g = GOLDEN["tp_full_recompute_overhead"]
    tp2 = C.comm_bytes("TP", "fwd+bwd", c, b, s, d)
    tp3 = C.comm_bytes("TP", "fwd+bwd+recomp", c, b, s, d)
    assert tp3 / tp2 - 1 == pytest.approx(g["overhead"])
    assert tp2 == pytest.approx(g["fwd_bwd_coeff"] * bsh * (d - 1) / d)
    assert C.comm_bytes("DP", "fwd+bwd", c, b, s, d) == C.comm_bytes("DP", "fwd+bwd+recomp",
                                                                     c, b, s, d)
    # TSP against SP with the gradient exchange upper-bounded: the difference is the
    # weight movement, once per pass
    w = C.comm_terms_fwd("TSP", c, b, s, d)[1]
    assert C.comm_bytes("TSP", "fwd+bwd", c, b, s, d, tsp_grad="allreduce") - \
        C.comm_bytes("SP", "fwd+bwd", c, b, s, d) == pytest.approx(2 * w)
    # the tight reduce-to-owner volume is half the all-reduce
    pl = C.params_layer(c) * c.beta_g
    assert C.comm_bytes("TSP", "fwd+bwd", c, b, s, d, tsp_grad="allreduce") - \
        C.comm_bytes("TSP", "fwd+bwd", c, b, s, d, tsp_grad="reduce") == \
        pytest.approx(pl * (d - 1) / d)
    assert C.comm_bytes("TSP", "fwd+bwd", c, b, s, d) == \
        pytest.approx(C.comm_bytes("TSP", "fwd+bwd", c, b, s, d, tsp_grad="reduce"))
    assert C.comm_bytes("TSP", "fwd+bwd+recomp", c, b, s, d) == \
        pytest.approx(C.comm_bytes("TSP", "fwd+bwd+recomp", c, b, s, d, tsp_grad="allreduce"))


@pytest.mark.parametrize("c,b,s,d", CASES)
def test_memory_and_flop_sharding(c, b, s, d):
    for rc in C.RECOMPUTE:
        dp = C.memory_bytes("DP", c, b, s, d, rc)
        tsp = C.memory_bytes("TSP", c, b, s, d, rc)
        tp = C.memory_bytes("TP", c, b, s, d, rc)
        sp = C.memory_bytes("SP", c, b, s, d, rc)
        for k in ("params", "grads", "optim", "acts", "total"):
            assert tsp[k] == pytest.approx(dp[k] / d)       # the only 1/D in every class
        for k in ("params", "grads", "optim"):
            assert tp[k] == pytest.approx(tsp[k]) and sp[k] == pytest.approx(dp[k])
        assert tp["acts"] == pytest.approx(dp["acts"]) and sp["acts"] == pytest.approx(tsp["acts"])
    f = C.layer_flops(c, b, s)
    assert C.flops_per_device("DP", c, b, s, d) == f
    for st in ("TP", "SP", "TSP"):
        assert C.flops_per_device(st, c, b, s, d) == pytest.approx(f / d)
    assert C.flops_per_device("TP+SP", c, b, s, d, t=2, sigma=d // 2) == pytest.approx(f / d)


def test_activation_memory_attention_matrices():
    """Without recomputation the extra memory over the selective regime is the n_h
    S x S score, softmax and dropout-mask matrices per layer: (2 beta_P + 1) bytes
    per element."""
    for c, b, s in ((REF, 1, 8192), (GQA, 2, 1024)):
        extra = C.activation_bytes(c, b, s, "none") - C.activation_bytes(c, b, s, "sel")
        assert extra == pytest.approx(c.layers * b * c.n_heads * s * s * (2 * c.beta_p + 1))
        assert C.activation_bytes(c, b, s, "full") == c.layers * b * s * c.hidden * c.beta_p
    with pytest.raises(ValueError):
        C.activation_bytes(REF, 1, 1, "some")


def test_breakeven_is_8h_for_mha_f4():
    g = GOLDEN["tsp_tp_breakeven"]
    assert REF.g == g["g"] and REF.ffn_factor == g["ffn_factor"]
    assert C.breakeven_tokens(REF) == pytest.approx(g["tokens_per_hidden"] * REF.hidden)
    # the asymptotic comparison flips exactly there, and matches (4 + 3F) h < 2 B S
    bs0 = g["tokens_per_hidden"] * REF.hidden
    for bs in (bs0 // 2, bs0 - 1, bs0, bs0 + 1, 4 * bs0):
        assert C.tsp_beats_tp_large_d(REF, 1, bs) == (bs > bs0)
        assert C.tsp_beats_tp_large_d(REF, 1, bs) == ((4 + 3 * REF.ffn_factor) * REF.hidden < 2 * bs)


@pytest.mark.parametrize("c", [REF, GQA], ids=["ref7b", "gqa"])
@pytest.mark.parametrize("d", [2, 4, 8, 64])
def test_breakeven_at_finite_degree(c, d):
    """At the finite-D break-even token count the two forward volumes are equal, TSP
    is cheaper above it and dearer below it; as D grows it tends to the large-D value."""
    bs = C.breakeven_tokens(c, d)
    tsp = lambda n: C.comm_bytes("TSP", "fwd", c, 1, n, d)
    tp = lambda n: C.comm_bytes("TP", "fwd", c, 1, n, d)
    assert tsp(bs) == pytest.approx(tp(bs), rel=1e-12)
    assert tsp(1.01 * bs) < tp(1.01 * bs) and tsp(0.99 * bs) > tp(0.99 * bs)
    big = C.breakeven_tokens(c, 1 << 20)
    assert big == pytest.approx(C.breakeven_tokens(c), rel=1e-5)
    if c.g > 1:   # general GQA form P_L < 2 B S h (2 - 1/g)
        lim = C.params_layer(c) / (2 * c.hidden * (2 - 1 / c.g))
        assert C.breakeven_tokens(c) == pytest.approx(lim)


def test_bad_arguments_raise():
    with pytest.raises(ValueError):
        C.comm_bytes("ZeRO", "fwd", REF, 1, 1024, 8)
    with pytest.raises(ValueError):
        C.comm_bytes("TP", "bwd", REF, 1, 1024, 8)
    with pytest.raises(ValueError):
        C.comm_bytes("TP+SP", "fwd", REF, 1, 1024, 8, t=3, sigma=2)
    with pytest.raises(ValueError):
        C.comm_bytes("TSP", "fwd+bwd", REF, 1, 1024, 8, tsp_grad="other")


def test_report_runs(capsys):
    C.main(["--seq", "16384", "--degree", "8", "--tp", "2"])
    out = capsys.readouterr().out
    assert "L*P_L=8.59 B" in out and "break-even: B S = 32768" in out
    assert not math.isnan(C.breakeven_tokens(REF, 8))
