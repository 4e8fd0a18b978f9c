"""Pins of the fp64 oracle against what the paper and mathematics fix.

None of these compares the oracle with itself: each check uses an independent
route -- scalar brute force, a hand-derived closed form, an invariant, or the
fold == unsharded identity that the paper's schedules are built to satisfy
(Section 3.1: after visiting all D shards a rank holds the full attention output
for its tokens, and every MLP shard has been applied to its chunk).
"""
import math

import numpy as np
import pytest

from oracle import brute
from oracle import tsp_oracle as O
from paper_2604_26294_amd import inputs as I
from paper_2604_26294_amd.workloads import TINY, Workload


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def _inputs(wl: Workload):
    x = I.bf16_bits_to_f64(I.make_x_full(wl))
    w = {k: I.bf16_bits_to_f64(v) for k, v in I.make_weights(wl).items()}
    return x, w


def _shards(wl, w_bits_or_vals):
    D = wl.degree
    attn = [I.attn_shard_packed(w_bits_or_vals, r, D, wl.n_heads, wl.n_kv_heads, wl.head_dim)
            for r in range(D)]
    mlp = [I.mlp_shard(w_bits_or_vals, j, D) for j in range(D)]
    return attn, [m[0] for m in mlp], [m[1] for m in mlp], [m[2] for m in mlp]


def _micro(n_heads, n_kv, degree, seq=8, d=4, ffn=12, batch=1, seed=3):
    return Workload("micro", batch, seq, n_heads * d, ffn, n_heads, n_kv, d, degree, 0,
                    w_std=0.3, seed=seed)


# ---------------------------------------------------------------------------
# Input generator (shared by both sides; holds no method arithmetic)
# ---------------------------------------------------------------------------

def test_bf16_round_to_nearest_even():
    vals = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.5, 0.0, np.inf,
                     1.0 + 2.0 ** -8 + 2.0 ** -20], dtype=np.float32)
    bits = I.round_to_bf16_bits(vals)
    # 1+2^-8 is a tie between 0x3F80 and 0x3F81 -> even 0x3F80; 1+3*2^-8 ties -> 0x3F82;
    # just above the tie rounds up.
    assert list(bits) == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x0000, 0x7F80, 0x3F81]
    assert np.isnan(I.bf16_bits_to_f32(I.round_to_bf16_bits(np.array([np.nan], np.float32))))[0]
    back = I.bf16_bits_to_f32(bits)
    assert back[0] == 1.0 and back[2] == np.float32(1.0 + 2.0 ** -6)


def test_gaussian_chunking_does_not_change_values(monkeypatch):
    ref = I.gaussian_bf16(0, 5, (37, 29), 0.02)
    monkeypatch.setattr(I, "_CHUNK_ELEMS", 100)
    assert np.array_equal(I.gaussian_bf16(0, 5, (37, 29), 0.02), ref)
    other = I.gaussian_bf16(0, 6, (37, 29), 0.02)
    assert not np.array_equal(other, ref)
    v = I.bf16_bits_to_f64(I.gaussian_bf16(1, 0, (200000,), 0.02))
    assert abs(v.std() - 0.02) < 0.0005 and abs(v.mean()) < 0.0005


# ---------------------------------------------------------------------------
# Hand-derived closed forms (orientation, mask, scale and GQA conventions)
# ---------------------------------------------------------------------------

def test_attention_two_token_closed_form():
    """S=2, h=d=2, one head, default scale 1/sqrt(2).

    x0=[1,0], x1=[0,1]; W_Q=I so q_t=x_t.  W_K=[[1,2],[0,sqrt(2) ln 3]] gives
    k0=[1,0], k1=[2, sqrt(2) ln 3]; scaled scores of query 1 are 0 and ln 3, so its
    softmax weights are 1/4 and 3/4.  Query 0 sees only key 0 (causal).
    W_V=[[1,2],[3,4]] gives v0=[1,3], v1=[2,4]:  o0=[1,3], o1=[1.75,3.75].
    W_O=[[1,0],[1,1]] and the block returns o W_O^T: [1,4] and [1.75,5.5].
    """
    x = np.array([[[1.0, 0.0], [0.0, 1.0]]])
    wq = np.eye(2)
    wk = np.array([[1.0, 2.0], [0.0, math.sqrt(2.0) * math.log(3.0)]])
    wv = np.array([[1.0, 2.0], [3.0, 4.0]])
    wo = np.array([[1.0, 0.0], [1.0, 1.0]])
    expect = np.array([[[1.0, 4.0], [1.75, 5.5]]])
    got = O.attention_full(x, wq, wk, wv, wo, 1, 1)
    assert _rel(got, expect) < 1e-14
    got_b = brute.attention_seq(x[0].tolist(), wq.tolist(), wk.tolist(), wv.tolist(),
                                wo.tolist(), 1, 1)
    assert _rel(got_b, expect[0]) < 1e-14
    got_r = O.attention_rows(x[0], wq, wk, wv, wo, 1, 1, [0, 1])
    assert _rel(got_r, expect[0]) < 1e-14


def test_gqa_head_mapping_closed_form():
    """n_h=4, n_kv=2 (g=2), d=1, h=4, W_Q=0 so every visible key weighs the same.

    Head i reads kv head i//2: heads 0,1 see V column 0, heads 2,3 see V column 1.
    With x0=[1,0,0,0], x1=[0,1,0,0], W_V=[[1,0,0,0],[0,0,0,5]] -> v0=[1,0], v1=[0,0]:
    o at t=1 is the mean of v0, v1 = [0.5, 0]; heads (0,1,2,3) -> [0.5,0.5,0,0].
    W_O=I returns it unchanged.
    """
    x = np.array([[[1.0, 0, 0, 0], [0, 1.0, 0, 0]]])
    wq = np.zeros((4, 4))
    wk = np.ones((2, 4))
    wv = np.array([[1.0, 0, 0, 0], [0, 0, 0, 5.0]])
    wo = np.eye(4)
    got = O.attention_full(x, wq, wk, wv, wo, 4, 2)
    assert _rel(got[0, 1], [0.5, 0.5, 0.0, 0.0]) < 1e-15
    assert _rel(got[0, 0], [1.0, 1.0, 0.0, 0.0]) < 1e-15
    gb = brute.attention_seq(x[0].tolist(), wq.tolist(), wk.tolist(), wv.tolist(),
                             wo.tolist(), 4, 2)
    assert _rel(gb, got[0]) < 1e-15


def test_mlp_closed_form():
    """u=[1,2], W1=[[ln 3, 0]] -> gate pre-activation ln 3, sigmoid(ln 3)=3/4;
    W3=[[0,1]] -> up = 2;  W2=[[1,-2]] (applied untransposed) ->
    y = 0.75 ln3 * 2 * [1,-2] = [1.5 ln 3, -3 ln 3]."""
    u = np.array([[1.0, 2.0]])
    w1 = np.array([[math.log(3.0), 0.0]])
    w3 = np.array([[0.0, 1.0]])
    w2 = np.array([[1.0, -2.0]])
    expect = np.array([[1.5 * math.log(3.0), -3.0 * math.log(3.0)]])
    assert _rel(O.mlp_full(u, w1, w3, w2), expect) < 1e-15
    assert _rel(brute.mlp_seq(u.tolist(), w1.tolist(), w3.tolist(), w2.tolist()), expect) < 1e-15
    assert O.silu(np.array([0.0]))[0] == 0.0
    assert abs(O.silu(np.array([-800.0]))[0]) < 1e-300
    assert O.silu(np.array([40.0]))[0] == pytest.approx(40.0, rel=1e-15)


# ---------------------------------------------------------------------------
# O1 (NumPy) against O3 (scalar loops) on micro shapes
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n_heads,n_kv", [(2, 2), (2, 1), (4, 2)])
def test_unsharded_layer_matches_brute_force(n_heads, n_kv):
    wl = _micro(n_heads, n_kv, 1, seq=7, d=3, ffn=5, batch=2)
    x, w = _inputs(wl)
    ref = O.layer_full(x, w, n_heads, n_kv)
    for b in range(wl.batch):
        bw = {k: v.tolist() for k, v in w.items()}
        got = brute.layer_seq(x[b].tolist(), bw, n_heads, n_kv)
        for key in ("attn", "u", "mlp", "y"):
            assert _rel(got[key], ref[key][b]) < 1e-12, key


# ---------------------------------------------------------------------------
# The fold identity and the special cases of the folded schedule
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n_heads,n_kv,degree", [(2, 2, 1), (2, 2, 2), (4, 4, 4),
                                                 (4, 2, 2), (8, 4, 4), (8, 8, 2)])
def test_fold_concat_equals_unsharded(n_heads, n_kv, degree):
    wl = _micro(n_heads, n_kv, degree, seq=16, d=4, ffn=24, batch=2)
    x, w = _inputs(wl)
    ref = O.layer_full(x, w, n_heads, n_kv)
    attn_sh, w1s, w3s, w2s = _shards(wl, w)
    chunks = [I.local_chunk(x, p, degree) for p in range(degree)]
    outs = [O.layer_rank(chunks, attn_sh, w1s, w3s, w2s, p, n_heads, n_kv, wl.head_dim)
            for p in range(degree)]
    for key in ("attn", "u", "mlp", "y"):
        got = np.concatenate([o[key] for o in outs], axis=1)
        assert _rel(got, ref[key]) < 1e-12, key


def test_fold_tiny_workload_equals_unsharded():
    wl = TINY
    x, w = _inputs(wl)
    ref = O.layer_full(x, w, wl.n_heads, wl.n_kv_heads)
    attn_sh, w1s, w3s, w2s = _shards(wl, w)
    chunks = [I.local_chunk(x, p, wl.degree) for p in range(wl.degree)]
    for p in range(wl.degree):
        o = O.layer_rank(chunks, attn_sh, w1s, w3s, w2s, p, wl.n_heads, wl.n_kv_heads,
                         wl.head_dim)
        sl = slice(p * wl.s_loc, (p + 1) * wl.s_loc)
        for key in ("attn", "mlp", "y"):
            assert _rel(o[key], ref[key][:, sl]) < 1e-12, key


def test_mlp_ring_order_and_row_permutation_invariance():
    wl = _micro(2, 2, 4, seq=8, d=4, ffn=32)
    x, w = _inputs(wl)
    _, w1s, w3s, w2s = _shards(wl, w)
    x0 = I.local_chunk(x, 1, 4)
    base = O.mlp_rank(x0, w1s, w3s, w2s, 1)
    # any rank's ring order visits every shard once
    for p in range(4):
        assert _rel(O.mlp_rank(x0, w1s, w3s, w2s, p), base) < 1e-13
    # permuting intermediate rows consistently inside one shard changes nothing
    perm = np.random.default_rng(0).permutation(w1s[2].shape[0])
    w1p, w3p, w2p = list(w1s), list(w3s), list(w2s)
    w1p[2], w3p[2], w2p[2] = w1s[2][perm], w3s[2][perm], w2s[2][perm]
    assert _rel(O.mlp_rank(x0, w1p, w3p, w2p, 1), base) < 1e-13
    # dropping a shard does change it (the test is sensitive to every shard)
    assert _rel(O.mlp_rank(x0, w1s[:3], w3s[:3], w2s[:3], 1), base) > 1e-3


def test_linearity_in_output_projections():
    wl = _micro(4, 2, 2, seq=8, d=4, ffn=16)
    x, w = _inputs(wl)
    attn_sh, w1s, w3s, w2s = _shards(wl, w)
    chunks = [I.local_chunk(x, p, 2) for p in range(2)]
    p = 1
    y = O.mlp_rank(chunks[p], w1s, w3s, w2s, p)
    y2 = O.mlp_rank(chunks[p], w1s, w3s, [2 * m for m in w2s], p)
    assert np.array_equal(y2, 2 * y)
    kv = [O.gather_kv(chunks, attn_sh[r], 2, 1, 4) for r in range(2)]
    a = O.attn_rank(chunks[p], attn_sh, kv, p, 4, 2, 4)
    sh2 = []
    for s in attn_sh:
        s = s.copy()
        s[-8:] *= 2          # the W_O^(r)^T block (H_s*d = 8 rows)
        sh2.append(s)
    a2 = O.attn_rank(chunks[p], sh2, kv, p, 4, 2, 4)
    assert np.array_equal(a2, 2 * a)


def test_rank0_is_plain_causal_attention_on_its_chunk():
    wl = _micro(4, 4, 4, seq=32, d=4, ffn=8)
    x, w = _inputs(wl)
    attn_sh, *_ = _shards(wl, w)
    chunks = [I.local_chunk(x, p, 4) for p in range(4)]
    kv = [O.gather_kv(chunks, attn_sh[r], 1, 1, 4) for r in range(4)]
    got = O.attn_rank(chunks[0], attn_sh, kv, 0, 4, 4, 4)
    ref = O.attention_full(chunks[0], w["wq"], w["wk"], w["wv"], w["wo"], 4, 4)
    assert _rel(got, ref) < 1e-12


@pytest.mark.parametrize("p", [0, 1, 3])
def test_zero_queries_give_prefix_mean(p):
    """W_Q = 0 makes every score 0, so the context of global position t is the mean of
    v_0..v_t: a cumulative-sum closed form that fixes the rank offset p*S_loc.
    D=4, n_h=8, n_kv=4 (g=2): each shard holds 2 query heads and 1 kv head."""
    n_h, n_kv, d, D = 8, 4, 4, 4
    wl = _micro(n_h, n_kv, D, seq=32, d=d, ffn=8, batch=2)
    x, w = _inputs(wl)
    w = dict(w)
    w["wq"] = np.zeros_like(w["wq"])
    attn_sh, *_ = _shards(wl, w)
    chunks = [I.local_chunk(x, q, D) for q in range(D)]
    kv = [O.gather_kv(chunks, attn_sh[r], n_h // D, n_kv // D, d) for r in range(D)]
    got = O.attn_rank(chunks[p], attn_sh, kv, p, n_h, n_kv, d)
    v = x @ w["wv"].T                                        # [B, S, n_kv*d]
    cnt = np.arange(1, x.shape[1] + 1)[None, :, None]
    mean = np.cumsum(v, axis=1) / cnt
    a = np.concatenate([mean[..., (i // 2) * d:(i // 2) * d + d] for i in range(n_h)], axis=-1)
    s_loc = wl.s_loc
    expect = (a @ w["wo"].T)[:, p * s_loc:(p + 1) * s_loc]
    assert _rel(got, expect) < 1e-12


def test_softmax_rows_sum_to_one_and_first_query_sees_key0():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((40, 8)) * 3
    k = rng.standard_normal((100, 8)) * 3
    for off in (0, 17, 60):
        pm = O.causal_probs(q, k, off, 0.5)
        assert np.max(np.abs(pm.sum(axis=1) - 1.0)) < 1e-12
        assert np.all(pm[:, :][np.arange(100)[None, :] > (off + np.arange(40))[:, None]] == 0)
    v = rng.standard_normal((100, 8))
    o = O.causal_attention_core(q, k, v, 0, 0.5)
    assert np.array_equal(o[0], v[0])
    # V == 1 gives exactly-normalised averages of ones
    o1 = O.causal_attention_core(q, k, np.ones((100, 8)), 30, 0.5)
    assert np.max(np.abs(o1 - 1.0)) < 1e-13


@pytest.mark.parametrize("n_heads,n_kv", [(4, 4), (8, 2)])
def test_attention_rows_matches_unsharded(n_heads, n_kv):
    wl = _micro(n_heads, n_kv, 1, seq=48, d=8, ffn=8, batch=2)
    x, w = _inputs(wl)
    ref = O.attention_full(x, w["wq"], w["wk"], w["wv"], w["wo"], n_heads, n_kv)
    pos = [0, 1, 13, 47, 30]
    for b in range(2):
        got = O.attention_rows(x[b], w["wq"], w["wk"], w["wv"], w["wo"], n_heads, n_kv, pos)
        assert _rel(got, ref[b, pos]) < 1e-12


def test_attn_rank_row_subset_matches_full_rank():
    wl = _micro(4, 4, 2, seq=32, d=4, ffn=8)
    x, w = _inputs(wl)
    attn_sh, *_ = _shards(wl, w)
    chunks = [I.local_chunk(x, q, 2) for q in range(2)]
    kv = [O.gather_kv(chunks, attn_sh[r], 2, 2, 4) for r in range(2)]
    full = O.attn_rank(chunks[1], attn_sh, kv, 1, 4, 4, 4)
    rows = [0, 5, 15]
    sub = O.attn_rank(chunks[1], attn_sh, kv, 1, 4, 4, 4, rows=rows)
    assert _rel(sub, full[:, rows]) < 1e-13


# ---------------------------------------------------------------------------
# Zigzag layout (Algorithm 1 as printed)
# ---------------------------------------------------------------------------

def test_zigzag_partition_and_causal_balance():
    """Rank p holds chunks p and 2D-1-p of 2D equal chunks; every rank then has the
    same number of unmasked (query, key) pairs, (2D-1) S_c^2 + S_c (S_c + 1)."""
    for degree in (1, 2, 3, 4, 8):
        s_c = 5
        seq = 2 * degree * s_c
        chunks = np.arange(seq).reshape(2 * degree, s_c)
        seen = []
        for p in range(degree):
            pos = O.zigzag_positions(seq, degree, p)
            assert np.array_equal(pos, np.concatenate([chunks[p], chunks[2 * degree - 1 - p]]))
            seen.append(pos)
            pairs = int(np.sum(pos + 1))          # query at position t sees t + 1 keys
            assert pairs == (2 * degree - 1) * s_c * s_c + s_c * (s_c + 1)
        assert np.array_equal(np.sort(np.concatenate(seen)), np.arange(seq))


@pytest.mark.parametrize("n_heads,n_kv,degree", [(2, 2, 1), (2, 2, 2), (4, 2, 2), (8, 4, 4),
                                                 (4, 4, 4)])
def test_zigzag_fold_equals_unsharded(n_heads, n_kv, degree):
    """Every zigzag rank's block outputs are the unsharded layer's rows at that rank's
    positions (the property Algorithm 1's split bounds s1, s2 and ZigZagReorder exist
    to guarantee)."""
    wl = _micro(n_heads, n_kv, degree, seq=16, d=4, ffn=24, batch=2)
    x, w = _inputs(wl)
    ref = O.layer_full(x, w, n_heads, n_kv)
    attn_sh, w1s, w3s, w2s = _shards(wl, w)
    seq = x.shape[1]
    parts = np.arange(seq).reshape(2 * degree, seq // (2 * degree))
    pos = [np.concatenate([parts[p], parts[2 * degree - 1 - p]]) for p in range(degree)]
    shards = [x[:, pos[p]] for p in range(degree)]
    for p in range(degree):
        o = O.layer_rank_zigzag(shards, attn_sh, w1s, w3s, w2s, p, n_heads, n_kv, wl.head_dim)
        for key in ("attn", "mlp", "y"):
            assert _rel(o[key], ref[key][:, pos[p]]) < 1e-12, (p, key)
