"""Each plausible mistake planted in the oracle must make at least one pin fail.

The mistakes are planted on the CPU by patching oracle functions for the duration
of one test; the pins are the functions of test_oracle_pins.
"""
import numpy as np
import pytest

import oracle.tsp_oracle as O
from tests import test_oracle_attn_bwd_pins as PA
from tests import test_oracle_bwd_pins as PB
from tests import test_oracle_pins as P

_orig_probs = O.causal_probs
_orig_unpack = O.unpack_attn_shard
_orig_silu = O.silu
_orig_core_bwd = O.causal_attention_core_bwd
_orig_kv_bwd = O.attn_kv_bwd
_orig_calls = O.causal_calls


def _probs_strict_mask(q, k, q_offset, scale):          # j < t instead of j <= t
    return _orig_probs(q, k, q_offset - 1, scale) if q_offset > 0 else _orig_probs(q, k, 0, scale)


def _probs_no_mask(q, k, q_offset, scale):              # causal mask dropped
    return _orig_probs(q, k, 10 ** 9, scale)


def _probs_no_scale(q, k, q_offset, scale):             # softmax scale dropped
    return _orig_probs(q, k, q_offset, 1.0)


def _unpack_swap_kv(packed, hs, ks, d):                 # W_K / W_V blocks swapped
    wq, wk, wv, wo = _orig_unpack(packed, hs, ks, d)
    return wq, wv, wk, wo


def _silu_sigmoid_only(z):                              # z * sigmoid(z) -> sigmoid(z)
    return _orig_silu(z) / np.where(z == 0, 1.0, z)


def _attention_full_wo_untransposed(x, wq, wk, wv, wo, n_heads, n_kv_heads, scale=None):
    return _orig_attention_full(x, wq, wk, wv, wo.T, n_heads, n_kv_heads, scale)


_orig_attention_full = O.attention_full


def _mlp_full_gate_up_swapped(u, w1, w3, w2):
    return (O.silu(u @ w3.T) * (u @ w1.T)) @ w2


def _attn_rank_zero_offset(x_loc, shards, kv, p, n_heads, n_kv, d, scale=None, rows=None,
                           positions=None):
    # forgets the rank's query offset: the local rows taken to start at position 0
    pos = np.arange(x_loc.shape[1]) if positions is None else \
        np.asarray(positions) - np.asarray(positions)[0]
    return _orig_attn_rank(x_loc, shards, kv, p, n_heads, n_kv, d, scale, rows, positions=pos)


_orig_attn_rank = O.attn_rank


def _mlp_rank_skips_last_step(x_loc, w1s, w3s, w2s, p):
    d = len(w1s)
    y = np.zeros_like(x_loc)
    for t in range(d - 1):
        j = (p - t) % d
        y += (O.silu(x_loc @ w1s[j].T) * (x_loc @ w3s[j].T)) @ w2s[j]
    return y


_orig_zz_pos = O.zigzag_positions
_orig_zz_gather = O.gather_kv_zigzag


def _zigzag_halves_swapped(seq, degree, p):             # [chunk 2D-1-p; chunk p]
    pos = _orig_zz_pos(seq, degree, p)
    half = pos.shape[0] // 2
    return np.concatenate([pos[half:], pos[:half]])


def _zigzag_reorder_dropped(x_shards, packed, hs, ks, d):  # gathered rows left in rank order
    parts = [O.kv_project(xs, packed, hs, ks, d) for xs in x_shards]
    return (np.concatenate([k for k, _ in parts], axis=1),
            np.concatenate([v for _, v in parts], axis=1))


def _zigzag_plain_prefix(x_loc, shards, kv, p, n_heads, n_kv, d, scale=None):
    # treats the zigzag shard like a contiguous chunk (one causal call, offset p S_loc)
    return _orig_attn_rank(x_loc, shards, kv, p, n_heads, n_kv, d, scale)


_orig_silu_grad = O.silu_grad
_orig_swiglu_bwd = O.swiglu_bwd
_orig_mlp_rank_bwd = O.mlp_rank_bwd


def _silu_grad_sigmoid_only(z):                         # drops the (1 + z (1 - s)) factor
    return 1.0 / (1.0 + np.exp(-z))


def _swiglu_bwd_swapped(g, u, dhs):                     # gate / up gradients exchanged
    dg, du = _orig_swiglu_bwd(g, u, dhs)
    return du, dg


def _mlp_rank_bwd_no_up_path(x_loc, w1s, w3s, w2s, dy, p):  # dX misses the dU W3 term
    degree, h = len(w1s), x_loc.shape[-1]
    x2, dy2 = x_loc.reshape(-1, h), dy.reshape(-1, h)
    dx = np.zeros_like(x2)
    dw1, dw3, dw2 = [None] * degree, [None] * degree, [None] * degree
    for t in range(degree):
        j = (p - t) % degree
        g, u, dhs = x2 @ w1s[j].T, x2 @ w3s[j].T, dy2 @ w2s[j].T
        dg, du = O.swiglu_bwd(g, u, dhs)
        dx += dg @ w1s[j]
        dw1[j], dw3[j], dw2[j] = dg.T @ x2, du.T @ x2, (O.silu(g) * u).T @ dy2
    return dx.reshape(x_loc.shape), dw1, dw3, dw2


def _mlp_rank_bwd_skips_last_step(x_loc, w1s, w3s, w2s, dy, p):
    degree = len(w1s)
    dx, dw1, dw3, dw2 = _orig_mlp_rank_bwd(x_loc, w1s[:-1] + [0 * w1s[-1]], w3s, w2s, dy, p)
    return dx, dw1, dw3, dw2


def _core_bwd_no_rowsum(q, k, v, do, q_offset, scale):   # dS = P * dP (softmax term lost)
    p = O.causal_probs(q, k[:q_offset + q.shape[0]], q_offset, scale)
    kk, vv = k[:p.shape[1]], v[:p.shape[1]]
    dp = do @ vv.T
    ds = p * dp
    dk, dv = np.zeros_like(k), np.zeros_like(v)
    dk[:p.shape[1]] = scale * ds.T @ q
    dv[:p.shape[1]] = p.T @ do
    return scale * ds @ kk, dk, dv


def _core_bwd_dq_unscaled(q, k, v, do, q_offset, scale):  # dQ misses the softmax scale
    dq, dk, dv = _orig_core_bwd(q, k, v, do, q_offset, scale)
    return dq / scale, dk, dv


def _core_bwd_dk_from_probs(q, k, v, do, q_offset, scale):  # dK built from P, not dS
    dq, _, dv = _orig_core_bwd(q, k, v, do, q_offset, scale)
    p = O.causal_probs(q, k[:q_offset + q.shape[0]], q_offset, scale)
    dk = np.zeros_like(k)
    dk[:p.shape[1]] = scale * p.T @ q
    return dq, dk, dv


def _kv_bwd_no_v_path(x_loc, shards, dk_own, dv_own, n_heads, n_kv, d):
    dx, dwk, dwv = _orig_kv_bwd(x_loc, shards, dk_own, [0 * t for t in dv_own], n_heads, n_kv, d)
    _, dwk2, dwv2 = _orig_kv_bwd(x_loc, shards, dk_own, dv_own, n_heads, n_kv, d)
    return dx, dwk2, dwv2


def _reduce_scatter_no_sum(contribs, degree, layout):       # each rank keeps only its own
    seq = contribs[0].shape[1]
    return [contribs[q][:, O.rank_positions(seq, degree, q, layout)] for q in range(degree)]


def _calls_zigzag_offsets_swapped(s_loc, degree, p, layout):
    calls = _orig_calls(s_loc, degree, p, layout)
    if len(calls) == 2:
        (a0, a1, o1, n1), (b0, b1, o2, n2) = calls
        return [(a0, a1, o2, n2), (b0, b1, o1, n1)]
    return calls


MUTATIONS = {
    "attn_bwd_rowsum_dropped": ("causal_attention_core_bwd", _core_bwd_no_rowsum),
    "attn_bwd_dq_unscaled": ("causal_attention_core_bwd", _core_bwd_dq_unscaled),
    "attn_bwd_dk_from_probs": ("causal_attention_core_bwd", _core_bwd_dk_from_probs),
    "attn_kv_bwd_misses_v_path": ("attn_kv_bwd", _kv_bwd_no_v_path),
    "kv_grad_not_reduced": ("reduce_scatter_rows", _reduce_scatter_no_sum),
    "attn_bwd_zigzag_calls_swapped": ("causal_calls", _calls_zigzag_offsets_swapped),
    "silu_grad_is_sigmoid": ("silu_grad", _silu_grad_sigmoid_only),
    "swiglu_bwd_swapped": ("swiglu_bwd", _swiglu_bwd_swapped),
    "bwd_dx_misses_up_path": ("mlp_rank_bwd", _mlp_rank_bwd_no_up_path),
    "bwd_last_shard_dropped": ("mlp_rank_bwd", _mlp_rank_bwd_skips_last_step),
    "zigzag_halves_swapped": ("zigzag_positions", _zigzag_halves_swapped),
    "zigzag_reorder_dropped": ("gather_kv_zigzag", _zigzag_reorder_dropped),
    "zigzag_as_contiguous": ("attn_rank_zigzag", _zigzag_plain_prefix),
    "mask_excludes_diagonal": ("causal_probs", _probs_strict_mask),
    "mask_dropped": ("causal_probs", _probs_no_mask),
    "scale_dropped": ("causal_probs", _probs_no_scale),
    "kv_blocks_swapped": ("unpack_attn_shard", _unpack_swap_kv),
    "silu_is_sigmoid": ("silu", _silu_sigmoid_only),
    "wo_not_transposed": ("attention_full", _attention_full_wo_untransposed),
    "gate_up_swapped": ("mlp_full", _mlp_full_gate_up_swapped),
    "rank_offset_dropped": ("attn_rank", _attn_rank_zero_offset),
    "ring_step_dropped": ("mlp_rank", _mlp_rank_skips_last_step),
}

PINS = [
    (P.test_attention_two_token_closed_form, ()),
    (P.test_gqa_head_mapping_closed_form, ()),
    (P.test_mlp_closed_form, ()),
    (P.test_unsharded_layer_matches_brute_force, (2, 1)),
    (P.test_fold_concat_equals_unsharded, (4, 2, 2)),
    (P.test_zero_queries_give_prefix_mean, (1,)),
    (P.test_softmax_rows_sum_to_one_and_first_query_sees_key0, ()),
    (P.test_linearity_in_output_projections, ()),
    (P.test_mlp_ring_order_and_row_permutation_invariance, ()),
    (P.test_zigzag_partition_and_causal_balance, ()),
    (P.test_zigzag_fold_equals_unsharded, (4, 2, 2)),
    (PB.test_rank_backward_matches_finite_differences, ()),
    (PB.test_weight_gradients_sum_to_owner_and_dx_is_local, ()),
    (PB.test_backward_special_cases, ()),
    (PA.test_two_stage_backward_is_the_unsharded_gradient, ("contiguous", 4, 2)),
    (PA.test_two_stage_backward_is_the_unsharded_gradient, ("zigzag", 4, 2)),
    (PA.test_first_stage_is_the_gradient_of_the_rank_forward, ("zigzag",)),
    (PA.test_backward_special_cases, ()),
]


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(O, attr, fn)
    failed = []
    for pin, args in PINS:
        try:
            pin(*args)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"no pin caught mutation {name}"
