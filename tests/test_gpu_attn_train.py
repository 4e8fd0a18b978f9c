"""GPU parity of the training pair tsp_attn_rank_fwd_train / tsp_attn_rank_bwd_saved
through the C ABI: the forward also keeps every shard's attention output A and each
query's base-2 log-sum-exp, and the first stage of the attention backward takes them
instead of recomputing the forward.

* The block output equals tsp_attn_rank_fwd's bit for bit (the same kernels, which then
  also store what they computed).
* A against the oracle's causal attention of each query head (the rank's rows at their
  global positions, over the shard's gathered K / V); the log-sum-exp against
  log2 sum_j 2^(s_tj) of the oracle's base-2 logits s = scale log2(e) q_t . k_j over the
  visible keys, both computed here from the oracle's fp64 projections.
* The saved-input backward against oracle.attn_rank_bwd, as the recomputing backward is
  checked, and against that backward itself.
"""
import math

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import tsp_oracle as O  # noqa: E402
from paper_2604_26294_amd import inputs as I  # noqa: E402
from paper_2604_26294_amd import tsp as T  # noqa: E402
from paper_2604_26294_amd.harness import (RankProblem, local_positions, local_rows,  # noqa: E402
                                          to_device_bf16)
from paper_2604_26294_amd.workloads import TINY  # noqa: E402
from tests.gpu_common import (MID_GQA64, MID_MHA128, ODD3, SUBL, assert_close,  # noqa: E402
                              f64)

# contiguous and zigzag; GQA; odd D; key-range splits (the log-sum-exp written by the
# combine kernel) and, in the forward, a shape whose launch pairs query tiles (written by
# the attention kernel itself)
CASES = [(TINY, 1), (MID_GQA64, 3), (MID_MHA128.with_layout(1), 0), (ODD3, 2)]
FWD_CASES = CASES + [(SUBL.with_layout(1), 1)]
_IDS = [f"{w.name}-{w.layout_name}-r{p}" for w, p in CASES]
_FWD_IDS = [f"{w.name}-{w.layout_name}-r{p}" for w, p in FWD_CASES]
_cache = {}


def _inputs(wl):
    if wl.name not in _cache:
        _cache[wl.name] = (I.make_x_full(wl), I.make_weights(wl), I.make_dy_full(wl))
    return _cache[wl.name]


def _oracle_setup(wl, p):
    x_bits, w_bits, dy_bits = _inputs(wl)
    D = wl.degree
    w = {k: f64(v) for k, v in w_bits.items()}
    shards = [I.attn_shard_packed(w, r, D, wl.n_heads, wl.n_kv_heads, wl.head_dim)
              for r in range(D)]
    xs = [f64(local_rows(x_bits, wl, q)) for q in range(D)]
    gather = O.gather_kv_zigzag if wl.layout == 1 else O.gather_kv
    kv = [gather(xs, shards[r], wl.n_heads // D, wl.n_kv_heads // D, wl.head_dim)
          for r in range(D)]
    return xs, shards, kv, f64(local_rows(dy_bits, wl, p))


def _oracle_a_lse(wl, p, xs, shards, kv):
    """A [B, S_loc, n_h, d] and the base-2 log-sum-exp [B, n_h, S_loc] of rank p."""
    D, d = wl.degree, wl.head_dim
    hs, ks, g = wl.n_heads // D, wl.n_kv_heads // D, wl.n_heads // wl.n_kv_heads
    scale = 1.0 / math.sqrt(d)
    pos = local_positions(wl, p)
    x = xs[p]
    b_, s_loc, _ = x.shape
    a = np.zeros((b_, s_loc, wl.n_heads, d))
    lse = np.zeros((b_, wl.n_heads, s_loc))
    for r in range(D):
        wq, _, _, _ = O.unpack_attn_shard(shards[r], hs, ks, d)
        q = (x @ wq.T).reshape(b_, s_loc, hs, d)
        k_hat, v_hat = kv[r]
        for b in range(b_):
            for i in range(hs):
                kk, vv = k_hat[b, :, i // g], v_hat[b, :, i // g]
                a[b, :, r * hs + i] = O.causal_attention_core(q[b, :, i], kk, vv, pos, scale)
                s2 = (q[b, :, i] @ kk.T) * (scale / math.log(2.0))
                s2 = np.where(np.arange(kk.shape[0])[None, :] <= pos[:, None], s2, -np.inf)
                m = s2.max(axis=1)
                lse[b, r * hs + i] = m + np.log2(np.exp2(s2 - m[:, None]).sum(axis=1))
    return a, lse


@pytest.mark.parametrize("wl,p", FWD_CASES, ids=_FWD_IDS)
def test_train_forward_keeps_a_and_lse(wl, p):
    print(f"[attn train fwd] {wl.name} {wl.layout_name} rank {p}", flush=True)
    x_bits, w_bits, _ = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv()
    y_plain = prob.attn_fwd().clone()
    y, a, lse = prob.attn_fwd_train()
    torch.cuda.synchronize()
    assert torch.equal(y, y_plain), "the kept-activation forward changed the block output"
    xs, shards, kv, _ = _oracle_setup(wl, p)
    ref_a, ref_lse = _oracle_a_lse(wl, p, xs, shards, kv)
    assert_close(a.double().cpu().numpy(), ref_a, f"{wl.name} r{p} A")
    assert_close(lse.double().cpu().numpy(), ref_lse, f"{wl.name} r{p} lse")
    assert float(np.max(np.abs(lse.double().cpu().numpy() - ref_lse))) < 0.1


@pytest.mark.parametrize("wl,p", CASES, ids=_IDS)
def test_backward_from_kept_activations(wl, p):
    print(f"[attn train bwd] {wl.name} {wl.layout_name} rank {p}", flush=True)
    x_bits, w_bits, dy_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv(include_self=True)
    dy = to_device_bf16(local_rows(dy_bits, wl, p))
    # the recomputing backward first (its outputs copied), then the kept-input one
    dx_r, dw_r, dk_r, dv_r = (t.clone() if torch.is_tensor(t) else [u.clone() for u in t]
                              for t in prob.attn_bwd(dy))
    prob.attn_fwd_train()
    dx, dw, dk, dv = prob.attn_bwd_saved(dy)
    torch.cuda.synchronize()
    xs, shards, kv, dy64 = _oracle_setup(wl, p)
    ref = O.attn_rank_bwd(xs[p], shards, kv, p, wl.n_heads, wl.n_kv_heads, wl.head_dim, dy64,
                          layout="zigzag" if wl.layout == 1 else "contiguous")
    D, d = wl.degree, wl.head_dim
    qd, kd, ks = wl.n_heads // D * d, wl.n_kv_heads // D * d, wl.n_kv_heads // D
    assert_close(dx.double().cpu().numpy(), ref["dx"], f"{wl.name} r{p} dX")
    assert_close(dx.double().cpu().numpy(), dx_r.double().cpu().numpy(), "dX vs recomputing")
    dk_all, dv_all = dk.double().cpu().numpy(), dv.double().cpu().numpy()
    for r in range(D):
        g = dw[r].double().cpu().numpy()
        assert_close(g[:qd], ref["dwq"][r], f"{wl.name} r{p} dW_Q[{r}]")
        assert_close(g[qd + 2 * kd:], ref["dwo_t"][r], f"{wl.name} r{p} dW_O^T[{r}]")
        assert_close(g, dw_r[r].double().cpu().numpy(), f"dW[{r}] vs recomputing")
        cols = slice(r * ks, (r + 1) * ks)
        assert_close(dk_all[:, :, cols], ref["dk"][r], f"{wl.name} r{p} dK-hat[{r}]")
        assert_close(dv_all[:, :, cols], ref["dv"][r], f"{wl.name} r{p} dV-hat[{r}]")
    assert_close(dk_all, dk_r.double().cpu().numpy(), "dK-hat vs recomputing")
    assert_close(dv_all, dv_r.double().cpu().numpy(), "dV-hat vs recomputing")


def test_dkdv_slot_wait_that_gives_up_is_loud():
    """The dK/dV kernel hands its query tiles over through bounded waits on LDS counters.
    With every wait capped at one poll (the C ABI's test hook) the waits give up and the
    dK-hat / dV-hat contributions must come back NaN, while dX (the query path, from the
    dQ kernel, which has no such waits) stays finite; with the default restored the next
    call reproduces the first bit for bit.  The kept-activation path is used so that no
    forward attention runs under the cap."""
    wl, p = MID_MHA128, 1
    print(f"[bwd poll limit] {wl.name} rank {p}", flush=True)
    x_bits, w_bits, dy_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv(include_self=True)
    dy = to_device_bf16(local_rows(dy_bits, wl, p))
    prob.attn_fwd_train()
    first = [t.clone() for t in prob.attn_bwd_saved(dy) if torch.is_tensor(t)]
    try:
        T.tsp_test_set_attn_poll_limit(1)
        dx, _, dk, dv = (t.clone() if torch.is_tensor(t) else t for t in prob.attn_bwd_saved(dy))
        torch.cuda.synchronize()
    finally:
        T.tsp_test_set_attn_poll_limit(0)
    assert bool(torch.isnan(dk).all()) and bool(torch.isnan(dv).all())
    assert bool(torch.isfinite(dx).all())
    again = [t.clone() for t in prob.attn_bwd_saved(dy) if torch.is_tensor(t)]
    torch.cuda.synchronize()
    for a, b in zip(again, first):
        assert torch.equal(a, b)
