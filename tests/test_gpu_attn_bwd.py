"""GPU parity of the two-stage attention backward (tsp_attn_rank_bwd, then
tsp_attn_kv_rank_bwd) against the fp64 oracle, through the C ABI, per output tensor at
the forward's tolerance (bf16 operands, fp32 accumulation).

Stage one is compared with oracle.attn_rank_bwd on the same seeded inputs: the query
path of dX, the W_Q and W_O^T blocks of every shard's weight-gradient contribution, and
the rank's contributions to the gradients of every shard's gathered K / V (all S rows,
zero where none of its queries looks).  Stage two takes seeded stand-ins for the
reduce-scattered K / V gradients and is compared with oracle.attn_kv_bwd."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import tsp_oracle as O  # noqa: E402
from paper_2604_26294_amd import inputs as I  # noqa: E402
from paper_2604_26294_amd.harness import RankProblem, local_rows, to_device_bf16  # noqa: E402
from paper_2604_26294_amd.workloads import TINY  # noqa: E402
from tests.gpu_common import (MID_GQA64, MID_GQA8, MID_MHA128, ODD3, SINGLE,  # noqa: E402
                              assert_close, f64)

# Ragged tails: S_loc = 128 / 192 / 640 / 256 / 320 against the 64-query stage and
# 128-query tile; the zigzag shard's two segments of 96 rows; GQA group 2 and 8.
CASES = [(TINY, 1), (MID_GQA64, 3), (MID_GQA64, 0), (MID_MHA128, 1), (MID_GQA8, 1),
         (SINGLE, 0), (MID_GQA64.with_layout(1), 2), (MID_MHA128.with_layout(1), 0),
         (ODD3, 2)]  # odd D: the dX product of the last shard runs alone
_cache = {}


def _inputs(wl):
    if wl.name not in _cache:
        _cache[wl.name] = (I.make_x_full(wl), I.make_weights(wl), I.make_dy_full(wl))
    return _cache[wl.name]


def _layout(wl):
    return "zigzag" if wl.layout == 1 else "contiguous"


def _reference_stage1(wl, p):
    x_bits, w_bits, dy_bits = _inputs(wl)
    D = wl.degree
    w = {k: f64(v) for k, v in w_bits.items()}
    shards = [I.attn_shard_packed(w, r, D, wl.n_heads, wl.n_kv_heads, wl.head_dim)
              for r in range(D)]
    xs = [f64(local_rows(x_bits, wl, q)) for q in range(D)]
    gather = O.gather_kv_zigzag if wl.layout == 1 else O.gather_kv
    kv = [gather(xs, shards[r], wl.n_heads // D, wl.n_kv_heads // D, wl.head_dim)
          for r in range(D)]
    dy = f64(local_rows(dy_bits, wl, p))
    return O.attn_rank_bwd(xs[p], shards, kv, p, wl.n_heads, wl.n_kv_heads, wl.head_dim, dy,
                           layout=_layout(wl))


def _blocks(wl):
    D, d = wl.degree, wl.head_dim
    qd, kd = wl.n_heads // D * d, wl.n_kv_heads // D * d
    return qd, kd


@pytest.mark.parametrize("wl,p", CASES, ids=[f"{w.name}-{w.layout_name}-r{p}" for w, p in CASES])
def test_attention_backward_first_stage(wl, p):
    print(f"[attn bwd 1] {wl.name} {wl.layout_name} rank {p}", flush=True)
    x_bits, w_bits, dy_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv(include_self=True)
    dy = to_device_bf16(local_rows(dy_bits, wl, p))
    dx, dw, dk, dv = prob.attn_bwd(dy)
    torch.cuda.synchronize()
    ref = _reference_stage1(wl, p)
    qd, kd = _blocks(wl)
    ks = wl.n_kv_heads // wl.degree
    assert_close(dx.double().cpu().numpy(), ref["dx"], f"{wl.name} r{p} dX")
    dk_all, dv_all = dk.double().cpu().numpy(), dv.double().cpu().numpy()
    for r in range(wl.degree):
        g = dw[r].double().cpu().numpy()
        assert_close(g[:qd], ref["dwq"][r], f"{wl.name} r{p} dW_Q[{r}]")
        assert_close(g[qd + 2 * kd:], ref["dwo_t"][r], f"{wl.name} r{p} dW_O^T[{r}]")
        assert not np.any(g[qd:qd + 2 * kd]), "the K/V blocks belong to the second stage"
        cols = slice(r * ks, (r + 1) * ks)
        assert_close(dk_all[:, :, cols], ref["dk"][r], f"{wl.name} r{p} dK-hat[{r}]")
        assert_close(dv_all[:, :, cols], ref["dv"][r], f"{wl.name} r{p} dV-hat[{r}]")
        # keys past every query of the rank get exactly zero
        last = int(np.max(np.nonzero(np.any(ref["dv"][r] != 0, axis=(0, 2, 3)))[0]))
        assert not np.any(dk_all[:, last + 1:, cols]) and not np.any(dv_all[:, last + 1:, cols])


@pytest.mark.parametrize("wl,p", [(TINY, 0), (MID_GQA64, 2), (MID_MHA128, 1), (SINGLE, 0)],
                         ids=["tiny-r0", "gqa64-r2", "mha128-r1", "single"])
def test_attention_backward_second_stage(wl, p):
    print(f"[attn bwd 2] {wl.name} rank {p}", flush=True)
    x_bits, w_bits, _ = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    dk_bits, dv_bits = I.make_dkv_own(wl, p)
    dx, dw = prob.attn_kv_bwd(to_device_bf16(dk_bits), to_device_bf16(dv_bits), accumulate=False)
    torch.cuda.synchronize()
    D, ks = wl.degree, wl.n_kv_heads // wl.degree
    w = {k: f64(v) for k, v in w_bits.items()}
    shards = [I.attn_shard_packed(w, r, D, wl.n_heads, wl.n_kv_heads, wl.head_dim)
              for r in range(D)]
    dk64, dv64 = f64(dk_bits), f64(dv_bits)
    ref_dx, ref_dwk, ref_dwv = O.attn_kv_bwd(
        f64(local_rows(x_bits, wl, p)), shards,
        [dk64[:, :, r * ks:(r + 1) * ks] for r in range(D)],
        [dv64[:, :, r * ks:(r + 1) * ks] for r in range(D)], wl.n_heads, wl.n_kv_heads,
        wl.head_dim)
    qd, kd = _blocks(wl)
    assert_close(dx.double().cpu().numpy(), ref_dx, f"{wl.name} r{p} dX (K/V path)")
    for r in range(D):
        g = dw[r].double().cpu().numpy()
        assert_close(g[qd:qd + kd], ref_dwk[r], f"{wl.name} r{p} dW_K[{r}]")
        assert_close(g[qd + kd:qd + 2 * kd], ref_dwv[r], f"{wl.name} r{p} dW_V[{r}]")


def test_two_stages_accumulate_into_one_dx():
    """Stage two with accumulate != 0 adds its K/V path onto the first stage's dX."""
    wl, p = MID_GQA64, 1
    x_bits, w_bits, dy_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv(include_self=True)
    dk_bits, dv_bits = I.make_dkv_own(wl, p)
    dkl, dvl = to_device_bf16(dk_bits), to_device_bf16(dv_bits)
    dy = to_device_bf16(local_rows(dy_bits, wl, p))
    first = prob.attn_bwd(dy)[0].clone()
    second_only = prob.attn_kv_bwd(dkl, dvl, accumulate=False)[0].clone()
    prob.attn_bwd(dy)
    both = prob.attn_kv_bwd(dkl, dvl, accumulate=True)[0]
    torch.cuda.synchronize()
    assert torch.allclose(both, first + second_only, rtol=1e-5, atol=1e-6)


def test_first_stage_accumulates():
    """A second first-stage call with accumulate != 0 adds the same dX, weight-gradient
    blocks and K/V-gradient contributions again (up to the fp32 summation order)."""
    wl, p = MID_GQA64, 2
    x_bits, w_bits, dy_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv(include_self=True)
    dy = to_device_bf16(local_rows(dy_bits, wl, p))
    dx, dw, dk, dv = prob.attn_bwd(dy)
    once = [dx.clone(), [t.clone() for t in dw], dk.clone(), dv.clone()]
    prob.attn_bwd(dy, accumulate=True)
    torch.cuda.synchronize()
    assert torch.allclose(dx, 2 * once[0], rtol=1e-5, atol=1e-6)
    for a, b in zip(dw, once[1]):
        assert torch.allclose(a, 2 * b, rtol=1e-5, atol=1e-6)
    assert torch.allclose(dk, 2 * once[2], rtol=1e-5, atol=1e-6)
    assert torch.allclose(dv, 2 * once[3], rtol=1e-5, atol=1e-6)
