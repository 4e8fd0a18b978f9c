"""GPU parity of libtsp against the fp64 oracle at sizes the oracle finishes in
seconds, plus the special cases the oracle pins (all through the C ABI)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import tsp_oracle as O  # noqa: E402
from paper_2604_26294_amd import inputs as I  # noqa: E402
from paper_2604_26294_amd import tsp as T  # noqa: E402
from paper_2604_26294_amd.harness import RankProblem  # noqa: E402
from paper_2604_26294_amd.workloads import TINY  # noqa: E402
from tests.gpu_common import (MID_GQA64, MID_GQA8, MID_MHA128, MLP_BIG, ODD3, SINGLE, SUBL,  # noqa: E402
                              assert_close, f64, gen, oracle_blocks)

CASES = [(TINY, 0), (TINY, 1), (MID_GQA64, 0), (MID_GQA64, 2), (MID_GQA64, 3),
         (MID_MHA128, 1), (MID_GQA8, 1), (SINGLE, 0), (ODD3, 2), (ODD3, 0),
         # zigzag shards (Algorithm 1 as printed): two query segments, K/V rows written
         # at reordered positions, every other rank's rows visible
         (TINY.with_layout(1), 0), (TINY.with_layout(1), 1), (MID_GQA64.with_layout(1), 0),
         (MID_GQA64.with_layout(1), 3), (MID_MHA128.with_layout(1), 0),
         (MID_GQA8.with_layout(1), 1), (SINGLE.with_layout(1), 0), (ODD3.with_layout(1), 1)]
_IDS = [f"{w.name}-{w.layout_name}-r{p}" for w, p in CASES]
_cache = {}


def _inputs(wl):
    if wl.name not in _cache:       # the inputs do not depend on the layout
        _cache[wl.name] = gen(wl)
    return _cache[wl.name]


def _run(wl, p, block, x_bits=None, w_bits=None):
    x_bits, w_bits = (x_bits, w_bits) if x_bits is not None else _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv()
    if block == "mlp":
        y = prob.mlp()
    elif block == "attn":
        y = prob.attn_fwd()
    else:
        y = prob.layer()
    torch.cuda.synchronize()
    return y.double().cpu().numpy(), prob


@pytest.mark.parametrize("wl,p", CASES, ids=_IDS)
@pytest.mark.parametrize("block", ["mlp", "attn", "layer"])
def test_block_parity(wl, p, block):
    print(f"[parity] {wl.name} rank {p} {block}", flush=True)
    got, _ = _run(wl, p, block)
    ref = oracle_blocks(wl, *_inputs(wl), p, blocks=(block,))[block]
    assert_close(got, ref, f"{wl.name} r{p} {block}")


@pytest.mark.parametrize("wl", [TINY, MID_GQA64, TINY.with_layout(1), MID_GQA64.with_layout(1)],
                         ids=lambda w: f"{w.name}-{w.layout_name}")
def test_rank_concat_equals_unsharded_layer(wl):
    """All ranks together give the unsharded layer, each row at its rank's positions."""
    x_bits, w_bits = _inputs(wl)
    outs = [_run(wl, p, "layer")[0] for p in range(wl.degree)]
    x = f64(x_bits)
    w = {k: f64(v) for k, v in w_bits.items()}
    ref = O.layer_full(x, w, wl.n_heads, wl.n_kv_heads)
    if wl.layout == 1:
        pos = np.concatenate([O.zigzag_positions(wl.seq, wl.degree, p)
                              for p in range(wl.degree)])
        ref = {k: v[:, pos] for k, v in ref.items()}
    assert_close(np.concatenate(outs, axis=1), ref["y"], "concat layer")
    attn = [_run(wl, p, "attn")[0] for p in range(wl.degree)]
    assert_close(np.concatenate(attn, axis=1), ref["attn"], "concat attn")


def test_v_ones_gives_output_projection_row_sums():
    """x[..., 0] = 1 and W_V = e_0 make every V row exactly 1, so every attention
    context is 1 and the block returns the row sums of W_O for every token."""
    wl = MID_GQA64
    x_bits, w_bits = _inputs(wl)
    x_bits = x_bits.copy()
    x_bits[..., 0] = I.round_to_bf16_bits(np.array([1.0], np.float32))[0]
    w_bits = dict(w_bits)
    wv = np.zeros_like(w_bits["wv"])
    wv[:, 0] = I.round_to_bf16_bits(np.array([1.0], np.float32))[0]
    w_bits["wv"] = wv
    for p in (0, 3):
        got, _ = _run(wl, p, "attn", x_bits, w_bits)
        rowsum = f64(w_bits["wo"]).sum(axis=1)
        expect = np.broadcast_to(rowsum, got.shape)
        assert np.max(np.abs(got - expect)) <= 1e-2 * np.max(np.abs(rowsum)), p


def test_zero_queries_give_prefix_mean():
    wl = MID_MHA128
    x_bits, w_bits = _inputs(wl)
    w_bits = dict(w_bits)
    w_bits["wq"] = np.zeros_like(w_bits["wq"])
    got, _ = _run(wl, 1, "attn", x_bits, w_bits)
    x = f64(x_bits)
    v = x @ f64(w_bits["wv"]).T
    mean = np.cumsum(v, axis=1) / np.arange(1, x.shape[1] + 1)[None, :, None]
    expect = (mean @ f64(w_bits["wo"]).T)[:, wl.s_loc:]          # MHA: head i reads kv head i
    assert_close(got, expect, "prefix mean")


def test_future_kv_rows_are_never_read():
    """Rows of the K/V buffer at or beyond (p+1) S/D are poisoned with NaN: the
    output must stay finite and bitwise equal to a run with a clean buffer."""
    wl, p = MID_GQA64, 1
    x_bits, w_bits = _inputs(wl)
    clean = RankProblem(wl, x_bits, w_bits, p, kv_fill=0.0)
    clean.prefill_kv()
    y_clean = clean.layer().clone()
    dirty = RankProblem(wl, x_bits, w_bits, p, kv_fill=float("nan"))
    dirty.prefill_kv()
    y_dirty = dirty.layer().clone()
    torch.cuda.synchronize()
    assert torch.isfinite(y_dirty).all()
    assert torch.equal(y_clean, y_dirty)


def test_deterministic_and_linear():
    wl, p = MID_MHA128, 1
    x_bits, w_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv()
    a = prob.layer().clone()
    b = prob.layer().clone()
    assert torch.equal(a, b)
    y1 = prob.mlp().clone()
    prob.w2 = [2 * t for t in prob.w2]                      # exact in bf16
    y2 = prob.mlp().clone()
    assert torch.equal(y2, 2 * y1)
    a1 = prob.attn_fwd().clone()
    qd = wl.n_heads // wl.degree * wl.head_dim
    kd = wl.n_kv_heads // wl.degree * wl.head_dim
    for s in prob.attn:
        s[qd + 2 * kd:] *= 2                               # the W_O^(r)^T block
    a2 = prob.attn_fwd().clone()
    torch.cuda.synchronize()
    assert torch.equal(a2, 2 * a1)


@pytest.mark.parametrize("wl,p", [(MID_GQA64, 2), (MID_GQA64.with_layout(1), 3), (MID_MHA128, 1)],
                         ids=["gqa64-contiguous-r2", "gqa64-zigzag-r3", "mha128-contiguous-r1"])
def test_back_to_back_calls_are_bit_identical(wl, p):
    """Calls enqueued back to back on one stream, with the three forward entry points
    interleaved and sharing one workspace, reproduce the first result of each entry
    point bit for bit (every reduction has a fixed order and nothing depends on what an
    earlier call left in the workspace)."""
    print(f"[overlap] {wl.name} {wl.layout_name} rank {p}", flush=True)
    prob = RankProblem(wl, *_inputs(wl), p)
    prob.prefill_kv()
    first = {"layer": prob.layer().clone(), "mlp": prob.mlp().clone(),
             "attn": prob.attn_fwd().clone()}
    again = []
    for _ in range(3):
        again.append(("layer", prob.layer().clone()))
        again.append(("attn", prob.attn_fwd().clone()))
        again.append(("mlp", prob.mlp().clone()))
    torch.cuda.synchronize()
    for name, t in again:
        assert torch.equal(t, first[name]), name
    ref = oracle_blocks(wl, *_inputs(wl), p, blocks=("layer",))["layer"]
    assert_close(first["layer"].double().cpu().numpy(), ref, f"{wl.name} r{p} layer")


@pytest.mark.parametrize("wl,p", [(MID_GQA8, 1), (MID_MHA128, 0)], ids=["gqa8-r1", "mha128-r0"])
def test_workspace_contents_do_not_matter(wl, p):
    """A workspace filled with 0xff bytes (every float a NaN) gives the same output bit
    for bit as a zeroed one: each call writes every workspace element it reads (these
    shapes split the down and output projections' contraction through fp32 partials
    there, next to the gated product with its zero padding, Q and A)."""
    print(f"[dirty ws] {wl.name} rank {p}", flush=True)
    prob = RankProblem(wl, *_inputs(wl), p)
    prob.prefill_kv()
    prob.ws.zero_()
    ref = {"layer": prob.layer().clone(), "mlp": prob.mlp().clone(),
           "attn": prob.attn_fwd().clone()}
    for name, run in (("layer", prob.layer), ("mlp", prob.mlp), ("attn", prob.attn_fwd)):
        prob.ws.fill_(255)
        got = run().clone()
        torch.cuda.synchronize()
        assert torch.equal(got, ref[name]), name


def test_mlp_block_on_large_gate_up_tiles():
    """The MLP block at a shape whose grouped gate+up product takes the 256 x 128 tiles
    (1024 tiles, F/D = 1000: ragged column tiles and the zero padding of Hs to 1024),
    every element against the oracle."""
    wl = MLP_BIG
    print(f"[mlp big tiles] {wl.name}", flush=True)
    x_bits, w_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, wl.rank)
    got = prob.mlp().double().cpu().numpy()
    torch.cuda.synchronize()
    ref = oracle_blocks(wl, x_bits, w_bits, wl.rank, blocks=("mlp",))["mlp"]
    assert_close(got, ref, f"{wl.name} MLP")


@pytest.mark.parametrize("wl,p", [(MID_MHA128, 1), (SUBL.with_layout(1), 1)],
                         ids=["key-range-split", "paired-tiles"])
def test_attention_slot_wait_that_gives_up_is_loud(wl, p):
    """The attention forward hands its K/V slots over through bounded waits on LDS
    counters.  With every wait capped at one poll (the C ABI's test hook) the waits give
    up, and every output of the attention block must come back NaN, not a quiet wrong
    value; with the default restored the next call reproduces the first bit for bit."""
    print(f"[poll limit] {wl.name} {wl.layout_name} rank {p}", flush=True)
    prob = RankProblem(wl, *_inputs(wl), p)
    prob.prefill_kv()
    good = prob.attn_fwd().clone()
    try:
        T.tsp_test_set_attn_poll_limit(1)
        bad = prob.attn_fwd().clone()
        torch.cuda.synchronize()
    finally:
        T.tsp_test_set_attn_poll_limit(0)
    again = prob.attn_fwd().clone()
    torch.cuda.synchronize()
    assert bool(torch.isnan(bad).all())
    assert torch.equal(again, good)


def test_accumulate_flag_adds_to_existing_output():
    wl, p = TINY, 1
    x_bits, w_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv()
    y_mlp = prob.mlp().clone()
    prob.y.fill_(1.5)
    y_acc = prob.mlp(accumulate=True).clone()
    torch.cuda.synchronize()
    assert torch.allclose(y_acc, y_mlp + 1.5, rtol=0, atol=1e-6)


def test_empty_batch_leaves_output_untouched():
    from dataclasses import replace
    wl = replace(TINY, batch=0)
    prob = RankProblem(TINY, *_inputs(TINY), 1)
    sh = T.shape_of(wl, 1)
    prob.y.fill_(3.0)
    T.tsp_layer_rank_fwd(sh, prob.x_loc, prob.attn, prob.w1, prob.w3, prob.w2, prob.k_buf,
                         prob.v_buf, prob.y, prob.ws)
    torch.cuda.synchronize()
    assert bool((prob.y == 3.0).all())
