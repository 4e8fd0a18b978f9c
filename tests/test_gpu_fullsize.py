"""Full-size parity on sampled rows, in the launch configuration the benchmark times.

For each of the study's layer shapes the GPU runs the rank's attention block, MLP
block and whole layer through the C ABI; the oracle recomputes a handful of output
rows of the unsharded layer exactly (every row of the fold equals the same row of
the unsharded layer, Section 3.1), from the full weights, in fp64.

With TSP_RESULTS_DIR set, each forward case appends its per-block max-rel / cosine and
the oracle's CPU seconds for the sampled rows to parity_fullsize.jsonl there.
"""
import json
import os
import time

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import tsp_oracle as O  # noqa: E402
from paper_2604_26294_amd import inputs as I  # noqa: E402
from paper_2604_26294_amd.harness import RankProblem  # noqa: E402
from paper_2604_26294_amd.workloads import L7B_8K, L7B_64K, L13B_B4, L70B_GQA, TINY  # noqa: E402
from tests.gpu_common import assert_close  # noqa: E402

CASES = [(TINY, 1), (L7B_8K, 7), (L7B_64K, 7), (L7B_64K.with_layout(1), 0), (L70B_GQA, 7),
         (L13B_B4, 0), (L13B_B4, 1), (L13B_B4, 2), (L13B_B4, 3),
         (L13B_B4.with_layout(1), 0), (L13B_B4.with_layout(1), 1),
         (L13B_B4.with_layout(1), 2), (L13B_B4.with_layout(1), 3)]
_cache = {}


def _data(wl):
    if _cache.get("name") != wl.name:
        _cache.clear()
        x = I.make_x_full(wl)
        w = I.make_weights(wl)
        _cache.update(name=wl.name, x=x, w=w, wf={k: I.bf16_bits_to_f64(v) for k, v in w.items()})
    return _cache["x"], _cache["w"], _cache["wf"]


def _rows(s_loc):
    """Both ends of the local rows and of each half (the zigzag layout's two chunks),
    and one row in every 128-row block at an offset that walks through the block (so
    every 256-query attention tile, every 128- or 256-row GEMM tile and every wavefront
    position within them is sampled somewhere)."""
    ends = {0, 1, 127, 128, s_loc // 2 - 1, s_loc // 2, s_loc // 2 + 7, s_loc - 1}
    blocks = {min(128 * i + (37 * i + 5) % 128, s_loc - 1) for i in range((s_loc + 127) // 128)}
    return sorted(r for r in ends | blocks if r < s_loc)


def _attention_rows(x_b, wf, wl, pos, chunk=16):
    """O.attention_rows over the positions in chunks (bounds the oracle's memory)."""
    return np.concatenate([O.attention_rows(x_b, wf["wq"], wf["wk"], wf["wv"], wf["wo"],
                                            wl.n_heads, wl.n_kv_heads, pos[i:i + chunk])
                           for i in range(0, len(pos), chunk)], axis=0)


@pytest.mark.parametrize("wl,p", CASES, ids=[f"{w.name}-{w.layout_name}-r{p}" for w, p in CASES])
def test_sampled_rows_match_unsharded_layer(wl, p):
    print(f"[fullsize] {wl.name} rank {p}", flush=True)
    x_bits, w_bits, wf = _data(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv()
    y_layer = prob.layer().clone()
    y_attn = prob.attn_fwd().clone()
    y_mlp = prob.mlp().clone()
    torch.cuda.synchronize()
    rows = _rows(wl.s_loc)
    batches = sorted({0, wl.batch - 1})
    if wl.layout == 1:
        pos = O.zigzag_positions(wl.seq, wl.degree, p)[rows]
    else:
        pos = [p * wl.s_loc + r for r in rows]
    record = {"workload": wl.name, "rank": p, "layout": wl.layout_name, "rows": len(rows),
              "batches": batches, "oracle_s": 0.0}
    for b in batches:
        t0 = time.perf_counter()
        x_b = I.bf16_bits_to_f64(x_bits[b, :max(pos) + 1])
        attn = _attention_rows(x_b, wf, wl, list(pos))
        xr = x_b[pos]
        mlp_x = O.mlp_full(xr, wf["w1"], wf["w3"], wf["w2"])
        u = xr + attn
        y = u + O.mlp_full(u, wf["w1"], wf["w3"], wf["w2"])
        record["oracle_s"] += time.perf_counter() - t0
        got = {k: v[b, rows].double().cpu().numpy()
               for k, v in (("attn", y_attn), ("mlp", y_mlp), ("layer", y_layer))}
        for blk, ref in (("attn", attn), ("mlp", mlp_x), ("layer", y)):
            mr, cos = assert_close(got[blk], ref, f"{wl.name} r{p} b{b} {blk}")
            worst = record.setdefault(blk, {"max_rel": 0.0, "cos": 1.0})
            worst["max_rel"] = max(worst["max_rel"], mr)
            worst["cos"] = min(worst["cos"], cos)
    out_dir = os.environ.get("TSP_RESULTS_DIR")
    if out_dir:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        record["oracle_threads"] = max((i.get("num_threads", 1) for i in blas), default=1)
        record["cpus_usable"] = len(os.sched_getaffinity(0))
        os.makedirs(out_dir, exist_ok=True)
        with open(os.path.join(out_dir, "parity_fullsize.jsonl"), "a") as f:
            f.write(json.dumps(record) + "\n")
    del prob
    torch.cuda.empty_cache()


BWD_CASES = [(L7B_64K, 7), (L70B_GQA, 7)]


@pytest.mark.parametrize("wl,p", BWD_CASES, ids=[f"{w.name}-r{p}" for w, p in BWD_CASES])
def test_mlp_backward_sampled_rows(wl, p):
    """The ring-MLP backward at full size: sampled rows of dX and sampled feature rows of
    two shards' weight gradients against the oracle's exact per-row sums."""
    from paper_2604_26294_amd.harness import local_rows, to_device_bf16
    print(f"[fullsize bwd] {wl.name} rank {p}", flush=True)
    x_bits, w_bits, wf = _data(wl)
    dy_bits = I.gaussian_bf16(wl.seed, I.TENSOR_ID["dy"], (wl.batch, wl.s_loc, wl.hidden),
                              wl.x_std)
    prob = RankProblem(wl, x_bits, w_bits, p)
    dx, dwg, dwu, dwd = prob.mlp_bwd(to_device_bf16(dy_bits))
    torch.cuda.synchronize()
    D, h = wl.degree, wl.hidden
    fs = wl.ffn // D
    m = wl.batch * wl.s_loc
    rows = sorted({0, 1, m // 2, m - 1})
    feats = sorted({0, 1, fs // 2, fs - 1})
    shards = sorted({p, (p + 1) % D})
    shard = [I.mlp_shard(wf, j, D) for j in range(D)]
    x2 = I.bf16_bits_to_f64(local_rows(x_bits, wl, p)).reshape(m, h)
    dy2 = I.bf16_bits_to_f64(dy_bits).reshape(m, h)
    ref_dx, ref_dw = O.mlp_rank_bwd_rows(x2, [s[0] for s in shard], [s[1] for s in shard],
                                         [s[2] for s in shard], dy2, rows, shards, feats)
    assert_close(dx.reshape(m, h)[rows].double().cpu().numpy(), ref_dx, f"{wl.name} dX rows")
    for j in shards:
        for name, got, ref in zip(("dW_gate", "dW_up", "dW_down"), (dwg[j], dwu[j], dwd[j]),
                                  ref_dw[j]):
            assert_close(got[feats].double().cpu().numpy(), ref, f"{wl.name} {name}[{j}] rows")
    del prob, dx, dwg, dwu, dwd
    torch.cuda.empty_cache()


@pytest.mark.parametrize("wl,p", BWD_CASES, ids=[f"{w.name}-r{p}" for w, p in BWD_CASES])
def test_attention_backward_full_size(wl, p):
    """The attention backward's first stage at full size, in the benchmark's launch
    configuration, on both paths (recomputing the forward, and from the A and log-sum-exp
    that the training forward kept): sampled rows of dX's query path (every head), and for
    the first head of the last shard every token's contribution to its W_Q and W_O^T
    gradient rows and, with one query head per kv head, every key's dK-hat / dV-hat, from
    the oracle's per-head attention backward in fp64."""
    from paper_2604_26294_amd.harness import to_device_bf16
    print(f"[fullsize attn bwd] {wl.name} rank {p}", flush=True)
    assert wl.layout == 0 and wl.batch == 1
    x_bits, w_bits, wf = _data(wl)
    dy_bits = I.gaussian_bf16(wl.seed, I.TENSOR_ID["dy"], (wl.batch, wl.s_loc, wl.hidden),
                              wl.x_std)
    D, d, s_loc = wl.degree, wl.head_dim, wl.s_loc
    kv_len = (p + 1) * s_loc
    g = wl.n_heads // wl.n_kv_heads
    hs, qd, kd = wl.n_heads // D, wl.n_heads // D * d, wl.n_kv_heads // D * d
    r, i = D - 1, 0
    gh = r * hs + i
    kvh = gh // g
    o0 = qd + 2 * kd
    rows = [0, 127, s_loc // 2, s_loc - 1]

    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv(include_self=True)
    dy = to_device_bf16(dy_bits)
    got = {}
    for path in ("recompute", "saved"):
        if path == "recompute":
            dx, dw, dk, dv = prob.attn_bwd(dy)
        else:
            prob.attn_fwd_train()
            dx, dw, dk, dv = prob.attn_bwd_saved(dy)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(dk).all()) and bool(torch.isfinite(dv).all()), path
        got[path] = {"dx": dx[0, rows].double().cpu().numpy(),
                     "dwq": dw[r][i * d:(i + 1) * d].double().cpu().numpy(),
                     "dwo": dw[r][o0 + i * d:o0 + (i + 1) * d].double().cpu().numpy(),
                     "dk": dk[0, :kv_len, kvh].double().cpu().numpy(),
                     "dv": dv[0, :kv_len, kvh].double().cpu().numpy()}
    del prob, dx, dw, dk, dv
    torch.cuda.empty_cache()

    x_b = I.bf16_bits_to_f64(x_bits[0, :kv_len])
    dy_loc = I.bf16_bits_to_f64(dy_bits[0])
    ref_dx = O.attention_bwd_rows(x_b, wf["wq"], wf["wk"], wf["wv"], wf["wo"], wl.n_heads,
                                  wl.n_kv_heads, [p * s_loc + r_ for r_ in rows], dy_loc[rows])
    x_loc = x_b[p * s_loc:]
    q = x_loc @ wf["wq"][gh * d:(gh + 1) * d].T
    k = x_b @ wf["wk"][kvh * d:(kvh + 1) * d].T
    v = x_b @ wf["wv"][kvh * d:(kvh + 1) * d].T
    da = dy_loc @ wf["wo"][:, gh * d:(gh + 1) * d]
    sc = 1.0 / np.sqrt(d)
    a = O.causal_attention_core(q, k, v, p * s_loc, sc)
    dq, dk_ref, dv_ref = O.causal_attention_core_bwd(q, k, v, da, p * s_loc, sc)
    for path, t in got.items():
        assert_close(t["dx"], ref_dx, f"{wl.name} {path} dX query-path rows")
        assert_close(t["dwq"], dq.T @ x_loc, f"{wl.name} {path} dW_Q head {gh}")
        assert_close(t["dwo"], a.T @ dy_loc, f"{wl.name} {path} dW_O^T head {gh}")
        if g == 1:
            assert_close(t["dk"], dk_ref, f"{wl.name} {path} dK-hat kv head {kvh}")
            assert_close(t["dv"], dv_ref, f"{wl.name} {path} dV-hat kv head {kvh}")
    for key in got["saved"]:
        assert_close(got["saved"][key], got["recompute"][key], f"{wl.name} saved vs recompute {key}")


def test_long_context_layer_output_is_finite_everywhere():
    """Every output element of the last rank of the long-context shape is finite."""
    wl = L7B_64K
    x_bits, w_bits, _ = _data(wl)
    prob = RankProblem(wl, x_bits, w_bits, 7)
    prob.prefill_kv()
    y = prob.layer()
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all())
    assert float(y.abs().max()) < 1e3
    np.testing.assert_equal(tuple(y.shape), (1, 8192, 4096))
