"""Pins of the oracle's attention backward (attn_rank_bwd, reduce_scatter_rows,
attn_kv_bwd in oracle.tsp_oracle).

Each is pinned to a forward that is already pinned, by a route that shares none of the
backward's formulas: central finite differences in fp64 of L = sum(dY * block output).
The whole two-stage backward, summed over ranks, must equal the gradient of the
unsharded attention block (sum-to-owner of each weight shard, and every rank's dX on
its own rows), in both sequence layouts; each rank's first stage alone must equal the
gradient of that rank's own forward with respect to its inputs and to the gathered
K-hat / V-hat it read.  A closed form (all-zero queries give uniform attention weights)
and the trivial cases complete the set.
"""
import numpy as np
import pytest

import oracle.tsp_oracle as O

EPS = 1e-6


def _problem(layout, seed=0, b=2, s=8, h=6, n_heads=4, n_kv=2, d=3, degree=2):
    rng = np.random.default_rng(seed)
    w = {
        "wq": rng.standard_normal((n_heads * d, h)) * 0.5,
        "wk": rng.standard_normal((n_kv * d, h)) * 0.5,
        "wv": rng.standard_normal((n_kv * d, h)) * 0.5,
        "wo": rng.standard_normal((h, n_heads * d)) * 0.5,
    }
    x = rng.standard_normal((b, s, h))
    dy = rng.standard_normal((b, s, h))
    return dict(x=x, w=w, dy=dy, n_heads=n_heads, n_kv=n_kv, d=d, degree=degree,
                layout=layout)


def _packed(w, r, degree, n_heads, n_kv, d):
    hs, ks = n_heads // degree * d, n_kv // degree * d
    return np.concatenate([w["wq"][r * hs:(r + 1) * hs], w["wk"][r * ks:(r + 1) * ks],
                           w["wv"][r * ks:(r + 1) * ks], w["wo"][:, r * hs:(r + 1) * hs].T])


def _two_stage(pb):
    """Run every rank's two stages and assemble the unsharded gradients."""
    x, w, dy = pb["x"], pb["w"], pb["dy"]
    D, nh, nkv, d, layout = pb["degree"], pb["n_heads"], pb["n_kv"], pb["d"], pb["layout"]
    seq = x.shape[1]
    shards = [_packed(w, r, D, nh, nkv, d) for r in range(D)]
    pos = [O.rank_positions(seq, D, p, layout) for p in range(D)]
    xs = [x[:, pos[p]] for p in range(D)]
    gather = O.gather_kv_zigzag if layout == "zigzag" else O.gather_kv
    kv = [gather(xs, shards[r], nh // D, nkv // D, d) for r in range(D)]
    first = [O.attn_rank_bwd(xs[p], shards, kv, p, nh, nkv, d, dy[:, pos[p]], layout=layout)
             for p in range(D)]
    dk_own = [O.reduce_scatter_rows([f["dk"][r] for f in first], D, layout) for r in range(D)]
    dv_own = [O.reduce_scatter_rows([f["dv"][r] for f in first], D, layout) for r in range(D)]
    dx = np.zeros_like(x)
    grads = {k: np.zeros_like(v) for k, v in w.items()}
    hs, ks = nh // D * d, nkv // D * d
    for p in range(D):
        dx2, dwk, dwv = O.attn_kv_bwd(xs[p], shards, [dk_own[r][p] for r in range(D)],
                                      [dv_own[r][p] for r in range(D)], nh, nkv, d)
        dx[:, pos[p]] += first[p]["dx"] + dx2
        for r in range(D):
            grads["wq"][r * hs:(r + 1) * hs] += first[p]["dwq"][r]
            grads["wo"][:, r * hs:(r + 1) * hs] += first[p]["dwo_t"][r].T
            grads["wk"][r * ks:(r + 1) * ks] += dwk[r]
            grads["wv"][r * ks:(r + 1) * ks] += dwv[r]
    return dx, grads


def _loss_full(pb):
    w = pb["w"]
    return float(np.sum(pb["dy"] * O.attention_full(pb["x"], w["wq"], w["wk"], w["wv"],
                                                    w["wo"], pb["n_heads"], pb["n_kv"])))


def _fd_dir(loss, arr, direction):
    old = arr.copy()
    arr += EPS * direction
    up = loss()
    arr[...] = old - EPS * direction
    dn = loss()
    arr[...] = old
    return (up - dn) / (2 * EPS)


@pytest.mark.parametrize("layout,n_heads,n_kv", [("contiguous", 4, 2), ("zigzag", 4, 2),
                                                 ("contiguous", 4, 4), ("zigzag", 2, 2)])
def test_two_stage_backward_is_the_unsharded_gradient(layout, n_heads, n_kv):
    pb = _problem(layout, n_heads=n_heads, n_kv=n_kv)
    dx, grads = _two_stage(pb)
    loss = lambda: _loss_full(pb)  # noqa: E731
    rng = np.random.default_rng(7)
    for arr, grad in [(pb["x"], dx)] + [(pb["w"][k], grads[k]) for k in ("wq", "wk", "wv", "wo")]:
        for _ in range(3):                       # random directions: one number checks all
            v = rng.standard_normal(arr.shape)
            fd = _fd_dir(loss, arr, v)
            assert abs(fd - np.sum(grad * v)) < 1e-7 * max(1.0, abs(fd))
        for _ in range(4):                       # and single entries
            idx = tuple(int(rng.integers(n)) for n in arr.shape)
            e = np.zeros_like(arr)
            e[idx] = 1.0
            fd = _fd_dir(loss, arr, e)
            assert abs(fd - grad[idx]) < 1e-7 * max(1.0, abs(fd))


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
def test_first_stage_is_the_gradient_of_the_rank_forward(layout):
    """dx, dwq, dwo_t and the K-hat / V-hat contributions of one rank are the gradients
    of that rank's own forward output with the gathered K-hat / V-hat held as inputs."""
    pb = _problem(layout, seed=3, n_heads=4, n_kv=2, degree=2)
    x, w = pb["x"], pb["w"]
    D, nh, nkv, d = pb["degree"], pb["n_heads"], pb["n_kv"], pb["d"]
    seq = x.shape[1]
    shards = [_packed(w, r, D, nh, nkv, d) for r in range(D)]
    pos = [O.rank_positions(seq, D, p, layout) for p in range(D)]
    xs = [x[:, pos[p]] for p in range(D)]
    gather = O.gather_kv_zigzag if layout == "zigzag" else O.gather_kv
    kv = [list(gather(xs, shards[r], nh // D, nkv // D, d)) for r in range(D)]
    fwd = O.attn_rank_zigzag if layout == "zigzag" else O.attn_rank
    rng = np.random.default_rng(11)
    for p in range(D):
        dyl = pb["dy"][:, pos[p]]
        xl = xs[p].copy()
        out = O.attn_rank_bwd(xl, shards, kv, p, nh, nkv, d, dyl, layout=layout)
        loss = lambda: float(np.sum(dyl * fwd(xl, shards, kv, p, nh, nkv, d)))  # noqa: E731
        v = rng.standard_normal(xl.shape)
        assert abs(_fd_dir(loss, xl, v) - np.sum(out["dx"] * v)) < 1e-7
        hs = nh // D * d
        for r in range(D):
            for key, lo in (("dwq", 0), ("dwo_t", hs + 2 * (nkv // D) * d)):
                v = rng.standard_normal(out[key][r].shape)
                direction = np.zeros_like(shards[r])
                direction[lo:lo + hs] = v
                fd = _fd_dir(loss, shards[r], direction)
                assert abs(fd - np.sum(out[key][r] * v)) < 1e-7 * max(1.0, abs(fd)), (p, r, key)
            for t, key in ((0, "dk"), (1, "dv")):
                v = rng.standard_normal(kv[r][t].shape)
                fd = _fd_dir(loss, kv[r][t], v)
                assert abs(fd - np.sum(out[key][r] * v)) < 1e-7 * max(1.0, abs(fd)), (p, r, key)
            # keys beyond every query of the rank get nothing
            last = int(pos[p].max())
            assert not np.any(out["dk"][r][:, last + 1:]) and not np.any(out["dv"][r][:, last + 1:])


def test_backward_special_cases():
    """dY = 0 gives zero gradients; zero queries give uniform weights, where dV and dQ
    have closed forms; the first position's query sees one key and gets dQ = 0."""
    pb = _problem("contiguous", seed=5, n_heads=2, n_kv=2, degree=1)
    pb["dy"][:] = 0.0
    dx, grads = _two_stage(pb)
    assert not np.any(dx) and all(not np.any(g) for g in grads.values())

    # one head, W_Q = 0: P_tj = 1/(t+1) for j <= t.
    rng = np.random.default_rng(2)
    s, d = 6, 3
    q = np.zeros((s, d))
    k, v, do = (rng.standard_normal((s, d)) for _ in range(3))
    dq, dk, dv = O.causal_attention_core_bwd(q, k, v, do, 0, 0.7)
    for j in range(s):
        want = sum(do[t] / (t + 1) for t in range(j, s))
        assert np.allclose(dv[j], want, rtol=0, atol=1e-13)
    assert np.allclose(dk, 0.0, atol=1e-15)     # dK = scale dS^T Q with Q = 0
    for t in range(s):
        dp = np.array([do[t] @ v[j] for j in range(t + 1)])
        ds = (dp - dp.mean()) / (t + 1)
        want = 0.7 * sum(ds[j] * k[j] for j in range(t + 1))
        assert np.allclose(dq[t], want, rtol=0, atol=1e-13)
    q = rng.standard_normal((s, d))
    dq, _, _ = O.causal_attention_core_bwd(q, k, v, do, 0, 0.7)
    assert np.allclose(dq[0], 0.0, atol=1e-15)


@pytest.mark.parametrize("n_heads,n_kv", [(4, 2), (4, 4)])
def test_sampled_rows_backward_is_the_query_path(n_heads, n_kv):
    """attention_bwd_rows (the full-size checker) against finite differences of the
    unsharded block with the input of the K / V projections held fixed, and against the
    query path of the first stage on every rank."""
    pb = _problem("contiguous", seed=9, n_heads=n_heads, n_kv=n_kv, degree=2)
    x, w, dy = pb["x"], pb["w"], pb["dy"]
    d, seq = pb["d"], x.shape[1]
    rows = np.array([0, 3, seq - 1])
    got = O.attention_bwd_rows(x[1], w["wq"], w["wk"], w["wv"], w["wo"], n_heads, n_kv, rows,
                               dy[1, rows])

    def block(xq):   # the attention block with queries from xq, keys / values from x
        b_, s_, _ = x.shape
        g = n_heads // n_kv
        q = (xq @ w["wq"].T).reshape(b_, s_, n_heads, d)
        k = (x @ w["wk"].T).reshape(b_, s_, n_kv, d)
        v = (x @ w["wv"].T).reshape(b_, s_, n_kv, d)
        a = np.empty_like(q)
        for b in range(b_):
            for i in range(n_heads):
                a[b, :, i] = O.causal_attention_core(q[b, :, i], k[b, :, i // g], v[b, :, i // g],
                                                     0, 1 / np.sqrt(d))
        return a.reshape(b_, s_, -1) @ w["wo"].T

    xq = x.copy()
    loss = lambda: float(np.sum(dy * block(xq)))  # noqa: E731
    rng = np.random.default_rng(4)
    for n, t in enumerate(rows):
        v = np.zeros_like(xq)
        v[1, t] = rng.standard_normal(x.shape[2])
        assert abs(_fd_dir(loss, xq, v) - got[n] @ v[1, t]) < 1e-7
    D = pb["degree"]
    shards = [_packed(w, r, D, n_heads, n_kv, d) for r in range(D)]
    xs = [x[:, O.rank_positions(seq, D, p, "contiguous")] for p in range(D)]
    kv = [O.gather_kv(xs, shards[r], n_heads // D, n_kv // D, d) for r in range(D)]
    s_loc = seq // D
    for n, t in enumerate(rows):
        p = t // s_loc
        out = O.attn_rank_bwd(xs[p], shards, kv, p, n_heads, n_kv, d, dy[:, p * s_loc:(p + 1) * s_loc])
        assert np.allclose(out["dx"][1, t - p * s_loc], got[n], rtol=1e-10, atol=1e-12)
