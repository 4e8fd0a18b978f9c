"""Pins of the oracle's ring-MLP backward (oracle.tsp_oracle.mlp_rank_bwd).

The backward is pinned to the oracle's own forward by a route that shares none of its
formulas: central finite differences of L = sum(dY * Y) in fp64.  Two identities that
the paper states for TSP's backward are checked the same way: summing a weight shard's
per-rank contributions over all ranks gives the gradient of the unsharded MLP
(sum-to-owner), and each rank's dX is the unsharded dX on its own rows.
"""
import numpy as np

import oracle.tsp_oracle as O

EPS = 1e-6


def _problem(seed=0, b=2, s=6, h=8, f=12, degree=3):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((b, s, h))
    w1 = rng.standard_normal((f, h)) * 0.4
    w3 = rng.standard_normal((f, h)) * 0.4
    w2 = rng.standard_normal((f, h)) * 0.4
    dy = rng.standard_normal((b, s, h))
    return x, w1, w3, w2, dy, degree


def _shards(w, degree):
    fs = w.shape[0] // degree
    return [w[j * fs:(j + 1) * fs].copy() for j in range(degree)]


def _loss_full(x, w1, w3, w2, dy):
    return float(np.sum(dy * O.mlp_full(x, w1, w3, w2)))


def _fd(fn, arr, idx):
    old = arr[idx]
    arr[idx] = old + EPS
    up = fn()
    arr[idx] = old - EPS
    dn = fn()
    arr[idx] = old
    return (up - dn) / (2 * EPS)


def test_rank_backward_matches_finite_differences():
    x, w1, w3, w2, dy, degree = _problem()
    s_loc = x.shape[1] // degree
    rng = np.random.default_rng(1)
    for p in range(degree):
        xl = x[:, p * s_loc:(p + 1) * s_loc].copy()
        dyl = dy[:, p * s_loc:(p + 1) * s_loc]
        s1, s3, s2 = _shards(w1, degree), _shards(w3, degree), _shards(w2, degree)
        dx, dw1, dw3, dw2 = O.mlp_rank_bwd(xl, s1, s3, s2, dyl, p)
        loss = lambda: float(np.sum(dyl * O.mlp_rank(xl, s1, s3, s2, p)))  # noqa: E731
        for _ in range(6):
            idx = tuple(int(rng.integers(n)) for n in xl.shape)
            assert abs(_fd(loss, xl, idx) - dx[idx]) < 1e-7 * max(1.0, abs(dx[idx]))
        for arrs, grads in ((s1, dw1), (s3, dw3), (s2, dw2)):
            for _ in range(4):
                j = int(rng.integers(degree))
                idx = tuple(int(rng.integers(n)) for n in arrs[j].shape)
                g = grads[j][idx]
                assert abs(_fd(loss, arrs[j], idx) - g) < 1e-7 * max(1.0, abs(g))


def test_weight_gradients_sum_to_owner_and_dx_is_local():
    x, w1, w3, w2, dy, degree = _problem(seed=3)
    s_loc = x.shape[1] // degree
    fs = w1.shape[0] // degree
    s1, s3, s2 = _shards(w1, degree), _shards(w3, degree), _shards(w2, degree)
    tot = {"w1": np.zeros_like(w1), "w3": np.zeros_like(w3), "w2": np.zeros_like(w2)}
    dx_ranks = []
    for p in range(degree):
        sl = slice(p * s_loc, (p + 1) * s_loc)
        dx, dw1, dw3, dw2 = O.mlp_rank_bwd(x[:, sl], s1, s3, s2, dy[:, sl], p)
        dx_ranks.append(dx)
        for j in range(degree):
            rows = slice(j * fs, (j + 1) * fs)
            tot["w1"][rows] += dw1[j]
            tot["w3"][rows] += dw3[j]
            tot["w2"][rows] += dw2[j]
    rng = np.random.default_rng(4)
    loss = lambda: _loss_full(x, w1, w3, w2, dy)  # noqa: E731
    for name, w in (("w1", w1), ("w3", w3), ("w2", w2)):
        for _ in range(6):
            idx = tuple(int(rng.integers(n)) for n in w.shape)
            g = tot[name][idx]
            assert abs(_fd(loss, w, idx) - g) < 1e-7 * max(1.0, abs(g)), name
    dx_all = np.concatenate(dx_ranks, axis=1)
    for _ in range(8):
        idx = tuple(int(rng.integers(n)) for n in x.shape)
        assert abs(_fd(loss, x, idx) - dx_all[idx]) < 1e-7 * max(1.0, abs(dx_all[idx]))


def test_backward_special_cases():
    x, w1, w3, w2, dy, degree = _problem(seed=5)
    s1, s3, s2 = _shards(w1, degree), _shards(w3, degree), _shards(w2, degree)
    xl = x[:, :2]
    # zero upstream gradient -> zero everywhere; the map is linear in dY
    dx0, a, b, c = O.mlp_rank_bwd(xl, s1, s3, s2, np.zeros_like(xl), 1)
    assert not np.any(dx0) and not any(np.any(m) for m in a + b + c)
    dxa, *_ = O.mlp_rank_bwd(xl, s1, s3, s2, dy[:, :2], 1)
    dxb, *_ = O.mlp_rank_bwd(xl, s1, s3, s2, 3 * dy[:, :2], 1)
    assert np.allclose(dxb, 3 * dxa, rtol=1e-12, atol=1e-12)
    # SiLU'(0) = 1/2 and SiLU' tends to 1 / 0 for large positive / negative z
    assert O.silu_grad(np.array([0.0]))[0] == 0.5
    assert abs(O.silu_grad(np.array([40.0]))[0] - 1.0) < 1e-12
    assert abs(O.silu_grad(np.array([-40.0]))[0]) < 1e-12


def test_sampled_rows_equal_the_full_backward():
    x, w1, w3, w2, dy, degree = _problem(seed=7)
    s1, s3, s2 = _shards(w1, degree), _shards(w3, degree), _shards(w2, degree)
    xl, dyl = x[:, 2:4], dy[:, 2:4]
    dx, dw1, dw3, dw2 = O.mlp_rank_bwd(xl, s1, s3, s2, dyl, 1)
    h = x.shape[-1]
    rows, feats, shards = [0, 3], [1, 2], [0, 2]
    dxr, dwr = O.mlp_rank_bwd_rows(xl.reshape(-1, h), s1, s3, s2, dyl.reshape(-1, h), rows,
                                   shards, feats)
    assert np.allclose(dxr, dx.reshape(-1, h)[rows], rtol=1e-12, atol=1e-12)
    for j in shards:
        for got, full in zip(dwr[j], (dw1[j], dw3[j], dw2[j])):
            assert np.allclose(got, full[feats], rtol=1e-12, atol=1e-12)
