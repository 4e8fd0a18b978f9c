"""fp64 oracle for the per-rank forward of a folded TSP transformer layer.

TEST INFRASTRUCTURE ONLY -- imported by tests/, the smoke check and the benchmark's
CPU-baseline leg; never by the product path.  Shares no code with the HIP library.

Every array argument holds float64 values (the caller converts bf16 bit patterns
with the input generator).  Nothing here rounds to bf16: the GPU path rounds some
intermediates (Q, K, V, P, A, the gated product, the layer's MLP input) and the
tests absorb that in their tolerance.

Conventions (paper, Sections 3-4):
  x        [B, S, h]  layer input;  rank p holds the contiguous chunk
           x[:, p*S_loc:(p+1)*S_loc], S_loc = S/D (or, in the zigzag layout,
           the rows at zigzag_positions(S, D, p)).
  W_Q      [n_h d, h], W_K / W_V [n_kv d, h]; Q = X W_Q^T etc.
  W_O      [h, n_h d]; the attention block returns Flatten(A) W_O^T.
  W1 (gate), W3 (up), W2 (down)  [F, h]; MLP(u) = (SiLU(u W1^T) * (u W3^T)) W2.
  Query head i reads key/value head floor(i / g), g = n_h / n_kv (GQA).
  Softmax scale defaults to 1/sqrt(d).
  Causal rule: a query at global position t sees keys at positions j <= t.
"""
from __future__ import annotations

import math

import numpy as np

_Q_CHUNK = 512


# ---------------------------------------------------------------------------
# Shared definitions of the two nonlinear pieces.
# ---------------------------------------------------------------------------

def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z * sigmoid(z): the gate activation of a SwiGLU MLP (Section 4 model)."""
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def _positions(q_pos, lq: int) -> np.ndarray:
    """Global positions of Lq query rows: q_pos itself (one per row), or, for an
    integer, the consecutive positions q_pos, q_pos + 1, ..."""
    if np.ndim(q_pos) == 0:
        return int(q_pos) + np.arange(lq)
    return np.asarray(q_pos)


def causal_probs(q: np.ndarray, k: np.ndarray, q_pos, scale: float) -> np.ndarray:
    """Softmax probabilities P[i, j] of query row i over keys j (key j at position j),
    with the keys after the row's global position masked out; q_pos gives the rows'
    positions (or the first of consecutive ones).  q [Lq, d], k [Lk, d]."""
    s = (q @ k.T) * scale
    lq, lk = s.shape
    allowed = np.arange(lk)[None, :] <= _positions(q_pos, lq)[:, None]
    s = np.where(allowed, s, -np.inf)
    s = s - s.max(axis=1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=1, keepdims=True)


def causal_attention_core(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos,
                          scale: float) -> np.ndarray:
    """o_i = sum_j P[i, j] v_j for one head; q [Lq, d], k/v [Lk, d] -> [Lq, d].

    Query row i sits at global position q_pos[i] (or q_pos + i for an integer) and sees
    the keys at positions j <= that position: causal attention of any set of query rows
    against keys held in sequence order (Algorithm 1's CausalAttn with its alignment).
    Queries are processed in chunks only to bound memory.
    """
    lq = q.shape[0]
    pos = _positions(q_pos, lq)
    out = np.empty((lq, v.shape[1]), dtype=np.float64)
    for lo in range(0, lq, _Q_CHUNK):
        hi = min(lq, lo + _Q_CHUNK)
        kmax = min(k.shape[0], int(pos[lo:hi].max()) + 1)  # later keys are masked for the chunk
        p = causal_probs(q[lo:hi], k[:kmax], pos[lo:hi], scale)
        out[lo:hi] = p @ v[:kmax]
    return out


def default_scale(head_dim: int, scale: float | None) -> float:
    return 1.0 / math.sqrt(head_dim) if scale is None or scale <= 0 else float(scale)


# ---------------------------------------------------------------------------
# O1 -- the unsharded layer (what the folded schedule must reproduce).
# ---------------------------------------------------------------------------

def attention_full(x, wq, wk, wv, wo, n_heads, n_kv_heads, scale=None):
    """Causal multi-head / grouped-query attention block on the whole sequence.

    Section 4 model: learned Q, K, V, O projections, no biases, no positional
    encoding, no normalisation.  x [B, S, h] -> [B, S, h].
    """
    b_, s_, _ = x.shape
    d = wq.shape[0] // n_heads
    g = n_heads // n_kv_heads
    sc = default_scale(d, scale)
    q = (x @ wq.T).reshape(b_, s_, n_heads, d)
    k = (x @ wk.T).reshape(b_, s_, n_kv_heads, d)
    v = (x @ wv.T).reshape(b_, s_, n_kv_heads, d)
    a = np.empty((b_, s_, n_heads, d), dtype=np.float64)
    for b in range(b_):
        for i in range(n_heads):
            a[b, :, i] = causal_attention_core(q[b, :, i], k[b, :, i // g], v[b, :, i // g], 0, sc)
    return a.reshape(b_, s_, n_heads * d) @ wo.T


def mlp_full(u, w1, w3, w2):
    """Gated MLP: (SiLU(u W1^T) * (u W3^T)) W2, Algorithm 2's three projections unsharded."""
    return (silu(u @ w1.T) * (u @ w3.T)) @ w2


def layer_full(x, w, n_heads, n_kv_heads, scale=None):
    """Pre-norm residual layer with the norms left out (Section 4 model):
    u = x + Attn(x);  y = u + MLP(u).  Returns every block output."""
    attn = attention_full(x, w["wq"], w["wk"], w["wv"], w["wo"], n_heads, n_kv_heads, scale)
    u = x + attn
    mlp = mlp_full(u, w["w1"], w["w3"], w["w2"])
    return {"attn": attn, "u": u, "mlp": mlp, "y": u + mlp}


# ---------------------------------------------------------------------------
# O2 -- the folded per-rank computation (Algorithms 1 and 2), from the definitions:
# a rank's block output is the sum over all weight shards of that shard's term for the
# rank's own tokens.
# ---------------------------------------------------------------------------

def ring_order(p, degree):
    """The order in which rank p applies the MLP shards (Algorithm 2): the shard that
    started on rank j reaches rank p after (p - j) mod D hand-offs to the right."""
    return [(p - t) % degree for t in range(degree)]


def mlp_rank(x_loc, w1_shards, w3_shards, w2_shards, p):
    """Rank p's output of the folded gated MLP (Algorithm 2), x_loc [B, S_loc, h].

    The MLP acts on each token separately and shard j holds rows j F/D .. (j+1) F/D - 1
    of W1, W3 and W2, so the MLP of the rank's tokens is the sum over the shards of
    (SiLU(X W1_j^T) * (X W3_j^T)) W2_j, here added in ring_order(p, D).
    """
    terms = ((silu(x_loc @ w1_shards[j].T) * (x_loc @ w3_shards[j].T)) @ w2_shards[j]
             for j in ring_order(p, len(w1_shards)))
    return sum(terms, np.zeros_like(x_loc, dtype=np.float64))


# ---------------------------------------------------------------------------
# Backward of the ring MLP (per rank).  The paper costs TSP's backward (Section 4: it
# mirrors the forward weight movement, and each weight shard's partial gradients are
# summed to the shard's owner) but prints no algorithm; these are the gradients of
# Algorithm 2's forward, by the chain rule.
# ---------------------------------------------------------------------------

def silu_grad(z: np.ndarray) -> np.ndarray:
    """d SiLU(z) / dz = sigmoid(z) (1 + z (1 - sigmoid(z)))."""
    with np.errstate(over="ignore"):
        sg = 1.0 / (1.0 + np.exp(-z))
    return sg * (1.0 + z * (1.0 - sg))


def swiglu_bwd(g, u, dhs):
    """Gradients of Hs = SiLU(G) * U with respect to G and U, given dL/dHs."""
    return dhs * u * silu_grad(g), dhs * silu(g)


def mlp_rank_bwd(x_loc, w1_shards, w3_shards, w2_shards, dy, p):
    """Backward of mlp_rank on rank p for the upstream gradient dy = dL/dY
    [B, S_loc, h].  Visits the shards in the forward's ring order and returns dX
    [B, S_loc, h] and this rank's contribution to each shard's weight gradients:
    lists dW1, dW3, dW2 indexed by shard, [F/D, h] each.  Summing shard j's
    contributions over the D ranks gives the gradient of shard j (sum-to-owner)."""
    degree = len(w1_shards)
    h = x_loc.shape[-1]
    x2 = x_loc.reshape(-1, h)
    dy2 = dy.reshape(-1, h)
    dx = np.zeros_like(x2, dtype=np.float64)
    dw1, dw3, dw2 = [None] * degree, [None] * degree, [None] * degree
    for t in range(degree):
        j = (p - t) % degree
        g = x2 @ w1_shards[j].T
        u = x2 @ w3_shards[j].T
        dhs = dy2 @ w2_shards[j].T
        dg, du = swiglu_bwd(g, u, dhs)
        dx += dg @ w1_shards[j] + du @ w3_shards[j]
        dw1[j] = dg.T @ x2
        dw3[j] = du.T @ x2
        dw2[j] = (silu(g) * u).T @ dy2
    return dx.reshape(x_loc.shape), dw1, dw3, dw2


def mlp_rank_bwd_rows(x2, w1_shards, w3_shards, w2_shards, dy2, rows, shards, feats):
    """Selected entries of mlp_rank_bwd for large shapes, each computed exactly from its
    own definition: dX rows `rows` (sum over every shard) and, for each shard j in
    `shards`, rows `feats` of dW1_j, dW3_j, dW2_j (sums over every token).  x2 and dy2
    are the rank's tokens flattened, [M, h].  Returns (dx [len(rows), h], {j: (dW1,
    dW3, dW2) rows [len(feats), h]})."""
    dx = np.zeros((len(rows), x2.shape[1]))
    for j in range(len(w1_shards)):
        xr, dyr = x2[rows], dy2[rows]
        dg, du = swiglu_bwd(xr @ w1_shards[j].T, xr @ w3_shards[j].T, dyr @ w2_shards[j].T)
        dx += dg @ w1_shards[j] + du @ w3_shards[j]
    dw = {}
    for j in shards:
        g = x2 @ w1_shards[j][feats].T          # [M, len(feats)]: columns feats of G
        u = x2 @ w3_shards[j][feats].T
        dhs = dy2 @ w2_shards[j][feats].T
        dg, du = swiglu_bwd(g, u, dhs)
        dw[j] = (dg.T @ x2, du.T @ x2, (silu(g) * u).T @ dy2)
    return dx, dw


def unpack_attn_shard(packed, heads_per_shard, kv_heads_per_shard, head_dim):
    """Split a packed shard [W_Q^(r); W_K^(r); W_V^(r); W_O^(r)^T] (Algorithm 1's
    packed broadcast buffer) into its four row blocks."""
    hs = heads_per_shard * head_dim
    ks = kv_heads_per_shard * head_dim
    wq = packed[:hs]
    wk = packed[hs:hs + ks]
    wv = packed[hs + ks:hs + 2 * ks]
    wo_t = packed[hs + 2 * ks:hs + 2 * ks + hs]
    assert wo_t.shape[0] == hs, "packed shard has the wrong number of rows"
    return wq, wk, wv, wo_t


def kv_project(x_chunk, packed, heads_per_shard, kv_heads_per_shard, head_dim):
    """One rank's K, V for shard r on its own tokens: [B, S_loc, K_s, d] each.
    This is what the rank contributes to the sequence-wise all-gather."""
    _, wk, wv, _ = unpack_attn_shard(packed, heads_per_shard, kv_heads_per_shard, head_dim)
    b_, s_loc, _ = x_chunk.shape
    k = (x_chunk @ wk.T).reshape(b_, s_loc, kv_heads_per_shard, head_dim)
    v = (x_chunk @ wv.T).reshape(b_, s_loc, kv_heads_per_shard, head_dim)
    return k, v


def gather_kv(x_chunks, packed, heads_per_shard, kv_heads_per_shard, head_dim):
    """The sequence-wise all-gather of shard r's K and V over all ranks, in
    sequence order (contiguous chunks need no reordering): [B, S, K_s, d]."""
    parts = [kv_project(xc, packed, heads_per_shard, kv_heads_per_shard, head_dim)
             for xc in x_chunks]
    return (np.concatenate([k for k, _ in parts], axis=1),
            np.concatenate([v for _, v in parts], axis=1))


def attn_rank(x_loc, shards, kv_gathered, p, n_heads, n_kv_heads, head_dim, scale=None,
              rows=None, positions=None):
    """Rank p's output of the folded attention block (Algorithm 1), x_loc [B, S_loc, h].

    Shard r holds query heads r H_s .. (r+1) H_s - 1 (their W_Q rows and W_O columns) and
    kv heads r K_s .. (r+1) K_s - 1, whose keys and values for the whole sequence are
    ``kv_gathered[r]`` (the all-gather, in sequence order: :func:`gather_kv` or
    :func:`gather_kv_zigzag`).  The block output of a token is the sum over the shards of
    Flatten(A_r) W_O^(r)^T, A_r the causal attention of the shard's query heads of that
    token, at its global position, over the shard's keys.  The rank's local row t sits at
    ``positions[t]`` (default p S_loc + t: contiguous chunks).  ``rows`` optionally
    restricts the computation to some local rows (a row depends only on its own query).
    """
    degree = len(shards)
    hs_heads = n_heads // degree
    ks_heads = n_kv_heads // degree
    g = n_heads // n_kv_heads
    d = head_dim
    sc = default_scale(d, scale)
    b_, s_loc, h = x_loc.shape
    pos = p * s_loc + np.arange(s_loc) if positions is None else np.asarray(positions)
    if rows is not None:
        x_loc, pos = x_loc[:, rows], pos[np.asarray(rows)]
    lq = x_loc.shape[1]
    y = np.zeros((b_, lq, h), dtype=np.float64)
    for r in range(degree):
        wq, _, _, wo_t = unpack_attn_shard(shards[r], hs_heads, ks_heads, d)
        q = (x_loc @ wq.T).reshape(b_, lq, hs_heads, d)
        k_hat, v_hat = kv_gathered[r]
        a = np.empty((b_, lq, hs_heads, d), dtype=np.float64)
        for b in range(b_):
            for i in range(hs_heads):
                a[b, :, i] = causal_attention_core(q[b, :, i], k_hat[b, :, i // g],
                                                   v_hat[b, :, i // g], pos, sc)
        y += a.reshape(b_, lq, hs_heads * d) @ wo_t
    return y


def layer_rank(x_chunks, attn_shards, w1_shards, w3_shards, w2_shards, p, n_heads,
               n_kv_heads, head_dim, scale=None):
    """One rank's layer forward: u = x_loc + TSP-Attn(x), y = u + TSP-MLP(u).

    The K/V all-gather is built from every rank's chunk of the layer input.
    Returns the block outputs and the layer output for rank p's tokens.
    """
    degree = len(attn_shards)
    hsh, ksh = n_heads // degree, n_kv_heads // degree
    kv = [gather_kv(x_chunks, attn_shards[r], hsh, ksh, head_dim) for r in range(degree)]
    x_loc = x_chunks[p]
    attn = attn_rank(x_loc, attn_shards, kv, p, n_heads, n_kv_heads, head_dim, scale)
    u = x_loc + attn
    mlp = mlp_rank(u, w1_shards, w3_shards, w2_shards, p)
    return {"attn": attn, "u": u, "mlp": mlp, "y": u + mlp}


# ---------------------------------------------------------------------------
# O2, zigzag layout (Algorithm 1's load-balanced causal partition).
# ---------------------------------------------------------------------------

def zigzag_positions(seq, degree, p):
    """Global positions of rank p's local rows in the zigzag layout.

    The sequence is cut into 2D chunks of S_c = S / (2D) tokens; rank p holds chunk p
    followed by chunk 2D - 1 - p (Section 2 on causal load balancing; Algorithm 1's
    S_c = S_loc / 2), so its local rows are [chunk p; chunk 2D-1-p]."""
    s_c = seq // (2 * degree)
    return np.concatenate([p * s_c + np.arange(s_c),
                           (2 * degree - 1 - p) * s_c + np.arange(s_c)])


def gather_kv_zigzag(x_shards, packed, heads_per_shard, kv_heads_per_shard, head_dim):
    """Shard r's K and V over ranks holding zigzag shards: the all-gather
    concatenates the ranks' rows in rank order, then ZigZagReorder puts every row
    back at its global position, giving sequence order [B, S, K_s, d]."""
    degree = len(x_shards)
    parts = [kv_project(xs, packed, heads_per_shard, kv_heads_per_shard, head_dim)
             for xs in x_shards]
    k_cat = np.concatenate([k for k, _ in parts], axis=1)
    v_cat = np.concatenate([v for _, v in parts], axis=1)
    seq = k_cat.shape[1]
    # row n of the gathered tensor came from global position order[n]
    order = np.concatenate([zigzag_positions(seq, degree, q) for q in range(degree)])
    k_hat = np.empty_like(k_cat)
    v_hat = np.empty_like(v_cat)
    k_hat[:, order] = k_cat
    v_hat[:, order] = v_cat
    return k_hat, v_hat


def attn_rank_zigzag(x_loc, shards, kv_gathered, p, n_heads, n_kv_heads, head_dim,
                     scale=None):
    """Rank p's output of the folded attention block with zigzag shards (Algorithm 1):
    :func:`attn_rank` with the local rows at ``zigzag_positions(S, D, p)`` and the
    gathered keys in sequence order (:func:`gather_kv_zigzag`).  Algorithm 1's two
    CausalAttn calls, the first half of the rows against the first s1 = (p+1) S_c keys
    and the second against the first s2 = (2D - p) S_c, are this per-row causal rule:
    the last row of each half sits at position s1 - 1 and s2 - 1."""
    seq = kv_gathered[0][0].shape[1]
    return attn_rank(x_loc, shards, kv_gathered, p, n_heads, n_kv_heads, head_dim, scale,
                     positions=zigzag_positions(seq, len(shards), p))


def layer_rank_zigzag(x_shards, attn_shards, w1_shards, w3_shards, w2_shards, p, n_heads,
                      n_kv_heads, head_dim, scale=None):
    """One rank's layer forward with zigzag shards: u = x_loc + TSP-Attn(x),
    y = u + TSP-MLP(u) (the MLP is row-local, so its ring is unchanged)."""
    degree = len(attn_shards)
    hsh, ksh = n_heads // degree, n_kv_heads // degree
    kv = [gather_kv_zigzag(x_shards, attn_shards[r], hsh, ksh, head_dim)
          for r in range(degree)]
    x_loc = x_shards[p]
    attn = attn_rank_zigzag(x_loc, attn_shards, kv, p, n_heads, n_kv_heads, head_dim, scale)
    u = x_loc + attn
    mlp = mlp_rank(u, w1_shards, w3_shards, w2_shards, p)
    return {"attn": attn, "u": u, "mlp": mlp, "y": u + mlp}


# ---------------------------------------------------------------------------
# Backward of the attention block (per rank).  As for the MLP, the paper costs the
# backward (Section 4) without printing it; these are the chain-rule gradients of
# Algorithm 1's forward.  The all-gather of K and V becomes, in the backward, a
# reduce-scatter of their gradients, so the work splits in two stages: every rank
# produces contributions to the gradient of the whole gathered K-hat / V-hat of each
# shard (attn_rank_bwd); the sum over ranks, restricted to a rank's own rows, is what
# that rank back-propagates through its K / V projections (attn_kv_bwd).
# ---------------------------------------------------------------------------

def causal_attention_core_bwd(q, k, v, do, q_offset, scale):
    """Gradients of o = causal_attention_core(q, k, v, q_offset, scale) for one head,
    given do = dL/do [Lq, d].  With P the masked softmax of scale q k^T and o = P v:
      dv = P^T do,   dP = do v^T,   dS_tj = P_tj (dP_tj - sum_m P_tm dP_tm),
      dq = scale dS k,   dk = scale dS^T q.
    Returns dq [Lq, d], dk [Lk, d], dv [Lk, d] (keys no query sees get zero)."""
    lq = q.shape[0]
    dq = np.zeros_like(q, dtype=np.float64)
    dk = np.zeros_like(k, dtype=np.float64)
    dv = np.zeros_like(v, dtype=np.float64)
    for lo in range(0, lq, _Q_CHUNK):
        hi = min(lq, lo + _Q_CHUNK)
        kmax = min(k.shape[0], q_offset + hi)
        p = causal_probs(q[lo:hi], k[:kmax], q_offset + lo, scale)
        dp = do[lo:hi] @ v[:kmax].T
        ds = p * (dp - np.sum(p * dp, axis=1, keepdims=True))
        dv[:kmax] += p.T @ do[lo:hi]
        dq[lo:hi] = scale * (ds @ k[:kmax])
        dk[:kmax] += scale * (ds.T @ q[lo:hi])
    return dq, dk, dv


def rank_positions(seq, degree, p, layout):
    """Global positions of rank p's local rows: a contiguous chunk, or the zigzag pair."""
    if layout == "zigzag":
        return zigzag_positions(seq, degree, p)
    s_loc = seq // degree
    return p * s_loc + np.arange(s_loc)


def causal_calls(s_loc, degree, p, layout):
    """Algorithm 1's CausalAttn calls on rank p as (first local row, end row, global
    position of the first row, number of gathered keys the block attends to)."""
    if layout == "zigzag":
        s_c = s_loc // 2
        s1, s2 = (p + 1) * s_c, (2 * degree - p) * s_c
        return [(0, s_c, s1 - s_c, s1), (s_c, s_loc, s2 - s_c, s2)]
    return [(0, s_loc, p * s_loc, (p + 1) * s_loc)]


def attn_rank_bwd(x_loc, shards, kv_gathered, p, n_heads, n_kv_heads, head_dim, dy,
                  scale=None, layout="contiguous"):
    """First stage of the attention backward on rank p, for dy = dL/dY [B, S_loc, h].

    For each shard r: recompute Q = X W_Q^(r)^T and A as the forward does; the block
    output is Flatten(A) W_O^(r)^T, so dA = dY W_O^(r) and W_O^(r)^T's gradient gets
    A^T dY; per query head, the causal attention backward against the gathered K-hat,
    V-hat of shard r (prefix and alignment of each CausalAttn call as in the forward);
    then dX gets dQ W_Q^(r) and W_Q^(r) gets dQ^T X.

    Returns a dict:
      dx        [B, S_loc, h]         the query path's part of dX;
      dwq[r]    [H_s d, h]            this rank's contribution to dW_Q^(r);
      dwo_t[r]  [H_s d, h]            its contribution to the gradient of W_O^(r)^T
                                      (the packed shard's last block);
      dk[r], dv[r]  [B, S, K_s, d]    its contributions to the gradients of shard r's
                                      gathered K-hat and V-hat, in sequence order (zero
                                      for keys none of its queries sees).
    """
    degree = len(shards)
    hs_heads, ks_heads = n_heads // degree, n_kv_heads // degree
    g = n_heads // n_kv_heads
    d = head_dim
    sc = default_scale(d, scale)
    b_, s_loc, h = x_loc.shape
    calls = causal_calls(s_loc, degree, p, layout)
    x2 = x_loc.reshape(-1, h)
    dy2 = dy.reshape(-1, h)
    dx = np.zeros_like(x2, dtype=np.float64)
    out = {"dwq": [None] * degree, "dwo_t": [None] * degree,
           "dk": [None] * degree, "dv": [None] * degree}
    for r in range(degree):
        wq, _, _, wo_t = unpack_attn_shard(shards[r], hs_heads, ks_heads, d)
        k_hat, v_hat = kv_gathered[r]
        q = (x_loc @ wq.T).reshape(b_, s_loc, hs_heads, d)
        da = (dy @ wo_t.T).reshape(b_, s_loc, hs_heads, d)
        a = np.empty_like(q)
        dq = np.empty_like(q)
        dk = np.zeros_like(k_hat, dtype=np.float64)
        dv = np.zeros_like(v_hat, dtype=np.float64)
        for b in range(b_):
            for i in range(hs_heads):
                kh = i // g
                for lo, hi, off, n_keys in calls:
                    kk, vv = k_hat[b, :n_keys, kh], v_hat[b, :n_keys, kh]
                    a[b, lo:hi, i] = causal_attention_core(q[b, lo:hi, i], kk, vv, off, sc)
                    gq, gk, gv = causal_attention_core_bwd(q[b, lo:hi, i], kk, vv,
                                                           da[b, lo:hi, i], off, sc)
                    dq[b, lo:hi, i] = gq
                    dk[b, :n_keys, kh] += gk
                    dv[b, :n_keys, kh] += gv
        dq2 = dq.reshape(-1, hs_heads * d)
        dx += dq2 @ wq
        out["dwq"][r] = dq2.T @ x2
        out["dwo_t"][r] = a.reshape(-1, hs_heads * d).T @ dy2
        out["dk"][r], out["dv"][r] = dk, dv
    out["dx"] = dx.reshape(x_loc.shape)
    return out


def reduce_scatter_rows(contribs, degree, layout):
    """The backward of the sequence-wise all-gather: sum the ranks' contributions
    [B, S, ...] and hand rank q the rows at its own positions."""
    total = np.sum(contribs, axis=0)
    seq = total.shape[1]
    return [total[:, rank_positions(seq, degree, q, layout)] for q in range(degree)]


def attn_kv_bwd(x_loc, shards, dk_own, dv_own, n_heads, n_kv_heads, head_dim):
    """Second stage of the attention backward on one rank: K = X W_K^(r)^T and
    V = X W_V^(r)^T on its own rows, so with dk_own[r], dv_own[r] [B, S_loc, K_s, d] the
    reduce-scattered gradients of its rows of K-hat, V-hat: dX gets dK W_K^(r) + dV W_V^(r),
    and the rank contributes dK^T X to dW_K^(r) and dV^T X to dW_V^(r).
    Returns (dx [B, S_loc, h], dwk list, dwv list)."""
    degree = len(shards)
    hs_heads, ks_heads = n_heads // degree, n_kv_heads // degree
    h = x_loc.shape[-1]
    x2 = x_loc.reshape(-1, h)
    dx = np.zeros_like(x2, dtype=np.float64)
    dwk, dwv = [None] * degree, [None] * degree
    for r in range(degree):
        _, wk, wv, _ = unpack_attn_shard(shards[r], hs_heads, ks_heads, head_dim)
        gk = dk_own[r].reshape(-1, ks_heads * head_dim)
        gv = dv_own[r].reshape(-1, ks_heads * head_dim)
        dx += gk @ wk + gv @ wv
        dwk[r] = gk.T @ x2
        dwv[r] = gv.T @ x2
    return dx.reshape(x_loc.shape), dwk, dwv


# ---------------------------------------------------------------------------
# Sampled rows of the unsharded attention block, for full-size checks.
# ---------------------------------------------------------------------------

def attention_rows(x_b, wq, wk, wv, wo, n_heads, n_kv_heads, positions, scale=None):
    """Attention-block output rows at the given global positions of one sequence.

    x_b [S, h] is one batch entry of the layer input.  Uses only associativity of
    the matrix products: the score of key j is (W_K,i^T q_t) . x_j and the context
    is W_V,i (sum_j P_tj x_j), so no K or V for the whole prefix is ever formed.
    Returns [len(positions), h].
    """
    positions = np.asarray(positions, dtype=np.int64)
    d = wq.shape[0] // n_heads
    g = n_heads // n_kv_heads
    sc = default_scale(d, scale)
    t_max = int(positions.max()) + 1
    x_pre = x_b[:t_max]
    n_r = positions.shape[0]
    q = (x_b[positions] @ wq.T).reshape(n_r, n_heads, d)
    wk_h = wk.reshape(n_kv_heads, d, -1)
    wv_h = wv.reshape(n_kv_heads, d, -1)
    u = np.empty((n_r, n_heads, x_b.shape[1]), dtype=np.float64)
    for i in range(n_heads):
        u[:, i] = q[:, i] @ wk_h[i // g]
    s = (u.reshape(n_r * n_heads, -1) @ x_pre.T) * sc
    pos_rows = np.repeat(positions, n_heads)
    allowed = np.arange(t_max)[None, :] <= pos_rows[:, None]
    s = np.where(allowed, s, -np.inf)
    s -= s.max(axis=1, keepdims=True)
    e = np.exp(s)
    pmat = e / e.sum(axis=1, keepdims=True)
    z = (pmat @ x_pre).reshape(n_r, n_heads, -1)
    a = np.empty((n_r, n_heads, d), dtype=np.float64)
    for i in range(n_heads):
        a[:, i] = z[:, i] @ wv_h[i // g].T
    return a.reshape(n_r, n_heads * d) @ wo.T


def attention_bwd_rows(x_b, wq, wk, wv, wo, n_heads, n_kv_heads, positions, dy_rows,
                       scale=None):
    """Query path of the attention block's dX (K and V held fixed) at the given global
    positions of one sequence: sum over heads i of dq_i W_Q,i, where dq_i is the gradient
    of head i's query for the upstream rows dy_rows [len(positions), h] at those
    positions.  Uses only associativity, as attention_rows does: with k_j = W_K x_j and
    v_j = W_V x_j, every product over keys runs against the layer input rows x_b [S, h],
    so no K or V of the prefix is formed.  Per head (dA = dY W_O):
      P = causal softmax of scale q k^T;  dP_tj = dA_t . v_j;  o_t = sum_j P_tj v_j;
      dS = P * (dP - dA . o);  dq_t = scale sum_j dS_tj k_j.
    Returns [len(positions), h]."""
    positions = np.asarray(positions, dtype=np.int64)
    d = wq.shape[0] // n_heads
    g = n_heads // n_kv_heads
    sc = default_scale(d, scale)
    t_max = int(positions.max()) + 1
    x_pre = x_b[:t_max]
    n_r, h = positions.shape[0], x_b.shape[1]
    q = (x_b[positions] @ wq.T).reshape(n_r, n_heads, d)
    da = (dy_rows @ wo).reshape(n_r, n_heads, d)
    wk_h = wk.reshape(n_kv_heads, d, h)
    wv_h = wv.reshape(n_kv_heads, d, h)
    u = np.empty((n_r, n_heads, h))
    w = np.empty((n_r, n_heads, h))
    for i in range(n_heads):
        u[:, i] = q[:, i] @ wk_h[i // g]     # score of key j = u . x_j
        w[:, i] = da[:, i] @ wv_h[i // g]    # dP of key j = w . x_j
    pos_rows = np.repeat(positions, n_heads)
    allowed = np.arange(t_max)[None, :] <= pos_rows[:, None]
    s = np.where(allowed, (u.reshape(-1, h) @ x_pre.T) * sc, -np.inf)
    s -= s.max(axis=1, keepdims=True)
    e = np.exp(s)
    pmat = e / e.sum(axis=1, keepdims=True)
    dp = np.where(allowed, w.reshape(-1, h) @ x_pre.T, 0.0)
    z = (pmat @ x_pre).reshape(n_r, n_heads, h)          # o_i = W_V z_i
    o = np.empty((n_r, n_heads, d))
    for i in range(n_heads):
        o[:, i] = z[:, i] @ wv_h[i // g].T
    delta = np.sum(da * o, axis=2).reshape(-1)
    ds = pmat * (dp - delta[:, None])
    y = (ds @ x_pre).reshape(n_r, n_heads, h)            # dq_i = scale W_K y_i
    dq = np.empty((n_r, n_heads, d))
    for i in range(n_heads):
        dq[:, i] = sc * (y[:, i] @ wk_h[i // g].T)
    return dq.reshape(n_r, n_heads * d) @ wq
