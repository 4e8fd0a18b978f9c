"""O3: scalar-loop brute force of the unsharded layer, for micro shapes only.

TEST INFRASTRUCTURE ONLY.  Written with explicit Python loops over indices and
``math.exp`` -- no matrix library -- so that it shares no arithmetic with the NumPy
oracle it pins.  Inputs are nested lists or arrays of floats; outputs are nested
lists.  Index conventions (paper, Section 4 and Algorithms 1-2):

  q[t][i*d+e] = sum_c x[t][c] * WQ[i*d+e][c]          (Q = X W_Q^T)
  score(t, j) = scale * sum_e q[t][i*d+e] * k[j][kv*d+e],  kv = i // g, j <= t
  o[t][i*d+e] = sum_{j<=t} softmax_j(score(t, .)) * v[j][kv*d+e]
  attn[t][c]  = sum_m o[t][m] * WO[c][m]                (A W_O^T)
  mlp[t][c]   = sum_f silu(sum_k u[t][k] W1[f][k]) * (sum_k u[t][k] W3[f][k]) * W2[f][c]
"""
from __future__ import annotations

import math


def _silu(z: float) -> float:
    if z < -700.0:
        return 0.0
    return z / (1.0 + math.exp(-z))


def attention_seq(x, wq, wk, wv, wo, n_heads, n_kv_heads, scale=None):
    """One sequence x [S][h] -> attention block output [S][h]."""
    s_len = len(x)
    h = len(x[0])
    d = len(wq) // n_heads
    g = n_heads // n_kv_heads
    sc = 1.0 / math.sqrt(d) if scale is None else scale

    def proj(w, t, row):
        acc = 0.0
        for c in range(h):
            acc += x[t][c] * w[row][c]
        return acc

    q = [[proj(wq, t, m) for m in range(n_heads * d)] for t in range(s_len)]
    k = [[proj(wk, t, m) for m in range(n_kv_heads * d)] for t in range(s_len)]
    v = [[proj(wv, t, m) for m in range(n_kv_heads * d)] for t in range(s_len)]
    o = [[0.0] * (n_heads * d) for _ in range(s_len)]
    for t in range(s_len):
        for i in range(n_heads):
            kv = i // g
            scores = []
            for j in range(t + 1):
                acc = 0.0
                for e in range(d):
                    acc += q[t][i * d + e] * k[j][kv * d + e]
                scores.append(acc * sc)
            mx = max(scores)
            w = [math.exp(sv - mx) for sv in scores]
            tot = sum(w)
            for e in range(d):
                acc = 0.0
                for j in range(t + 1):
                    acc += w[j] / tot * v[j][kv * d + e]
                o[t][i * d + e] = acc
    out = []
    for t in range(s_len):
        row = []
        for c in range(h):
            acc = 0.0
            for m in range(n_heads * d):
                acc += o[t][m] * wo[c][m]
            row.append(acc)
        out.append(row)
    return out


def mlp_seq(u, w1, w3, w2):
    """Gated MLP on rows u [S][h] -> [S][h]."""
    h = len(u[0])
    f = len(w1)
    out = []
    for t in range(len(u)):
        gated = []
        for ff in range(f):
            a = 0.0
            b = 0.0
            for c in range(h):
                a += u[t][c] * w1[ff][c]
                b += u[t][c] * w3[ff][c]
            gated.append(_silu(a) * b)
        row = []
        for c in range(h):
            acc = 0.0
            for ff in range(f):
                acc += gated[ff] * w2[ff][c]
            row.append(acc)
        out.append(row)
    return out


def layer_seq(x, w, n_heads, n_kv_heads, scale=None):
    """u = x + Attn(x), y = u + MLP(u) for one sequence; returns the four blocks."""
    attn = attention_seq(x, w["wq"], w["wk"], w["wv"], w["wo"], n_heads, n_kv_heads, scale)
    u = [[x[t][c] + attn[t][c] for c in range(len(x[0]))] for t in range(len(x))]
    mlp = mlp_seq(u, w["w1"], w["w3"], w["w2"])
    y = [[u[t][c] + mlp[t][c] for c in range(len(x[0]))] for t in range(len(x))]
    return {"attn": attn, "u": u, "mlp": mlp, "y": y}
