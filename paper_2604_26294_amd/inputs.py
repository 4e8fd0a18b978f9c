"""Seeded synthetic inputs shared by the HIP path's tests/bench and the oracle's tests.

This module holds no arithmetic of the method: it draws Gaussian tensors, rounds
them to bfloat16 (round-to-nearest-even), and slices/concatenates the full
(unsharded) weights into the per-shard buffers the C ABI takes.  Both sides of a
parity test start from the same bf16 bit patterns.

Recipe: tensor ``k`` of a workload is drawn with
``numpy.random.default_rng([seed, k]).standard_normal(..., dtype=float32) * std``,
then rounded to bf16.  Tensor ids: x=0, W_Q=1, W_K=2, W_V=3, W_O=4, W1=5, W3=6, W2=7,
and dY=8 (the upstream gradient of the MLP output for the backward).
Activations use ``x_std`` (1.0), weights ``w_std`` (0.02, or 0.015 for the 70B shape).

Weight orientations are the paper's (Algorithms 1 and 2): W_Q [n_h d, h],
W_K and W_V [n_kv d, h], W_O [h, n_h d] (attention output is A W_O^T),
W1 (gate), W3 (up) and W2 (down) all [F, h], with W2 applied untransposed.
"""
from __future__ import annotations

import numpy as np

from .workloads import Workload

TENSOR_ID = {"x": 0, "wq": 1, "wk": 2, "wv": 3, "wo": 4, "w1": 5, "w3": 6, "w2": 7, "dy": 8,
             "dk_own": 9, "dv_own": 10}

_CHUNK_ELEMS = 1 << 24


def round_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even; NaN stays NaN."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    out = ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(bits).astype(np.float64)


def gaussian_bf16(seed: int, tensor_id: int, shape, std: float) -> np.ndarray:
    """Draw N(0, std^2) as bf16 bits, generated in row chunks to bound host memory.

    Drawing consecutive chunks from one Generator yields the same stream as a
    single call, so the values do not depend on the chunk size.
    """
    shape = tuple(int(s) for s in shape)
    n = int(np.prod(shape)) if shape else 1
    rng = np.random.default_rng([seed, tensor_id])
    out = np.empty(n, dtype=np.uint16)
    std32 = np.float32(std)
    for lo in range(0, n, _CHUNK_ELEMS):
        hi = min(n, lo + _CHUNK_ELEMS)
        z = rng.standard_normal(hi - lo, dtype=np.float32)
        if std32 != 1:
            z *= std32
        out[lo:hi] = round_to_bf16_bits(z)
    return out.reshape(shape)


def make_x_full(wl: Workload) -> np.ndarray:
    """Activations of the whole sequence, [B, S, h] bf16 bits."""
    return gaussian_bf16(wl.seed, TENSOR_ID["x"], (wl.batch, wl.seq, wl.hidden), wl.x_std)


def make_dy_full(wl: Workload) -> np.ndarray:
    """Upstream gradient of the MLP output for the whole sequence, [B, S, h] bf16 bits."""
    return gaussian_bf16(wl.seed, TENSOR_ID["dy"], (wl.batch, wl.seq, wl.hidden), wl.x_std)


def make_dkv_own(wl: Workload, p: int) -> tuple:
    """Stand-ins for the reduce-scattered K / V gradients of rank p's own rows,
    [B, S_loc, n_kv, d] bf16 bits each (the input of the K/V projection backward)."""
    shape = (wl.batch, wl.s_loc, wl.n_kv_heads, wl.head_dim)
    return (gaussian_bf16(wl.seed + 7919 * (p + 1), TENSOR_ID["dk_own"], shape, wl.x_std),
            gaussian_bf16(wl.seed + 7919 * (p + 1), TENSOR_ID["dv_own"], shape, wl.x_std))


def make_weights(wl: Workload) -> dict:
    """Full (unsharded) layer weights as bf16 bits, in the paper's orientations."""
    h, d = wl.hidden, wl.head_dim
    shapes = {
        "wq": (wl.n_heads * d, h),
        "wk": (wl.n_kv_heads * d, h),
        "wv": (wl.n_kv_heads * d, h),
        "wo": (h, wl.n_heads * d),
        "w1": (wl.ffn, h),
        "w3": (wl.ffn, h),
        "w2": (wl.ffn, h),
    }
    return {k: gaussian_bf16(wl.seed, TENSOR_ID[k], s, wl.w_std) for k, s in shapes.items()}


def local_chunk(x_full: np.ndarray, p: int, degree: int) -> np.ndarray:
    """Rank p's contiguous sequence chunk x_full[:, p*S/D:(p+1)*S/D]."""
    s_loc = x_full.shape[1] // degree
    return np.ascontiguousarray(x_full[:, p * s_loc:(p + 1) * s_loc])


def attn_shard_packed(w: dict, r: int, degree: int, n_heads: int, n_kv_heads: int,
                      head_dim: int) -> np.ndarray:
    """Packed attention shard r: rows [W_Q^(r); W_K^(r); W_V^(r); W_O^(r)^T], each of length h.

    Shard r owns query heads [r*H_s, (r+1)*H_s) and kv heads [r*K_s, (r+1)*K_s)
    (H_s = n_h/D, K_s = n_kv/D); W_O^(r) is the matching column block of W_O.
    """
    hs = n_heads // degree * head_dim
    ks = n_kv_heads // degree * head_dim
    wo_t_block = w["wo"][:, r * hs:(r + 1) * hs].T
    return np.ascontiguousarray(np.concatenate([
        w["wq"][r * hs:(r + 1) * hs],
        w["wk"][r * ks:(r + 1) * ks],
        w["wv"][r * ks:(r + 1) * ks],
        wo_t_block,
    ], axis=0))


def mlp_shard(w: dict, j: int, degree: int):
    """MLP shard j: rows [j*F/D, (j+1)*F/D) of W1 (gate), W3 (up) and W2 (down)."""
    fs = w["w1"].shape[0] // degree
    sl = slice(j * fs, (j + 1) * fs)
    return (np.ascontiguousarray(w["w1"][sl]), np.ascontiguousarray(w["w3"][sl]),
            np.ascontiguousarray(w["w2"][sl]))
