"""Device-side setup of one rank's TSP problem from the seeded inputs.

Uploads the bf16 bit patterns drawn by :mod:`paper_2604_26294_amd.inputs`, builds
the per-shard device buffers the C ABI takes, and allocates outputs, the K/V
buffer and the workspace.  No arithmetic of the method lives here: everything is
computed by libtsp through :mod:`paper_2604_26294_amd.tsp`.
"""
from __future__ import annotations

import numpy as np
import torch

from . import inputs as I
from . import tsp as T
from .workloads import Workload


def to_device_bf16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16))
    return t.view(torch.bfloat16).to(device)


def local_positions(wl: Workload, p: int) -> np.ndarray:
    """Global sequence positions of rank p's local rows: a contiguous chunk, or for the
    zigzag layout chunk p then chunk 2D-1-p of S/(2D) tokens (the C ABI's mapping)."""
    if wl.layout == 0:
        return np.arange(p * wl.s_loc, (p + 1) * wl.s_loc)
    s_c = wl.s_loc // 2
    first = np.arange(p * s_c, (p + 1) * s_c)
    second = np.arange((2 * wl.degree - 1 - p) * s_c, (2 * wl.degree - p) * s_c)
    return np.concatenate([first, second])


def local_rows(x_full: np.ndarray, wl: Workload, p: int) -> np.ndarray:
    """Rank p's local input rows [B, S_loc, h] of the full-sequence input."""
    return np.ascontiguousarray(x_full[:, local_positions(wl, p)])


def bf16_tensor_to_f64(t: torch.Tensor) -> np.ndarray:
    bits = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return I.bf16_bits_to_f64(bits)


class RankProblem:
    """All device buffers of rank ``p`` of workload ``wl``.

    ``x_full`` / ``w`` are the bf16 bit patterns of the whole-sequence input and the
    full weights (see :func:`inputs.make_x_full`, :func:`inputs.make_weights`).
    ``softmax_scale`` is passed to every attention call (0 = the default 1/sqrt(d)),
    ``group_steps`` to every forward call (0 = the library's default grouping).
    """

    def __init__(self, wl: Workload, x_full: np.ndarray, w: dict, p: int | None = None,
                 device="cuda", kv_fill: float | None = 0.0, softmax_scale: float = 0.0,
                 group_steps: int = 0):
        self.wl = wl
        self.p = wl.rank if p is None else p
        self.device = device
        D = wl.degree
        # softmax_scale <= 0 selects 1/sqrt(head_dim) (tsp_shape)
        self.shape = T.shape_of(wl, self.p, softmax_scale, group_steps)
        # ranks whose K/V rows this rank's queries can see: the earlier ones for
        # contiguous chunks, every one for a zigzag shard
        self.kv_ranks = list(range(self.p)) if wl.layout == 0 else \
            [q for q in range(D) if q != self.p]
        self.x_chunks = {q: to_device_bf16(local_rows(x_full, wl, q), device)
                         for q in self.kv_ranks + [self.p]}
        self.x_loc = self.x_chunks[self.p]
        self.attn = [to_device_bf16(I.attn_shard_packed(w, r, D, wl.n_heads, wl.n_kv_heads,
                                                        wl.head_dim), device)
                     for r in range(D)]
        mlp = [I.mlp_shard(w, j, D) for j in range(D)]
        self.w1 = [to_device_bf16(m[0], device) for m in mlp]
        self.w3 = [to_device_bf16(m[1], device) for m in mlp]
        self.w2 = [to_device_bf16(m[2], device) for m in mlp]
        kv_shape = (wl.batch, wl.seq, wl.n_kv_heads, wl.head_dim)
        self.k_buf = torch.empty(kv_shape, dtype=torch.bfloat16, device=device)
        self.v_buf = torch.empty(kv_shape, dtype=torch.bfloat16, device=device)
        if kv_fill is not None:
            self.k_buf.fill_(kv_fill)
            self.v_buf.fill_(kv_fill)
        self.y = torch.zeros((wl.batch, wl.s_loc, wl.hidden), dtype=torch.float32, device=device)
        nbytes = max(T.workspace_bytes(self.shape, op) for op in (T.OP_MLP, T.OP_ATTN, T.OP_LAYER))
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)

    def prefill_kv(self, include_self=False):
        """The modelled all-gather: the other ranks write their K/V rows of every shard
        (and this rank its own, for a backward run without the forward before it)."""
        for q in self.kv_ranks + ([self.p] if include_self else []):
            T.tsp_kv_rank_fwd(T.shape_of(self.wl, q), self.x_chunks[q], self.attn, self.k_buf,
                              self.v_buf)

    def _attn_grads(self):
        if not hasattr(self, "adx"):
            wl, dev = self.wl, self.device
            rows = (2 * wl.n_heads // wl.degree + 2 * wl.n_kv_heads // wl.degree) * wl.head_dim
            self.adx = torch.zeros((wl.batch, wl.s_loc, wl.hidden), dtype=torch.float32,
                                   device=dev)
            self.adw = [torch.zeros((rows, wl.hidden), dtype=torch.float32, device=dev)
                        for _ in range(wl.degree)]
            kv_shape = (wl.batch, wl.seq, wl.n_kv_heads, wl.head_dim)
            self.dk_buf = torch.zeros(kv_shape, dtype=torch.float32, device=dev)
            self.dv_buf = torch.zeros(kv_shape, dtype=torch.float32, device=dev)
            nbytes = max(T.workspace_bytes(self.shape, op)
                         for op in (T.OP_ATTN_BWD, T.OP_ATTN_KV_BWD))
            self.ws_abwd = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)

    def attn_bwd(self, dy_loc, accumulate=False):
        """First stage of the attention backward for the bf16 gradient dy_loc [B, S_loc, h]
        of the block output (the K/V buffers must hold the gathered K/V).  Returns (dx,
        dw_attn list, dk_buf, dv_buf), fp32 device tensors."""
        self._attn_grads()
        T.tsp_attn_rank_bwd(self.shape, self.x_loc, dy_loc, self.attn, self.k_buf, self.v_buf,
                            self.adx, accumulate, self.adw, self.dk_buf, self.dv_buf, self.ws_abwd)
        return self.adx, self.adw, self.dk_buf, self.dv_buf

    def attn_fwd_train(self, accumulate=False):
        """The attention block forward that keeps A [B, S_loc, n_h, d] bf16 and the
        base-2 log-sum-exp [B, n_h, S_loc] fp32 for attn_bwd_saved.  Returns (y, a, lse)."""
        wl = self.wl
        if not hasattr(self, "a_saved"):
            self.a_saved = torch.empty((wl.batch, wl.s_loc, wl.n_heads, wl.head_dim),
                                       dtype=torch.bfloat16, device=self.device)
            self.lse_saved = torch.empty((wl.batch, wl.n_heads, wl.s_loc), dtype=torch.float32,
                                         device=self.device)
        T.tsp_attn_rank_fwd_train(self.shape, self.x_loc, self.attn, self.k_buf, self.v_buf,
                                  self.y, accumulate, self.a_saved, self.lse_saved, self.ws)
        return self.y, self.a_saved, self.lse_saved

    def attn_bwd_saved(self, dy_loc, accumulate=False):
        """attn_bwd with A and the log-sum-exp of the last attn_fwd_train call."""
        self._attn_grads()
        T.tsp_attn_rank_bwd_saved(self.shape, self.x_loc, dy_loc, self.attn, self.k_buf,
                                  self.v_buf, self.a_saved, self.lse_saved, self.adx, accumulate,
                                  self.adw, self.dk_buf, self.dv_buf, self.ws_abwd)
        return self.adx, self.adw, self.dk_buf, self.dv_buf

    def attn_kv_bwd(self, dk_loc, dv_loc, accumulate=True):
        """Second stage: the K/V projection backward for the bf16 reduce-scattered
        gradients of this rank's rows [B, S_loc, n_kv, d].  Returns (dx, dw_attn list)."""
        self._attn_grads()
        T.tsp_attn_kv_rank_bwd(self.shape, self.x_loc, self.attn, dk_loc, dv_loc, self.adx,
                               accumulate, self.adw, self.ws_abwd)
        return self.adx, self.adw

    def mlp(self, x=None, accumulate=False):
        T.tsp_mlp_rank_fwd(self.shape, self.x_loc if x is None else x, self.w1, self.w3,
                           self.w2, self.y, accumulate, self.ws)
        return self.y

    def attn_fwd(self, accumulate=False):
        T.tsp_attn_rank_fwd(self.shape, self.x_loc, self.attn, self.k_buf, self.v_buf, self.y,
                            accumulate, self.ws)
        return self.y

    def mlp_bwd(self, dy_loc, accumulate=False):
        """MLP backward of this rank for the bf16 upstream gradient dy_loc [B, S_loc, h];
        returns (dx, dw_gate, dw_up, dw_down), fp32 device tensors (lists per shard)."""
        wl = self.wl
        if not hasattr(self, "dx"):
            fs = wl.ffn // wl.degree
            dev = self.device
            self.dx = torch.zeros((wl.batch, wl.s_loc, wl.hidden), dtype=torch.float32, device=dev)
            self.dw = [[torch.zeros((fs, wl.hidden), dtype=torch.float32, device=dev)
                        for _ in range(wl.degree)] for _ in range(3)]
            nbytes = T.workspace_bytes(self.shape, T.OP_MLP_BWD)
            self.ws_bwd = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
        T.tsp_mlp_rank_bwd(self.shape, self.x_loc, dy_loc, self.w1, self.w3, self.w2, self.dx,
                           accumulate, self.dw[0], self.dw[1], self.dw[2], self.ws_bwd)
        return self.dx, self.dw[0], self.dw[1], self.dw[2]

    def layer(self):
        T.tsp_layer_rank_fwd(self.shape, self.x_loc, self.attn, self.w1, self.w3, self.w2,
                             self.k_buf, self.v_buf, self.y, self.ws)
        return self.y
