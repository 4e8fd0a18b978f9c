"""Thin ctypes binding of libtsp (see include/tsp.h).  Argument marshalling only:
every step of the per-rank forward runs in the library's HIP kernels.

Tensors are torch tensors on the GPU; bf16 operands are ``torch.bfloat16`` (passed
as their bit patterns), accumulators ``torch.float32``.  Shard lists are Python
sequences of tensors (one per shard).  Importing this module loads libtsp.so and
raises ImportError if it has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtsp.so")

TSP_OK = 0
TSP_ERR_HIP = 7
STATUS_NAMES = {0: "TSP_OK", 1: "TSP_ERR_NULL", 2: "TSP_ERR_SHAPE", 3: "TSP_ERR_RANK",
                4: "TSP_ERR_ALIGN", 5: "TSP_ERR_WORKSPACE", 6: "TSP_ERR_UNSUPPORTED",
                7: "TSP_ERR_HIP"}
OP_MLP, OP_ATTN, OP_LAYER, OP_MLP_BWD, OP_ATTN_BWD, OP_ATTN_KV_BWD = 0, 1, 2, 3, 4, 5
LAYOUT_CONTIGUOUS, LAYOUT_ZIGZAG = 0, 1
KERNELS = ("gate_up", "down", "qkv", "attn", "oproj",  # TSP_KERNEL_* order
           "bwd_gate", "bwd_dx", "bwd_dw",
           "abwd_proj", "abwd_fwd", "abwd_kv", "abwd_q", "abwd_dx", "abwd_dw", "abwd_aux")


class TspError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        self.hip_error = lib.tsp_last_hip_error() if status == TSP_ERR_HIP else 0
        msg = f"{where}: {lib.tsp_status_str(status).decode()}"
        if status == TSP_ERR_HIP:
            name = lib.tsp_hip_error_string(self.hip_error).decode()
            msg += f" ({name}, hipError_t {self.hip_error})"
        super().__init__(msg)


class tsp_shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seq", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("ffn", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("degree", ctypes.c_int32),
                ("rank", ctypes.c_int32), ("layout", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("group_steps", ctypes.c_int32)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built; run `python -m paper_2604_26294_amd.build`")
    # torch ships its own HIP runtime (libamdhip64.so, SONAME libamdhip64.so.7).  Loading
    # torch first lets libtsp's libamdhip64.so.7 dependency resolve to that same copy;
    # loaded the other way round, torch maps a second runtime next to the system one and
    # the process ends up with two HIP/HSA runtimes, the second of which sees no device.
    import torch  # noqa: F401
    L = ctypes.CDLL(_LIB_PATH)
    P, VP, SZ, I = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    SH = ctypes.POINTER(tsp_shape)
    PP = ctypes.POINTER(ctypes.c_void_p)
    sig = {
        "tsp_mlp_rank_fwd": [SH, P, PP, PP, PP, P, I, VP, SZ, VP],
        "tsp_mlp_rank_bwd": [SH, P, P, PP, PP, PP, P, I, PP, PP, PP, VP, SZ, VP],
        "tsp_kv_rank_fwd": [SH, P, PP, P, P, VP],
        "tsp_attn_rank_bwd": [SH, P, P, PP, P, P, P, I, PP, P, P, VP, SZ, VP],
        "tsp_attn_kv_rank_bwd": [SH, P, PP, P, P, P, I, PP, VP, SZ, VP],
        "tsp_attn_rank_fwd": [SH, P, PP, P, P, P, I, VP, SZ, VP],
        "tsp_attn_rank_fwd_train": [SH, P, PP, P, P, P, I, P, P, VP, SZ, VP],
        "tsp_attn_rank_bwd_saved": [SH, P, P, PP, P, P, P, P, P, I, PP, P, P, VP, SZ, VP],
        "tsp_layer_rank_fwd": [SH, P, PP, PP, PP, PP, P, P, P, VP, SZ, VP],
        "tsp_layer_rank_fwd_noalloc": [SH, P, PP, PP, PP, PP, P, P, P, VP],
        "tsp_workspace_bytes": [SH, I, ctypes.POINTER(ctypes.c_size_t)],
        "tsp_status_str": [I],
        "tsp_abi_version": [],
        "tsp_last_hip_error": [],
        "tsp_hip_error_string": [I],
        "tsp_profile_enable": [I],
        "tsp_test_set_attn_poll_limit": [I],
        "tsp_profile_read": [I, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)],
    }
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    L.tsp_status_str.restype = ctypes.c_char_p
    L.tsp_hip_error_string.restype = ctypes.c_char_p
    return L


lib = _load()


def make_shape(batch, seq, hidden, ffn, n_heads, n_kv_heads, head_dim, degree, rank,
               layout=0, softmax_scale=0.0, group_steps=0) -> tsp_shape:
    return tsp_shape(batch, seq, hidden, ffn, n_heads, n_kv_heads, head_dim, degree, rank,
                     layout, softmax_scale, group_steps)


def shape_of(wl, rank=None, softmax_scale=0.0, group_steps=0) -> tsp_shape:
    """tsp_shape of a :class:`~paper_2604_26294_amd.workloads.Workload`."""
    return make_shape(wl.batch, wl.seq, wl.hidden, wl.ffn, wl.n_heads, wl.n_kv_heads,
                      wl.head_dim, wl.degree, wl.rank if rank is None else rank, wl.layout,
                      softmax_scale, group_steps)


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _ptrs(ts: Sequence):
    arr = (ctypes.c_void_p * len(ts))(*[_ptr(t) for t in ts])
    return ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)), arr


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _check(st: int, where: str):
    if st != TSP_OK:
        raise TspError(st, where)


def workspace_bytes(shape: tsp_shape, op: int) -> int:
    out = ctypes.c_size_t(0)
    _check(lib.tsp_workspace_bytes(ctypes.byref(shape), op, ctypes.byref(out)),
           "tsp_workspace_bytes")
    return out.value


def _nbytes(ws) -> int:
    return ws.numel() * ws.element_size() if ws is not None else 0


def tsp_mlp_rank_fwd(shape, x_loc, w_gate, w_up, w_down, y_loc, accumulate, ws, stream=None):
    g, _g = _ptrs(w_gate)
    u, _u = _ptrs(w_up)
    d, _d = _ptrs(w_down)
    _check(lib.tsp_mlp_rank_fwd(ctypes.byref(shape), _ptr(x_loc), g, u, d, _ptr(y_loc),
                                int(accumulate), _ptr(ws), _nbytes(ws), _stream(stream)),
           "tsp_mlp_rank_fwd")


def tsp_mlp_rank_bwd(shape, x_loc, dy_loc, w_gate, w_up, w_down, dx_loc, accumulate, dw_gate,
                     dw_up, dw_down, ws, stream=None):
    g, _g = _ptrs(w_gate)
    u, _u = _ptrs(w_up)
    d, _d = _ptrs(w_down)
    dg, _dg = _ptrs(dw_gate)
    du, _du = _ptrs(dw_up)
    dd, _dd = _ptrs(dw_down)
    _check(lib.tsp_mlp_rank_bwd(ctypes.byref(shape), _ptr(x_loc), _ptr(dy_loc), g, u, d,
                                _ptr(dx_loc), int(accumulate), dg, du, dd, _ptr(ws),
                                _nbytes(ws), _stream(stream)), "tsp_mlp_rank_bwd")


def tsp_kv_rank_fwd(shape, x_loc, w_attn, k_buf, v_buf, stream=None):
    a, _a = _ptrs(w_attn)
    _check(lib.tsp_kv_rank_fwd(ctypes.byref(shape), _ptr(x_loc), a, _ptr(k_buf), _ptr(v_buf),
                               _stream(stream)), "tsp_kv_rank_fwd")


def tsp_attn_rank_fwd(shape, x_loc, w_attn, k_buf, v_buf, y_loc, accumulate, ws, stream=None):
    a, _a = _ptrs(w_attn)
    _check(lib.tsp_attn_rank_fwd(ctypes.byref(shape), _ptr(x_loc), a, _ptr(k_buf), _ptr(v_buf),
                                 _ptr(y_loc), int(accumulate), _ptr(ws), _nbytes(ws),
                                 _stream(stream)), "tsp_attn_rank_fwd")


def tsp_attn_rank_bwd(shape, x_loc, dy_loc, w_attn, k_buf, v_buf, dx_loc, accumulate, dw_attn,
                      dk_buf, dv_buf, ws, stream=None):
    a, _a = _ptrs(w_attn)
    dw, _dw = _ptrs(dw_attn)
    _check(lib.tsp_attn_rank_bwd(ctypes.byref(shape), _ptr(x_loc), _ptr(dy_loc), a, _ptr(k_buf),
                                 _ptr(v_buf), _ptr(dx_loc), int(accumulate), dw, _ptr(dk_buf),
                                 _ptr(dv_buf), _ptr(ws), _nbytes(ws), _stream(stream)),
           "tsp_attn_rank_bwd")


def tsp_attn_rank_fwd_train(shape, x_loc, w_attn, k_buf, v_buf, y_loc, accumulate, a_out, lse_out,
                            ws, stream=None):
    a, _a = _ptrs(w_attn)
    _check(lib.tsp_attn_rank_fwd_train(ctypes.byref(shape), _ptr(x_loc), a, _ptr(k_buf),
                                       _ptr(v_buf), _ptr(y_loc), int(accumulate), _ptr(a_out),
                                       _ptr(lse_out), _ptr(ws), _nbytes(ws), _stream(stream)),
           "tsp_attn_rank_fwd_train")


def tsp_attn_rank_bwd_saved(shape, x_loc, dy_loc, w_attn, k_buf, v_buf, a_saved, lse_saved,
                            dx_loc, accumulate, dw_attn, dk_buf, dv_buf, ws, stream=None):
    a, _a = _ptrs(w_attn)
    dw, _dw = _ptrs(dw_attn)
    _check(lib.tsp_attn_rank_bwd_saved(ctypes.byref(shape), _ptr(x_loc), _ptr(dy_loc), a,
                                       _ptr(k_buf), _ptr(v_buf), _ptr(a_saved), _ptr(lse_saved),
                                       _ptr(dx_loc), int(accumulate), dw, _ptr(dk_buf),
                                       _ptr(dv_buf), _ptr(ws), _nbytes(ws), _stream(stream)),
           "tsp_attn_rank_bwd_saved")


def tsp_attn_kv_rank_bwd(shape, x_loc, w_attn, dk_loc, dv_loc, dx_loc, accumulate, dw_attn, ws,
                         stream=None):
    a, _a = _ptrs(w_attn)
    dw, _dw = _ptrs(dw_attn)
    _check(lib.tsp_attn_kv_rank_bwd(ctypes.byref(shape), _ptr(x_loc), a, _ptr(dk_loc),
                                    _ptr(dv_loc), _ptr(dx_loc), int(accumulate), dw, _ptr(ws),
                                    _nbytes(ws), _stream(stream)), "tsp_attn_kv_rank_bwd")


def tsp_layer_rank_fwd(shape, x_loc, w_attn, w_gate, w_up, w_down, k_buf, v_buf, y_loc, ws,
                       stream=None):
    a, _a = _ptrs(w_attn)
    g, _g = _ptrs(w_gate)
    u, _u = _ptrs(w_up)
    d, _d = _ptrs(w_down)
    _check(lib.tsp_layer_rank_fwd(ctypes.byref(shape), _ptr(x_loc), a, g, u, d, _ptr(k_buf),
                                  _ptr(v_buf), _ptr(y_loc), _ptr(ws), _nbytes(ws),
                                  _stream(stream)), "tsp_layer_rank_fwd")


NOALLOC_SCRATCH_BYTES = 128 << 20  # TSP_NOALLOC_SCRATCH_BYTES
GROUP_STEPS_MAX = 8  # TSP_GROUP_STEPS_MAX


def tsp_layer_rank_fwd_noalloc(shape, x_loc, w_attn, w_gate, w_up, w_down, k_buf, v_buf, y_loc,
                               stream=None):
    a, _a = _ptrs(w_attn)
    g, _g = _ptrs(w_gate)
    u, _u = _ptrs(w_up)
    d, _d = _ptrs(w_down)
    _check(lib.tsp_layer_rank_fwd_noalloc(ctypes.byref(shape), _ptr(x_loc), a, g, u, d,
                                          _ptr(k_buf), _ptr(v_buf), _ptr(y_loc),
                                          _stream(stream)), "tsp_layer_rank_fwd_noalloc")


def tsp_test_set_attn_poll_limit(polls: int):
    """Test hook: cap the attention kernels' slot waits at ``polls`` (0: default)."""
    _check(lib.tsp_test_set_attn_poll_limit(int(polls)), "tsp_test_set_attn_poll_limit")


def tsp_profile_enable(enable: bool = True):
    _check(lib.tsp_profile_enable(int(enable)), "tsp_profile_enable")


def tsp_profile_read(kernel: int):
    """(total milliseconds, launches) recorded for kernel class ``kernel``."""
    ms, n = ctypes.c_double(0), ctypes.c_int64(0)
    _check(lib.tsp_profile_read(kernel, ctypes.byref(ms), ctypes.byref(n)), "tsp_profile_read")
    return ms.value, n.value
