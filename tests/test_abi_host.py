"""Host-only checks of the C ABI: the library loads, exports every function that
include/tsp.h declares, and rejects bad arguments before touching the GPU.

These tests never make a call that passes validation with a non-empty problem, so
no kernel is launched and no GPU is needed.  Fake device pointers are plain
aligned integers that the library never dereferences on an error path.
"""
import ctypes
import os
import re

import pytest

from paper_2604_26294_amd import tsp as T
from paper_2604_26294_amd.workloads import ALL, BY_NAME, TINY

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "tsp.h")
FAKE = 0x7F0000000000  # 16-byte aligned stand-in for a device address


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tsp_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert {"tsp_mlp_rank_fwd", "tsp_attn_rank_fwd", "tsp_layer_rank_fwd", "tsp_kv_rank_fwd",
            "tsp_mlp_rank_bwd", "tsp_attn_rank_bwd", "tsp_attn_kv_rank_bwd",
            "tsp_workspace_bytes", "tsp_status_str", "tsp_abi_version"} <= set(names)
    raw = ctypes.CDLL(T._LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


def test_version_and_status_strings():
    assert T.lib.tsp_abi_version() == 2
    for code, name in T.STATUS_NAMES.items():
        assert T.lib.tsp_status_str(code).decode().startswith(name)
    assert T.lib.tsp_status_str(99).decode() == "TSP_ERR_UNKNOWN"


@pytest.mark.parametrize("wl", ALL, ids=lambda w: w.name)
def test_workspace_covers_intermediates(wl):
    sh = T.shape_of(wl)
    m = wl.batch * wl.s_loc
    mlp = T.workspace_bytes(sh, T.OP_MLP)
    attn = T.workspace_bytes(sh, T.OP_ATTN)
    layer = T.workspace_bytes(sh, T.OP_LAYER)
    assert mlp >= m * (wl.ffn // wl.degree) * 2                        # gated product
    assert attn >= 2 * m * (wl.n_heads // wl.degree) * wl.head_dim * 2  # Q and A
    assert layer >= m * wl.hidden * 2 + max(mlp, attn)                 # + bf16(u)
    bwd = T.workspace_bytes(sh, T.OP_MLP_BWD)
    m_pad = (m + 63) // 64 * 64
    fs = wl.ffn // wl.degree
    assert bwd >= 2 * m * fs * 2 + 3 * fs * m_pad * 2  # dG, dU and three transposes
    qd = wl.n_heads // wl.degree * wl.head_dim
    kd = wl.n_kv_heads // wl.degree * wl.head_dim
    abwd = T.workspace_bytes(sh, T.OP_ATTN_BWD)
    akv = T.workspace_bytes(sh, T.OP_ATTN_KV_BWD)
    # Q, A, dA, dQ; lse and delta; A^T and dQ^T
    assert abwd >= 4 * m * qd * 2 + 2 * m * (wl.n_heads // wl.degree) * 4 + 2 * qd * m_pad * 2
    assert akv >= kd * m_pad * 2                        # one transposed K or V gradient
    for v in (mlp, attn, layer, bwd, abwd, akv):
        assert v % 256 == 0
    # the default groups min(D, TSP_GROUP_STEPS_MAX) steps: the gated products, Q and A of
    # a whole group are held at once; one step at a time needs a single step's share
    g = min(wl.degree, T.GROUP_STEPS_MAX)
    assert mlp >= g * m * fs * 2
    assert attn >= 2 * g * m * qd * 2
    one = T.shape_of(wl, group_steps=1)
    assert T.workspace_bytes(one, T.OP_MLP) < m * (fs + 64) * 2 + 256
    assert T.workspace_bytes(one, T.OP_MLP) <= mlp
    assert T.workspace_bytes(one, T.OP_ATTN) <= attn


def _shape(**kw):
    base = dict(batch=1, seq=256, hidden=256, ffn=688, n_heads=4, n_kv_heads=4, head_dim=64,
                degree=2, rank=1, layout=0, softmax_scale=0.0)
    base.update(kw)
    return T.tsp_shape(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(rank=2), 3), (dict(rank=-1), 3),
    (dict(seq=255), 2), (dict(hidden=250), 2), (dict(n_kv_heads=3), 2),
    (dict(n_heads=2, hidden=128, n_kv_heads=2, degree=4, rank=0, ffn=688 * 2), 2),
    (dict(ffn=687), 2), (dict(degree=0, rank=0), 2), (dict(batch=-1), 2),
    (dict(layout=2), 6), (dict(layout=-1), 6), (dict(layout=1, seq=258), 2),
    (dict(layout=1), 0), (dict(head_dim=32, n_heads=8), 6), (dict(ffn=680), 6),
    (dict(group_steps=-1), 2), (dict(group_steps=T.GROUP_STEPS_MAX + 1), 6),
    (dict(group_steps=T.GROUP_STEPS_MAX), 0), (dict(group_steps=1), 0),
    # a 4 GiB per-rank operand (M h bf16 = 2^18 x 8192 x 2 bytes) and just below it
    (dict(hidden=8192, n_heads=64, n_kv_heads=64, head_dim=128, ffn=1024, seq=2 ** 19,
          degree=2, rank=0), 6),
    (dict(hidden=8192, n_heads=64, n_kv_heads=64, head_dim=128, ffn=1024, seq=2 ** 19 - 2,
          degree=2, rank=0), 0),
])
def test_shape_validation(kw, code):
    out = ctypes.c_size_t(0)
    assert T.lib.tsp_workspace_bytes(ctypes.byref(_shape(**kw)), 0, ctypes.byref(out)) == code


def _arr(n, val=FAKE):
    a = (ctypes.c_void_p * n)(*([val] * n))
    return ctypes.cast(a, ctypes.POINTER(ctypes.c_void_p)), a


def test_entry_points_reject_bad_arguments():
    sh = _shape()
    ws_need = T.workspace_bytes(sh, T.OP_LAYER)
    good, _k1 = _arr(2)
    nul, _k2 = _arr(2, 0)
    mis, _k3 = _arr(2, FAKE + 2)
    L = T.lib
    # NULL shape / tensors / shard arrays / shard entries
    assert L.tsp_mlp_rank_fwd(None, FAKE, good, good, good, FAKE, 0, FAKE, ws_need, None) == 1
    assert L.tsp_mlp_rank_fwd(ctypes.byref(sh), None, good, good, good, FAKE, 0, FAKE, ws_need,
                              None) == 1
    assert L.tsp_mlp_rank_fwd(ctypes.byref(sh), FAKE, None, good, good, FAKE, 0, FAKE, ws_need,
                              None) == 1
    assert L.tsp_mlp_rank_fwd(ctypes.byref(sh), FAKE, good, nul, good, FAKE, 0, FAKE, ws_need,
                              None) == 1
    # misaligned pointers
    assert L.tsp_mlp_rank_fwd(ctypes.byref(sh), FAKE + 8, good, good, good, FAKE, 0, FAKE,
                              ws_need, None) == 4
    assert L.tsp_attn_rank_fwd(ctypes.byref(sh), FAKE, mis, FAKE, FAKE, FAKE, 0, FAKE, ws_need,
                               None) == 4
    assert L.tsp_kv_rank_fwd(ctypes.byref(sh), FAKE, good, FAKE + 4, FAKE, None) == 4
    # workspace too small
    assert L.tsp_mlp_rank_fwd(ctypes.byref(sh), FAKE, good, good, good, FAKE, 0, FAKE,
                              T.workspace_bytes(sh, T.OP_MLP) - 1, None) == 5
    assert L.tsp_attn_rank_fwd(ctypes.byref(sh), FAKE, good, FAKE, FAKE, FAKE, 0, FAKE,
                               T.workspace_bytes(sh, T.OP_ATTN) - 1, None) == 5
    assert L.tsp_layer_rank_fwd(ctypes.byref(sh), FAKE, good, good, good, good, FAKE, FAKE, FAKE,
                                FAKE, ws_need - 1, None) == 5
    # bad rank on every entry point
    bad = _shape(rank=5)
    assert L.tsp_layer_rank_fwd(ctypes.byref(bad), FAKE, good, good, good, good, FAKE, FAKE,
                                FAKE, FAKE, ws_need, None) == 3
    assert L.tsp_kv_rank_fwd(ctypes.byref(bad), FAKE, good, FAKE, FAKE, None) == 3


def test_backward_rejects_bad_arguments():
    sh = _shape()
    need = T.workspace_bytes(sh, T.OP_MLP_BWD)
    good, _k1 = _arr(2)
    nul, _k2 = _arr(2, 0)
    mis, _k3 = _arr(2, FAKE + 4)
    L = T.lib
    # argument list that would pass validation; every call below breaks one argument, so
    # none of them reaches a launch
    args = [ctypes.byref(sh), FAKE, FAKE, good, good, good, FAKE, 0, good, good, good, FAKE, need,
            None]
    for pos, val, code in [(1, None, 1), (2, None, 1), (6, None, 1), (8, None, 1), (9, nul, 1),
                           (10, mis, 4), (2, FAKE + 2, 4), (12, need - 1, 5)]:
        a = list(args)
        a[pos] = val
        if pos == 12:
            a[11] = FAKE
        assert L.tsp_mlp_rank_bwd(*a) == code, (pos, code)
    bad = _shape(rank=7)
    a = list(args)
    a[0] = ctypes.byref(bad)
    assert L.tsp_mlp_rank_bwd(*a) == 3


def test_attention_backward_rejects_bad_arguments():
    sh = _shape()
    L = T.lib
    good, _k1 = _arr(2)
    nul, _k2 = _arr(2, 0)
    mis, _k3 = _arr(2, FAKE + 4)
    need = T.workspace_bytes(sh, T.OP_ATTN_BWD)
    # argument lists that would pass validation; every call below breaks one argument
    args = [ctypes.byref(sh), FAKE, FAKE, good, FAKE, FAKE, FAKE, 0, good, FAKE, FAKE, FAKE,
            need, None]
    for pos, val, code in [(1, None, 1), (2, None, 1), (3, nul, 1), (4, None, 1),
                           (5, FAKE + 2, 4), (6, None, 1), (8, mis, 4), (9, None, 1),
                           (10, FAKE + 4, 4), (11, None, 1), (12, need - 1, 5)]:
        a = list(args)
        a[pos] = val
        assert L.tsp_attn_rank_bwd(*a) == code, (pos, code)
    a = list(args)
    a[0] = ctypes.byref(_shape(rank=5))
    assert L.tsp_attn_rank_bwd(*a) == 3
    need = T.workspace_bytes(sh, T.OP_ATTN_KV_BWD)
    args = [ctypes.byref(sh), FAKE, good, FAKE, FAKE, FAKE, 1, good, FAKE, need, None]
    for pos, val, code in [(1, FAKE + 8, 4), (2, nul, 1), (3, None, 1), (4, FAKE + 2, 4),
                           (5, None, 1), (7, mis, 4), (8, None, 1), (9, need - 1, 5)]:
        a = list(args)
        a[pos] = val
        assert L.tsp_attn_kv_rank_bwd(*a) == code, (pos, code)
    a = list(args)
    a[0] = ctypes.byref(_shape(seq=255))
    assert L.tsp_attn_kv_rank_bwd(*a) == 2


def test_empty_batch_is_a_no_op():
    """batch = 0 passes validation and returns before any launch (no GPU involved)."""
    sh = _shape(batch=0)
    good, _k = _arr(2)
    assert T.lib.tsp_mlp_rank_fwd(ctypes.byref(sh), FAKE, good, good, good, FAKE, 0, FAKE, 0,
                                  None) == 0
    assert T.lib.tsp_layer_rank_fwd(ctypes.byref(sh), FAKE, good, good, good, good, FAKE, FAKE,
                                    FAKE, FAKE, 0, None) == 0
    assert T.workspace_bytes(sh, T.OP_LAYER) == 0
    assert T.workspace_bytes(sh, T.OP_ATTN_BWD) == 0
    assert T.lib.tsp_attn_rank_bwd(ctypes.byref(sh), FAKE, FAKE, good, FAKE, FAKE, FAKE, 0, good,
                                   FAKE, FAKE, FAKE, 0, None) == 0
    assert T.lib.tsp_attn_kv_rank_bwd(ctypes.byref(sh), FAKE, good, FAKE, FAKE, FAKE, 0, good,
                                      FAKE, 0, None) == 0


def test_python_binding_raises_named_errors():
    with pytest.raises(T.TspError, match="TSP_ERR_RANK"):
        T.workspace_bytes(_shape(rank=9), T.OP_MLP)
    assert T.workspace_bytes(T.shape_of(TINY), T.OP_MLP) > 0


def test_one_hip_runtime_whatever_the_import_order():
    """Importing the binding before torch must not map a second HIP runtime."""
    import subprocess
    import sys
    code = ("import paper_2604_26294_amd.tsp, torch\n"
            "maps = open('/proc/self/maps').read().splitlines()\n"
            "libs = {l.split()[-1] for l in maps if 'libamdhip64' in l}\n"
            "print(len(libs), sorted(libs))\n")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300,
                         cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    assert out.returncode == 0, out.stderr
    assert out.stdout.split()[0] == "1", out.stdout


def test_noalloc_layer_validates_before_touching_the_gpu():
    """tsp_layer_rank_fwd_noalloc rejects bad arguments, and shapes whose layer
    workspace exceeds its fixed scratch array, before any HIP call; the Python constant
    matches the header's."""
    src = open(HEADER).read()
    m = re.search(r"#define TSP_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", src)
    assert m and int(m.group(1)) << int(m.group(2)) == T.NOALLOC_SCRATCH_BYTES
    L = T.lib
    good, _k1 = _arr(2)
    nul, _k2 = _arr(2, 0)
    sh = _shape()
    args = [ctypes.byref(sh), FAKE, good, good, good, good, FAKE, FAKE, FAKE, None]
    for pos, val, code in [(0, None, 1), (1, None, 1), (2, nul, 1), (5, None, 1),
                           (6, FAKE + 2, 4), (8, None, 1)]:
        a = list(args)
        a[pos] = val
        assert L.tsp_layer_rank_fwd_noalloc(*a) == code, (pos, code)
    a = list(args)
    a[0] = ctypes.byref(_shape(rank=4))
    assert L.tsp_layer_rank_fwd_noalloc(*a) == 3
    big = T.shape_of(BY_NAME["7b-h4096-S65536-D8"])
    assert T.workspace_bytes(big, T.OP_LAYER) > T.NOALLOC_SCRATCH_BYTES
    g8, _k3 = _arr(8)
    assert L.tsp_layer_rank_fwd_noalloc(ctypes.byref(big), FAKE, g8, g8, g8, g8, FAKE, FAKE,
                                        FAKE, None) == 5
    empty = _shape(batch=0)
    assert L.tsp_layer_rank_fwd_noalloc(ctypes.byref(empty), FAKE, good, good, good, good, FAKE,
                                        FAKE, FAKE, None) == 0
    fits = T.shape_of(BY_NAME["7b-h4096-S8192-D8"])
    assert T.workspace_bytes(fits, T.OP_LAYER) <= T.NOALLOC_SCRATCH_BYTES


def test_training_pair_rejects_bad_arguments():
    """tsp_attn_rank_fwd_train and tsp_attn_rank_bwd_saved validate every argument,
    including the kept A / log-sum-exp buffers, before anything is enqueued."""
    sh = _shape()
    L = T.lib
    good, _k1 = _arr(2)
    nul, _k2 = _arr(2, 0)
    fwd_need = T.workspace_bytes(sh, T.OP_ATTN)
    fwd = [ctypes.byref(sh), FAKE, good, FAKE, FAKE, FAKE, 0, FAKE, FAKE, FAKE, fwd_need, None]
    for pos, val, code in [(1, None, 1), (2, nul, 1), (5, None, 1), (7, None, 1),
                           (7, FAKE + 2, 4), (8, None, 1), (8, FAKE + 4, 4), (9, None, 1),
                           (10, fwd_need - 1, 5)]:
        a = list(fwd)
        a[pos] = val
        assert L.tsp_attn_rank_fwd_train(*a) == code, ("fwd", pos, code)
    bwd_need = T.workspace_bytes(sh, T.OP_ATTN_BWD)
    bwd = [ctypes.byref(sh), FAKE, FAKE, good, FAKE, FAKE, FAKE, FAKE, FAKE, 0, good, FAKE, FAKE,
           FAKE, bwd_need, None]
    for pos, val, code in [(1, None, 1), (2, None, 1), (6, None, 1), (6, FAKE + 8, 4),
                           (7, None, 1), (7, FAKE + 4, 4), (8, None, 1), (10, nul, 1),
                           (13, None, 1), (14, bwd_need - 1, 5)]:
        a = list(bwd)
        a[pos] = val
        assert L.tsp_attn_rank_bwd_saved(*a) == code, ("bwd", pos, code)
    bad = _shape(rank=4)
    a = list(bwd)
    a[0] = ctypes.byref(bad)
    assert L.tsp_attn_rank_bwd_saved(*a) == 3


def test_attention_poll_limit_hook_validates():
    """The attention forward's poll-limit test hook takes 0 (the default) and positive
    caps, and rejects negative ones through the C ABI (no GPU work)."""
    from paper_2604_26294_amd import tsp as T
    assert T.STATUS_NAMES[T.lib.tsp_test_set_attn_poll_limit(-1)] == "TSP_ERR_SHAPE"
    assert T.lib.tsp_test_set_attn_poll_limit(3) == T.TSP_OK
    assert T.lib.tsp_test_set_attn_poll_limit(0) == T.TSP_OK
