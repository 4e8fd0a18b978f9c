"""GPU parity of the ring-MLP backward (tsp_mlp_rank_bwd) against the fp64 oracle,
through the C ABI: dX and every shard's weight-gradient contribution, per tensor at the
tolerance of the forward (bf16 operands, fp32 accumulation)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import tsp_oracle as O  # noqa: E402
from paper_2604_26294_amd import inputs as I  # noqa: E402
from paper_2604_26294_amd.harness import RankProblem, local_rows, to_device_bf16  # noqa: E402
from paper_2604_26294_amd.workloads import TINY  # noqa: E402
from tests.gpu_common import MID_GQA64, MID_MHA128, ODD3, SINGLE, assert_close, f64  # noqa: E402

# Ragged tails: M = B S_loc = 384 / 640 / 320 against 128-row tiles, F/D = 344 / 1384 /
# 1024 against 128-column tiles and the 64-wide contraction step.
CASES = [(TINY, 1), (MID_GQA64, 3), (MID_MHA128, 0), (SINGLE, 0), (MID_GQA64.with_layout(1), 2),
         (ODD3, 1)]  # odd D: the weight gradients of the last ring step run alone
_cache = {}


def _inputs(wl):
    if wl.name not in _cache:
        _cache[wl.name] = (I.make_x_full(wl), I.make_weights(wl), I.make_dy_full(wl))
    return _cache[wl.name]


def _run(wl, p, accumulate_twice=False):
    x_bits, w_bits, dy_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    dy = to_device_bf16(local_rows(dy_bits, wl, p))
    out = prob.mlp_bwd(dy)
    if accumulate_twice:
        out = prob.mlp_bwd(dy, accumulate=True)
    torch.cuda.synchronize()
    dx, dwg, dwu, dwd = out
    return (dx.double().cpu().numpy(), [t.double().cpu().numpy() for t in dwg],
            [t.double().cpu().numpy() for t in dwu], [t.double().cpu().numpy() for t in dwd])


def _reference(wl, p):
    x_bits, w_bits, dy_bits = _inputs(wl)
    D = wl.degree
    mlp = [I.mlp_shard({k: f64(v) for k, v in w_bits.items()}, j, D) for j in range(D)]
    x = f64(local_rows(x_bits, wl, p))
    dy = f64(local_rows(dy_bits, wl, p))
    return O.mlp_rank_bwd(x, [m[0] for m in mlp], [m[1] for m in mlp], [m[2] for m in mlp],
                          dy, p)


@pytest.mark.parametrize("wl,p", CASES, ids=[f"{w.name}-{w.layout_name}-r{p}" for w, p in CASES])
def test_mlp_backward_parity(wl, p):
    print(f"[mlp bwd] {wl.name} {wl.layout_name} rank {p}", flush=True)
    got = _run(wl, p)
    ref = _reference(wl, p)
    assert_close(got[0], ref[0], f"{wl.name} r{p} dX")
    for name, g, r in zip(("dW_gate", "dW_up", "dW_down"), got[1:], ref[1:]):
        for j in range(wl.degree):
            assert_close(g[j], r[j], f"{wl.name} r{p} {name}[{j}]")


def test_mlp_backward_accumulates():
    """A second call with accumulate != 0 adds the same gradients again (up to the fp32
    summation order of the running sums)."""
    wl, p = MID_GQA64, 1
    once = _run(wl, p)
    twice = _run(wl, p, accumulate_twice=True)
    assert np.allclose(twice[0], 2 * once[0], rtol=1e-5, atol=1e-5)
    for a, b in zip(once[1:], twice[1:]):
        for j in range(wl.degree):
            assert np.allclose(b[j], 2 * a[j], rtol=1e-5, atol=1e-5)
