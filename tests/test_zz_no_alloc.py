"""The allocation-free layer entry point, tsp_layer_rank_fwd_noalloc, against the
workspace entry point tsp_layer_rank_fwd, through the C ABI.  Two calls in a row share
the device's fixed scratch array, the second with a smaller problem than the first;
each must equal the workspace call on the same inputs bit for bit (same kernels, same
launch shapes, fixed reduction orders) and meet the parity tolerance against the fp64
oracle."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2604_26294_amd import tsp as T  # noqa: E402
from paper_2604_26294_amd.harness import RankProblem  # noqa: E402
from paper_2604_26294_amd.workloads import TINY  # noqa: E402
from tests.gpu_common import MID_MHA128, assert_close, gen, oracle_blocks  # noqa: E402


def _noalloc(prob):
    y = torch.full_like(prob.y, float("nan"))
    T.tsp_layer_rank_fwd_noalloc(prob.shape, prob.x_loc, prob.attn, prob.w1, prob.w3, prob.w2,
                                 prob.k_buf, prob.v_buf, y)
    return y


def test_noalloc_layer_matches_workspace_call_twice_in_a_row():
    cases = [(MID_MHA128, 1), (TINY, 1)]   # larger problem first, then a smaller one
    probs, refs = [], []
    for wl, p in cases:
        print(f"[noalloc] {wl.name} rank {p}", flush=True)
        prob = RankProblem(wl, *gen(wl), p)
        prob.prefill_kv()
        assert T.workspace_bytes(prob.shape, T.OP_LAYER) <= T.NOALLOC_SCRATCH_BYTES
        refs.append(prob.layer().clone())
        probs.append(prob)
    torch.cuda.synchronize()
    outs = [_noalloc(prob) for prob in probs]
    torch.cuda.synchronize()
    for (wl, p), prob, ref, got in zip(cases, probs, refs, outs):
        assert torch.equal(got, ref), f"{wl.name} r{p}: differs from the workspace call"
        want = oracle_blocks(wl, *gen(wl), p, blocks=("layer",))["layer"]
        assert_close(got.double().cpu().numpy(), want, f"{wl.name} r{p} noalloc layer")
