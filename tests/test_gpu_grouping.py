"""GPU parity of the forward under every shard-step grouping (tsp_shape.group_steps):
one step per launch, groups that divide D, groups that leave a smaller last group, and
more shards than one group holds.  Whatever the grouping, the result is the sum of
Algorithm 1's and Algorithm 2's shard terms in schedule order, so each run is checked
element by element against the fp64 oracle at the usual tolerance, and the groupings
against each other (they differ only in fp32 summation order)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2604_26294_amd.harness import RankProblem  # noqa: E402
from tests.gpu_common import (DEG16, MID_GQA64, MID_MHA128, ODD3, SUBL, assert_close,  # noqa: E402
                              gen, oracle_blocks)

# (workload, rank, group_steps values); 0 is the library default, min(D, 8)
CASES = [(MID_GQA64, 3, (1, 2, 3)), (MID_GQA64.with_layout(1), 1, (1, 3)),
         (ODD3, 2, (1, 2)), (ODD3.with_layout(1), 0, (2,)), (MID_MHA128, 1, (1,)),
         (DEG16, 13, (0, 5)), (DEG16.with_layout(1), 6, (0,))]
_IDS = [f"{w.name}-{w.layout_name}-r{p}" for w, p, _ in CASES]
_cache = {}


def _inputs(wl):
    if wl.name not in _cache:
        _cache[wl.name] = gen(wl)
    return _cache[wl.name]


@pytest.mark.parametrize("wl,p,groups", CASES, ids=_IDS)
@pytest.mark.parametrize("block", ["mlp", "attn", "layer"])
def test_grouping_parity(wl, p, groups, block):
    x_bits, w_bits = _inputs(wl)
    ref = oracle_blocks(wl, x_bits, w_bits, p, blocks=(block,))[block]
    outs = {}
    for g in groups:
        print(f"[grouping] {wl.name} {wl.layout_name} rank {p} {block} group_steps={g}",
              flush=True)
        prob = RankProblem(wl, x_bits, w_bits, p, group_steps=g)
        prob.prefill_kv()
        y = {"mlp": prob.mlp, "attn": prob.attn_fwd, "layer": prob.layer}[block]()
        torch.cuda.synchronize()
        outs[g] = y.double().cpu().numpy()
        assert_close(outs[g], ref, f"{wl.name} r{p} {block} G={g}")
    # every grouping against the default one (all steps together where D <= 8)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv()
    base = {"mlp": prob.mlp, "attn": prob.attn_fwd, "layer": prob.layer}[block]()
    torch.cuda.synchronize()
    base = base.double().cpu().numpy()
    scale = np.max(np.abs(base))
    for g, y in outs.items():
        assert np.max(np.abs(y - base)) <= 1e-2 * scale, f"G={g} vs default"


@pytest.mark.parametrize("wl,p", [(SUBL, 2), (SUBL.with_layout(1), 1)],
                         ids=["paired-contiguous-r2", "paired-zigzag-r1"])
@pytest.mark.parametrize("block", ["attn", "layer"])
def test_attention_with_paired_query_tiles(wl, p, block):
    """A group's attention with two query tiles per workgroup (the i-th most and the i-th
    fewest keys), as the launch plan takes it for shapes with many work items per shard;
    launches over part of a group's shards (heads' columns inside group-wide Q and A rows)
    are covered at full size (7B S=65536, 70B: 4 of 8 shards per launch; 13B: 1 of 4)."""
    print(f"[grouping] {wl.name} {wl.layout_name} rank {p} {block}", flush=True)
    x_bits, w_bits = _inputs(wl)
    prob = RankProblem(wl, x_bits, w_bits, p)
    prob.prefill_kv()
    y = {"attn": prob.attn_fwd, "layer": prob.layer}[block]()
    torch.cuda.synchronize()
    ref = oracle_blocks(wl, x_bits, w_bits, p, blocks=(block,))[block]
    assert_close(y.double().cpu().numpy(), ref, f"{wl.name} r{p} {block}")
