"""The peaky-logit stress input of the GPU parity tests does what it is there for,
checked on the CPU from the same bf16 inputs in fp64."""
import numpy as np

from tests.gpu_common import MID_GQA64, MID_MHA128, RISING_ROWS, f64, stress_inputs


def test_peaky_logits_move_the_reference():
    """The stress input really exercises the rescale: walking each row's visible keys in
    64-key blocks, a reference that moves only when a block's largest logit (log2 units)
    exceeds it by more than 8 moves again after the first block in at least a third of
    the rows of the split-key case (computed from the bf16 inputs in fp64)."""
    wl, p = MID_MHA128, 1
    x_bits, w_bits = stress_inputs(wl, "peaky")
    x = f64(x_bits)
    wq, wk = f64(w_bits["wq"]), f64(w_bits["wk"])
    d = wl.head_dim
    q = x[0, p * wl.s_loc:, :] @ wq[:d].T
    k = x[0] @ wk[:d].T
    s = (q @ k.T) / np.sqrt(d) * np.log2(np.e)
    pos = p * wl.s_loc + np.arange(wl.s_loc)
    s = np.where(np.arange(k.shape[0])[None, :] <= pos[:, None], s, -np.inf)
    ref = s[:, :64].max(axis=1)
    moved = np.zeros(s.shape[0], dtype=bool)
    for t in range(64, s.shape[1], 64):
        m = s[:, t:t + 64].max(axis=1)
        mv = m > ref + 8.0
        moved |= mv
        ref = np.where(mv, m, ref)
    assert moved.mean() > 1 / 3


def test_rising_logits_pass_the_sum_bound():
    """The rising stress input does what it is there for: against the largest logit of a
    row's first 128 keys, the probabilities 2^(s - m) of some later 64-key block of the
    row sum to 2^40 or more in at least a third of the rows (every head of the rank, from
    the bf16 inputs in fp64), while the peaky input alone leaves that bound unreached."""
    wl, p = MID_GQA64, 3
    d, g = wl.head_dim, wl.n_heads // wl.n_kv_heads
    frac = {}
    for kind in ("peaky", "rising"):
        x_bits, w_bits = stress_inputs(wl, kind)
        x, wq, wk = f64(x_bits), f64(w_bits["wq"]), f64(w_bits["wk"])
        rows = passed = 0
        for b in range(wl.batch):
            for hd in range(wl.n_heads):
                q = x[b, p * wl.s_loc:] @ wq[hd * d:(hd + 1) * d].T
                k = x[b] @ wk[hd // g * d:(hd // g + 1) * d].T
                s = (q @ k.T) / np.sqrt(d) * np.log2(np.e)
                pos = p * wl.s_loc + np.arange(wl.s_loc)
                s = np.where(np.arange(k.shape[0])[None, :] <= pos[:, None], s, -np.inf)
                m = s[:, :RISING_ROWS].max(axis=1)
                over = np.zeros(s.shape[0], dtype=bool)
                for t in range(RISING_ROWS, s.shape[1], 64):
                    with np.errstate(over="ignore"):
                        over |= ~(np.exp2(s[:, t:t + 64] - m[:, None]).sum(axis=1) < 2.0 ** 40)
                rows += s.shape[0]
                passed += int(over.sum())
        frac[kind] = passed / rows
    assert frac["rising"] > 1 / 3
    assert frac["peaky"] < frac["rising"]
