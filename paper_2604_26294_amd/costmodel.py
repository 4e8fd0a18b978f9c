"""Analytic cost model of Section 4: per-layer communication volume, per-GPU memory
and per-device FLOPs of DP, TP, SP, TP+SP and TSP, and the TSP-versus-TP break-even.

Pure host arithmetic, no GPU.  Notation follows the paper's Section 4 notation table:
B micro-batch, S sequence, h hidden, n_h / n_kv heads, d head dim, g = n_h / n_kv,
F the MLP expansion factor (the gated MLP has width F h), L layers, D the parallel
degree (T x Sigma on a 2D mesh), beta_P / beta_g bytes per parameter / gradient
element, n_o optimizer states of beta_o bytes each.

Communication is bytes moved per layer per device; memory is bytes per GPU for the
whole model; FLOPs are leading-order forward FLOPs of one layer per device.  Three
training phases are modelled: ``"fwd"``, ``"fwd+bwd"`` (no recomputation) and
``"fwd+bwd+recomp"`` (full recomputation repeats the forward communication).

The one place where the section gives two figures for the same quantity is TSP's
gradient reduction: its training equations charge the tight reduce-to-owner volume
P_L beta_g (D-1)/D without recomputation but 2 P_L beta_g (D-1)/D with it, while the
TSP-versus-SP comparison upper-bounds both by the all-reduce volume.  ``tsp_grad``
selects ``"printed"`` (the training equations as given, the default),
``"reduce"`` (tight in both phases) or ``"allreduce"`` (the upper bound in both).

Run ``python -m paper_2604_26294_amd.costmodel`` for the three summary tables of a
configuration (defaults: the 7B reference model of Appendix C).
"""
from __future__ import annotations

import argparse
from dataclasses import dataclass

STRATEGIES = ("DP", "TP", "SP", "TP+SP", "TSP")
PHASES = ("fwd", "fwd+bwd", "fwd+bwd+recomp")
RECOMPUTE = ("full", "sel", "none")


@dataclass(frozen=True)
class ModelConfig:
    """Model dimensions and storage precisions (Section 4 notation table)."""
    hidden: int                  # h
    layers: int                  # L
    n_heads: int                 # n_h
    n_kv_heads: int              # n_kv
    head_dim: int                # d
    ffn_factor: float            # F (gated MLP width F h)
    beta_p: float = 2.0          # bytes per parameter / activation element
    beta_g: float = 2.0          # bytes per gradient element
    n_opt: int = 3               # n_o optimizer states per parameter
    beta_o: float = 4.0          # bytes per optimizer state element

    @property
    def g(self) -> float:
        return self.n_heads / self.n_kv_heads


def reference_7b() -> ModelConfig:
    """The 7B reference model of Appendix C: h 4096, 32 layers, 32 MHA heads of 128,
    F = 4, bf16 weights and gradients, mixed-precision AdamW (3 fp32 states)."""
    return ModelConfig(hidden=4096, layers=32, n_heads=32, n_kv_heads=32, head_dim=128,
                       ffn_factor=4.0, beta_p=2.0, beta_g=2.0, n_opt=3, beta_o=4.0)


def from_workload(wl, layers: int = 32) -> ModelConfig:
    """ModelConfig of a :class:`~paper_2604_26294_amd.workloads.Workload` layer shape."""
    return ModelConfig(hidden=wl.hidden, layers=layers, n_heads=wl.n_heads,
                       n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                       ffn_factor=wl.ffn / wl.hidden)


# ---- collective volumes (Section 4, "Communication volume") ------------------------

def allreduce_bytes(n: float, d: int) -> float:
    """Ring all-reduce of an n-byte message over d devices: 2 n (d-1)/d per device."""
    return 2.0 * n * (d - 1) / d


def allgather_bytes(n: float, d: int) -> float:
    """Ring all-gather of an n-byte total: n (d-1)/d per device."""
    return n * (d - 1) / d


def broadcast_bytes(n: float, d: int) -> float:
    """Broadcast of an n-byte message: n (independent of d)."""
    return float(n)


# ---- parameters, memory ------------------------------------------------------------

def params_attn(c: ModelConfig) -> float:
    """P_attn = 2 (1 + 1/g) h^2: Q and O are h x h, K and V are h x h/g."""
    return 2.0 * (1.0 + 1.0 / c.g) * c.hidden ** 2


def params_mlp(c: ModelConfig) -> float:
    """P_mlp = 3 F h^2: gate, up and down projections of the gated MLP."""
    return 3.0 * c.ffn_factor * c.hidden ** 2


def params_layer(c: ModelConfig) -> float:
    """P_L = P_attn + P_mlp = (2 (1 + 1/g) + 3 F) h^2."""
    return params_attn(c) + params_mlp(c)


def params_total(c: ModelConfig) -> float:
    """L P_L (embeddings and norms excluded, as in Appendix C)."""
    return c.layers * params_layer(c)


def activation_bytes(c: ModelConfig, b: int, s: int, recompute: str = "sel") -> float:
    """Unsharded activation memory M_a of the whole model (Section 4, "Activation
    memory"): full recomputation keeps only each layer's input, L B S h beta_P;
    selective keeps everything but the attention matrices, L B S h (16 beta_P + 2);
    none adds the attention matrices, L B S h (2 beta_P + 1) n_h S / h."""
    base = c.layers * b * s * c.hidden
    if recompute == "full":
        return base * c.beta_p
    if recompute == "sel":
        return base * (16.0 * c.beta_p + 2.0)
    if recompute == "none":
        return base * (16.0 * c.beta_p + 2.0 + (2.0 * c.beta_p + 1.0) * c.n_heads * s / c.hidden)
    raise ValueError(f"recompute must be one of {RECOMPUTE}, not {recompute!r}")


def _mesh(strategy: str, d: int, t: int | None, sigma: int | None) -> tuple[int, int]:
    """(weight-sharding factor, activation-sharding factor) of a strategy."""
    if strategy == "DP":
        return 1, 1
    if strategy == "TP":
        return d, 1
    if strategy == "SP":
        return 1, d
    if strategy == "TSP":
        return d, d
    if strategy == "TP+SP":
        if t is None or sigma is None or t * sigma != d:
            raise ValueError("TP+SP needs T and Sigma with T * Sigma = D")
        return t, sigma
    raise ValueError(f"strategy must be one of {STRATEGIES}, not {strategy!r}")


def memory_bytes(strategy: str, c: ModelConfig, b: int, s: int, d: int,
                 recompute: str = "sel", t: int | None = None,
                 sigma: int | None = None) -> dict[str, float]:
    """Per-GPU memory by category (table tab:mem_summary): parameters, gradients and
    optimizer states divide by the weight-sharding factor (D for TP and TSP, T for
    TP+SP), activations by the sequence-sharding factor (D for SP and TSP, Sigma for
    TP+SP).  Temporary communication buffers are not counted, as in the table."""
    wdiv, adiv = _mesh(strategy, d, t, sigma)
    lp = params_total(c)
    out = {"params": lp * c.beta_p / wdiv,
           "grads": lp * c.beta_g / wdiv,
           "optim": lp * c.n_opt * c.beta_o / wdiv,
           "acts": activation_bytes(c, b, s, recompute) / adiv}
    out["total"] = out["params"] + out["grads"] + out["optim"] + out["acts"]
    return out


# ---- communication -----------------------------------------------------------------

def comm_terms_fwd(strategy: str, c: ModelConfig, b: int, s: int, d: int,
                   t: int | None = None, sigma: int | None = None) -> tuple[float, float]:
    """(activation term, weight term) of the forward communication per layer per
    device (table tab:comm_summary)."""
    _mesh(strategy, d, t, sigma)
    bsh = b * s * c.hidden * c.beta_p
    if strategy == "DP":
        return 0.0, 0.0
    if strategy == "TP":          # two all-reduces of the B S h output (attention, MLP)
        return 2 * allreduce_bytes(bsh, d), 0.0
    if strategy == "SP":          # all-gather of K and V, 2 B S h / g in total
        return allgather_bytes(2 * bsh / c.g, d), 0.0
    if strategy == "TP+SP":       # K/V all-gather of the T-sharded heads over Sigma,
        #                           plus the two output all-reduces of the S/Sigma rows over T
        return (allgather_bytes(2 * bsh / (c.g * t), sigma)
                + 2 * allreduce_bytes(bsh / sigma, t)), 0.0
    # TSP: the K/V all-gather of SP, D broadcasts of the packed attention shard
    # (P_attn / D each) and D - 1 ring steps of an MLP shard (P_mlp / D each)
    act = allgather_bytes(2 * bsh / c.g, d)
    weights = (d * broadcast_bytes(params_attn(c) * c.beta_p / d, d)
               + (d - 1) * params_mlp(c) * c.beta_p / d)
    return act, weights


def comm_bytes(strategy: str, phase: str, c: ModelConfig, b: int, s: int, d: int,
               t: int | None = None, sigma: int | None = None,
               tsp_grad: str = "printed") -> float:
    """Communication volume per layer per device for a training phase (Section 4,
    per-strategy equations).  The backward pass repeats the forward exchange;
    full recomputation repeats it once more; DP, SP, TP+SP and TSP add the gradient
    reduction of the weights they replicate or circulate."""
    if phase not in PHASES:
        raise ValueError(f"phase must be one of {PHASES}, not {phase!r}")
    act, weights = comm_terms_fwd(strategy, c, b, s, d, t, sigma)
    reps = {"fwd": 1, "fwd+bwd": 2, "fwd+bwd+recomp": 3}[phase]
    grad_n = params_layer(c) * c.beta_g
    if phase == "fwd":
        return act + weights
    if strategy == "DP":          # forward is communication-free, recompute adds nothing
        return allreduce_bytes(grad_n, d)
    if strategy == "TP":
        return reps * act
    if strategy == "SP":
        return reps * act + allreduce_bytes(grad_n, d)
    if strategy == "TP+SP":       # gradients of the T-sharded weights, all-reduced over Sigma
        return reps * act + allreduce_bytes(grad_n / t, sigma)
    # TSP
    if tsp_grad == "printed":
        grad = allgather_bytes(grad_n, d) if phase == "fwd+bwd" else allreduce_bytes(grad_n, d)
    elif tsp_grad == "reduce":
        grad = allgather_bytes(grad_n, d)       # reduce-to-owner moves the same N (D-1)/D
    elif tsp_grad == "allreduce":
        grad = allreduce_bytes(grad_n, d)
    else:
        raise ValueError("tsp_grad must be 'printed', 'reduce' or 'allreduce'")
    return reps * (act + weights) + grad


# ---- FLOPs -------------------------------------------------------------------------

def layer_flops(c: ModelConfig, b: int, s: int) -> float:
    """F_layer = (4 (1 + 1/g) + 6 F) B S h^2 + 4 B S^2 h (Section 4, "FLOPs"):
    projections, gated MLP and the (non-causal) score and context products."""
    h = c.hidden
    return (4.0 * (1.0 + 1.0 / c.g) + 6.0 * c.ffn_factor) * b * s * h * h + 4.0 * b * s * s * h


def flops_per_device(strategy: str, c: ModelConfig, b: int, s: int, d: int,
                     t: int | None = None, sigma: int | None = None) -> float:
    """Leading-order forward FLOPs per device (table tab:flop_summary): DP runs the
    whole layer, every other scheme divides it by its D = T Sigma devices."""
    wdiv, adiv = _mesh(strategy, d, t, sigma)
    if strategy == "DP":
        return layer_flops(c, b, s)
    if strategy == "TP+SP":
        return layer_flops(c, b, s) / (wdiv * adiv)
    return layer_flops(c, b, s) / d


# ---- regime analysis ---------------------------------------------------------------

def tsp_beats_tp_large_d(c: ModelConfig, b: int, s: int) -> bool:
    """The large-D comparison of Section 4 ("Regime analysis"): with (D-1)/D taken
    as 1, TSP's forward volume is below TP's exactly when P_L < 2 B S h (2 - 1/g)."""
    return params_layer(c) < 2.0 * b * s * c.hidden * (2.0 - 1.0 / c.g)


def breakeven_tokens(c: ModelConfig, d: int | None = None) -> float:
    """Number of tokens B S at which TSP's and TP's forward volumes are equal.

    ``d=None`` is the large-D limit, P_L / (2 h (2 - 1/g)) (8 h for MHA with F = 4);
    a finite ``d`` solves the full table-row equality, whose weight term keeps the
    attention broadcast without the (D-1)/D factor."""
    h = c.hidden
    if d is None:
        return params_layer(c) / (2.0 * h * (2.0 - 1.0 / c.g))
    f = (d - 1) / d
    weights = params_attn(c) + params_mlp(c) * f
    return weights / (h * f * (4.0 - 2.0 / c.g))


# ---- report ------------------------------------------------------------------------

def _gb(x: float) -> str:
    return f"{x / 1e9:10.3f}"


def report(c: ModelConfig, b: int, s: int, d: int, t: int, sigma: int,
           recompute: str = "sel") -> str:
    lines = [f"model: h={c.hidden} L={c.layers} n_h={c.n_heads} n_kv={c.n_kv_heads} "
             f"d={c.head_dim} F={c.ffn_factor:g}; P_L={params_layer(c) / 1e6:.1f} M, "
             f"L*P_L={params_total(c) / 1e9:.2f} B",
             f"workload: B={b} S={s} D={d} (TP+SP: T={t} Sigma={sigma}), "
             f"activations: {recompute} recomputation", "",
             "communication per layer per device (GB)",
             f"{'strategy':8s} {'fwd':>10s} {'fwd+bwd':>10s} {'+recomp':>10s}"]
    for st in STRATEGIES:
        vals = [comm_bytes(st, ph, c, b, s, d, t, sigma) for ph in PHASES]
        lines.append(f"{st:8s} " + " ".join(_gb(v) for v in vals))
    lines += ["", "memory per GPU (GB)",
              f"{'strategy':8s} {'params':>10s} {'grads':>10s} {'optim':>10s} {'acts':>10s} "
              f"{'total':>10s}"]
    for st in STRATEGIES:
        m = memory_bytes(st, c, b, s, d, recompute, t, sigma)
        lines.append(f"{st:8s} " + " ".join(_gb(m[k]) for k in
                                            ("params", "grads", "optim", "acts", "total")))
    lines += ["", "forward FLOPs per layer per device (TFLOP)"]
    for st in STRATEGIES:
        lines.append(f"{st:8s} {flops_per_device(st, c, b, s, d, t, sigma) / 1e12:10.3f}")
    lines += ["", f"TSP/TP forward break-even: B S = {breakeven_tokens(c):.0f} tokens "
                  f"(large D), {breakeven_tokens(c, d):.0f} at D={d}; this workload has "
                  f"B S = {b * s}: TSP {'below' if tsp_beats_tp_large_d(c, b, s) else 'above'} "
                  f"TP at large D"]
    return "\n".join(lines)


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    r = reference_7b()
    ap.add_argument("--hidden", type=int, default=r.hidden)
    ap.add_argument("--layers", type=int, default=r.layers)
    ap.add_argument("--heads", type=int, default=r.n_heads)
    ap.add_argument("--kv-heads", type=int, default=r.n_kv_heads)
    ap.add_argument("--head-dim", type=int, default=r.head_dim)
    ap.add_argument("--ffn-factor", type=float, default=r.ffn_factor)
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--seq", type=int, default=16384)
    ap.add_argument("--degree", type=int, default=8)
    ap.add_argument("--tp", type=int, default=2, help="T of the TP+SP mesh (Sigma = D / T)")
    ap.add_argument("--recompute", choices=RECOMPUTE, default="sel")
    a = ap.parse_args(argv)
    if a.degree % a.tp:
        ap.error("--tp must divide --degree")
    c = ModelConfig(a.hidden, a.layers, a.heads, a.kv_heads, a.head_dim, a.ffn_factor)
    print(report(c, a.batch, a.seq, a.degree, a.tp, a.degree // a.tp, a.recompute))


if __name__ == "__main__":
    main()
