#!/usr/bin/env python3
"""Throughput of one rank's TSP layer forward (attention + gated MLP) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--rank P]
                    [--layout contiguous|zigzag] [--group-steps G] [--no-cpu-baseline]
                    [--rank-sweep]

A step is one ``tsp_layer_rank_fwd`` call: all D attention shard steps (Q/K/V
projection, causal flash attention, output projection) and all D ring MLP steps
(gate+up with SwiGLU, down projection) for the rank's S/D tokens, the shard steps taken
in groups of G (tsp_shape.group_steps; 0 = the library default, all D steps when
D <= 8, since every shard is resident).  Inputs, weight
shards and the K/V rows of the earlier ranks (the modelled all-gather) are resident
in HBM before timing starts.  Prints one JSON line on stdout; progress goes to stderr.

Besides the layer call the line reports the attention-only and MLP-only entry points
timed separately ("blocks"), the per-rank MLP backward (``tsp_mlp_rank_bwd``, with its
kernel classes) on the same rank ("blocks.mlp_bwd"), the two-stage attention backward
("blocks.attn_bwd": ``tsp_attn_rank_bwd_saved`` from the activations a
``tsp_attn_rank_fwd_train`` call kept, then ``tsp_attn_kv_rank_bwd``; the recomputing
``tsp_attn_rank_bwd`` beside it), the algorithmic HBM bytes of a step
and the bandwidth they imply ("hbm"), the paper's non-causal F_layer / D for reference,
and with --rank-sweep the layer time of every rank of the group and the max/min
imbalance.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "TFLOP/s per TSP rank layer fwd (MLP+attn), % of bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA: 256 CUs x 2.4 GHz x 4096 FLOP/clk/CU
PEAK_HBM_GBS = 8000.0


# HBM bytes per launch of a workload's dominant kernel, from rocprofv3 --pmc FETCH_SIZE and
# WRITE_SIZE runs (KiB per dispatch) scaled by what the same counters read for a 1 GiB device
# copy (FETCH x 2.0, WRITE x 1.0).  A record only applies to the kernel source it was taken
# on (sha256 prefix); after any change to that source the traffic is reported as null.
MEASURED_TRAFFIC = {
    # flash_fwd_kernel<128, false>: one launch over 4 shards' 16 heads with paired query
    # tiles (2 per layer step), no key-range split (668 450.8 / 32 768.3 KiB)
    ("7b-h4096-S65536-D8", 7, "attn"): {
        "source": "flash_attn.hip", "sha256": "7938e38808f946ca",
        "fetch_kib": 668450.8, "fetch_scale": 2.0, "write_kib": 32768.3, "write_scale": 1.0},
}


def measured_traffic(wl, kernel):
    rec = MEASURED_TRAFFIC.get((wl.name, wl.rank, kernel))
    if rec is None:
        return None
    path = os.path.join(ROOT, "paper_2604_26294_amd", "csrc", rec["source"])
    with open(path, "rb") as f:
        if hashlib.sha256(f.read()).hexdigest()[:16] != rec["sha256"]:
            return None
    return 1024.0 * (rec["fetch_kib"] * rec["fetch_scale"] + rec["write_kib"] * rec["write_scale"])


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def kernel_flops(wl):
    """Algorithmic FLOPs of each kernel class (TSP_KERNEL_* order) over one call of the
    entry point that launches it (all D shard steps), whatever the number of launches:
    the forward's products of one group of steps share a launch, and so do the two dX
    products of one MLP backward step."""
    from paper_2604_26294_amd.flops import step_attn_core_flops
    D = wl.degree
    m = wl.batch * wl.s_loc
    h = wl.hidden
    fs = wl.ffn // D
    qd = wl.n_heads // D * wl.head_dim
    kd = wl.n_kv_heads // D * wl.head_dim
    core = step_attn_core_flops(wl)
    per_step = {"gate_up": 2.0 * m * 2 * fs * h, "down": 2.0 * m * h * fs,
                "qkv": 2.0 * m * (qd + 2 * kd) * h, "attn": core,
                "oproj": 2.0 * m * qd * h,
                # MLP backward: G, U and dHs in one pass; dX = dG W1 + dU W3; the three
                # weight gradients
                "bwd_gate": 2.0 * m * 3 * fs * h, "bwd_dx": 2 * 2.0 * m * fs * h,
                "bwd_dw": 3 * 2.0 * m * fs * h,
                # attention backward, first stage: the Q and dA products; the forward
                # recomputation; dK/dV recomputes S and forms dP, dV, dK (2x the core); dQ
                # recomputes S, dP and forms dQ (1.5x); the dX product and the two
                # weight-gradient products
                "abwd_proj": 2 * 2.0 * m * qd * h, "abwd_fwd": core,
                "abwd_kv": 2.0 * core, "abwd_q": 1.5 * core,
                "abwd_dx": 2.0 * m * qd * h, "abwd_dw": 2 * 2.0 * m * qd * h}
    return {k: D * v for k, v in per_step.items()}


def host_cpu_info():
    """Logical CPUs of the host, the ones this process may run on, and the CPU model."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"nproc": usable, "logical_cpus": os.cpu_count(), "cpu_model": model}


def cpu_baseline(wl, x_bits, w_bits, rows: int):
    """Time the fp64 oracle on a bounded sample of the same rank's work."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import tsp_oracle as O
    from paper_2604_26294_amd import inputs as I

    p, D = wl.rank, wl.degree
    hs, ks, d = wl.n_heads // D, wl.n_kv_heads // D, wl.head_dim
    x = I.bf16_bits_to_f64(x_bits[:, :(p + 1) * wl.s_loc])
    w = {k: I.bf16_bits_to_f64(v) for k, v in w_bits.items()}
    chunks = [I.local_chunk(x, q, D) for q in range(p + 1)]
    attn_sh = [I.attn_shard_packed(w, r, D, wl.n_heads, wl.n_kv_heads, d) for r in range(D)]
    mlp_sh = [I.mlp_shard(w, j, D) for j in range(D)]
    log("cpu baseline: gathering K/V of the prefix (untimed)")
    kv = [O.gather_kv(chunks, attn_sh[r], hs, ks, d) for r in range(D)]
    sel = np.linspace(0, wl.s_loc - 1, rows).round().astype(int)
    x_loc = chunks[p]
    log(f"cpu baseline: timing the oracle on {rows} local rows")
    t0 = time.perf_counter()
    attn = O.attn_rank(x_loc, attn_sh, kv, p, wl.n_heads, wl.n_kv_heads, d, rows=sel)
    mlp = O.mlp_rank(x_loc[:, sel], [m[0] for m in mlp_sh], [m[1] for m in mlp_sh],
                     [m[2] for m in mlp_sh], p)
    dt = time.perf_counter() - t0
    assert np.isfinite(attn).all() and np.isfinite(mlp).all()
    b, h = wl.batch, wl.hidden
    qd = wl.n_heads * d
    keys = float(np.sum(p * wl.s_loc + sel + 1))
    flops = (b * rows * (6.0 * h * wl.ffn + 4.0 * h * qd)
             + 4.0 * b * wl.n_heads * d * keys)
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max((i.get("num_threads", 1) for i in blas), default=1)
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle", "seconds": round(dt, 3), "host": host_cpu_info(),
            "blas": [{"vendor": i.get("internal_api"), "version": i.get("version"),
                      "threads": i.get("num_threads"),
                      "architecture": i.get("architecture")} for i in blas],
            "sample": (f"rank {p}: {rows} of {wl.s_loc} local rows per batch entry, all heads "
                       f"and all {D} shards (Q/O projections, causal attention over the "
                       f"prefix, gated MLP) in fp64 NumPy; K/V of the prefix gathered "
                       f"beforehand, untimed")}


def time_calls(fn, steps, warmup):
    """Average ms of fn() over `steps` calls on the current stream, after `warmup`."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        fn()
    t1.record(stream)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def rank_sweep(wl, x_bits, w_bits, steps, warmup, group_steps=0):
    """Layer time of every rank of the group (each with its own K/V prefix pre-filled)."""
    import torch

    from paper_2604_26294_amd.flops import paper_layer_flops, rank_algorithmic_bytes, rank_flops
    from paper_2604_26294_amd.harness import RankProblem
    rows = []
    for p in range(wl.degree):
        w = wl.at_rank(p)
        prob = RankProblem(w, x_bits, w_bits, p, group_steps=group_steps)
        prob.prefill_kv()
        torch.cuda.synchronize()
        ms = time_calls(prob.layer, steps, warmup)
        rows.append({"rank": p, "ms": round(ms, 4),
                     "tflops": round(rank_flops(w).total / (ms * 1e-3) / 1e12, 2)})
        log(f"rank {p}: {ms:.3f} ms/step")
        del prob
        torch.cuda.empty_cache()
    times = [r["ms"] for r in rows]
    return {"ranks": rows, "imbalance_max_over_min": round(max(times) / min(times), 4)}


def main(argv=None):
    from paper_2604_26294_amd.workloads import BY_NAME, L7B_64K

    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=L7B_64K.name, choices=sorted(BY_NAME))
    ap.add_argument("--rank", type=int, default=None)
    ap.add_argument("--layout", default="contiguous", choices=["contiguous", "zigzag"],
                    help="sequence layout of the ranks (zigzag: Algorithm 1 as printed)")
    ap.add_argument("--group-steps", type=int, default=0,
                    help="forward shard steps per grouped launch (0 = library default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--forward-only", action="store_true",
                    help="skip the backward blocks (for short profiling runs)")
    ap.add_argument("--cpu-rows", type=int, default=1024)
    ap.add_argument("--rank-sweep", action="store_true",
                    help="also time the layer of every rank of the group")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MB",
                    help="run one plain device copy of MB MiB first (a known-size reference "
                         "for hardware byte counters)")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one rank of a TSP group on ONE GPU; this build has no "
              "multi-GPU path (--gpus must be 1)", file=sys.stderr)
        return 2

    import torch

    from paper_2604_26294_amd import inputs as I
    from paper_2604_26294_amd import tsp as T
    from paper_2604_26294_amd.flops import paper_layer_flops, rank_algorithmic_bytes, rank_flops
    from paper_2604_26294_amd.harness import RankProblem, to_device_bf16

    wl = BY_NAME[args.workload].with_layout(1 if args.layout == "zigzag" else 0)
    if args.rank is not None:
        wl = wl.at_rank(args.rank)
    torch.cuda.set_device(0)
    log(f"workload {wl.name} rank {wl.rank}: generating seeded inputs")
    x_bits = I.make_x_full(wl)
    w_bits = I.make_weights(wl)
    prob = RankProblem(wl, x_bits, w_bits, group_steps=args.group_steps)
    group = min(args.group_steps or T.GROUP_STEPS_MAX, wl.degree)
    log("pre-filling the K/V rows of earlier ranks (the modelled all-gather, untimed)")
    prob.prefill_kv()
    torch.cuda.synchronize()

    if args.copy_calibration > 0:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {n} bytes read, {n} bytes written")
        del src, dst

    for _ in range(args.warmup):
        prob.layer()
    torch.cuda.synchronize()

    # The headline: K steps between two events, the library's per-kernel timing off.
    stream = torch.cuda.current_stream()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(args.steps):
        prob.layer()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    log(f"{args.steps} steps: {ms:.3f} ms/step")

    # A second pass of K steps with every launch bracketed by HIP events on the launch
    # stream: per-kernel-class times and the dominant kernel's roofline.
    T.tsp_profile_enable(True)
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(args.steps):
        prob.layer()
    t1.record(stream)
    torch.cuda.synchronize()
    T.tsp_profile_enable(False)
    ms_prof = t0.elapsed_time(t1) / args.steps
    log(f"{args.steps} steps with per-kernel events: {ms_prof:.3f} ms/step")

    rf = rank_flops(wl)
    tflops = rf.total / (ms * 1e-3) / 1e12
    kf = kernel_flops(wl)
    kernels = {}
    for k, name in enumerate(T.KERNELS):
        tot, n = T.tsp_profile_read(k)
        if n == 0:
            continue
        avg = tot / n
        kernels[name] = {"avg_ms": round(avg, 5), "launches_per_step": n // args.steps,
                         "tflops": round(kf[name] / (tot / args.steps * 1e-3) / 1e12, 2),
                         "time_share": round(tot / args.steps / ms_prof, 4)}
    dom = max(kernels, key=lambda n: kernels[n]["time_share"])
    dom_avg = kernels[dom]["avg_ms"]
    dom_flops = kf[dom] / kernels[dom]["launches_per_step"]  # per launch
    achieved = dom_flops / (dom_avg * 1e-3) / 1e12
    roofline = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic(wl, dom),
                "flops_per_launch": dom_flops, "avg_launch_ms": dom_avg}

    # The attention and MLP entry points on their own (same rank, same buffers).
    ms_attn = time_calls(prob.attn_fwd, args.steps, 2)
    ms_mlp = time_calls(prob.mlp, args.steps, 2)
    blocks = {
        "attn": {"ms": round(ms_attn, 4), "flops": rf.attn,
                 "tflops": round(rf.attn / (ms_attn * 1e-3) / 1e12, 2)},
        "mlp": {"ms": round(ms_mlp, 4), "flops": rf.mlp,
                "tflops": round(rf.mlp / (ms_mlp * 1e-3) / 1e12, 2)},
    }
    if args.forward_only:
        return finish(args, wl, x_bits, w_bits, ms, ms_prof, rf, tflops, roofline, kernels,
                      blocks)
    # The per-rank MLP backward on the same rank: dX and this rank's contribution to
    # every shard's weight gradients, for a synthetic upstream gradient.  Executed
    # products: G, U (recomputed) and dHs, dX (two), the three weight gradients = 16 M F h
    # FLOPs; the backward alone (without recomputing G, U) is 12 M F h.
    dy = to_device_bf16(I.gaussian_bf16(wl.seed, I.TENSOR_ID["dy"],
                                        (wl.batch, wl.s_loc, wl.hidden), wl.x_std))
    for _ in range(2):
        prob.mlp_bwd(dy)
    torch.cuda.synchronize()
    T.tsp_profile_enable(True)
    ms_bwd = time_calls(lambda: prob.mlp_bwd(dy), args.steps, 0)
    T.tsp_profile_enable(False)
    m_tok = wl.batch * wl.s_loc
    bwd_flops = 16.0 * m_tok * wl.ffn * wl.hidden
    bwd_kernels = {}
    for k, name in enumerate(T.KERNELS):
        if not name.startswith("bwd_"):
            continue
        tot, n = T.tsp_profile_read(k)
        if n:
            bwd_kernels[name] = {"avg_ms": round(tot / n, 5), "launches": n // args.steps,
                                 "tflops": round(kf[name] / (tot / args.steps * 1e-3) / 1e12,
                                                 2)}
    blocks["mlp_bwd"] = {"ms": round(ms_bwd, 4), "flops": bwd_flops,
                         "tflops": round(bwd_flops / (ms_bwd * 1e-3) / 1e12, 2),
                         "flops_note": "16 M F h executed (G, U recomputed); 12 M F h without",
                         "kernels": bwd_kernels}

    # The per-rank attention backward: first stage (all D shards: dA, the flash backward,
    # dX query path, dW_Q and dW_O^T contributions, this rank's dK/dV contributions for
    # every key) and second stage (K/V projection backward on the rank's rows, fed with
    # synthetic reduce-scattered gradients).  The training path takes A and the
    # log-sum-exp kept by the forward (tsp_attn_rank_fwd_train, run once untimed); the
    # recomputing entry point (tsp_attn_rank_bwd) is timed beside it.
    prob.prefill_kv(include_self=True)
    dk_bits, dv_bits = I.make_dkv_own(wl, wl.rank)
    dkl, dvl = to_device_bf16(dk_bits), to_device_bf16(dv_bits)
    del dk_bits, dv_bits
    prob.attn_fwd_train()
    for _ in range(2):
        prob.attn_bwd_saved(dy)
        prob.attn_bwd(dy)
        prob.attn_kv_bwd(dkl, dvl)
    torch.cuda.synchronize()
    T.tsp_profile_enable(True)
    ms_ab1 = time_calls(lambda: prob.attn_bwd_saved(dy), args.steps, 0)
    ab1_kernels = {}
    for k, name in enumerate(T.KERNELS):
        if not name.startswith("abwd_"):
            continue
        tot, n = T.tsp_profile_read(k)
        if n:
            e = {"avg_ms": round(tot / n, 5), "launches": n // args.steps,
                 "time_share": round(tot / args.steps / ms_ab1, 4)}
            if name != "abwd_aux":
                e["tflops"] = round(kf[name] / (tot / args.steps * 1e-3) / 1e12, 2)
            ab1_kernels[name] = e
    T.tsp_profile_enable(False)
    ms_ab1_re = time_calls(lambda: prob.attn_bwd(dy), args.steps, 0)
    ms_ab2 = time_calls(lambda: prob.attn_kv_bwd(dkl, dvl), args.steps, 0)
    D = wl.degree
    core = kf["attn"] / D
    qd = wl.n_heads // D * wl.head_dim
    kd = wl.n_kv_heads // D * wl.head_dim
    gemm1 = 5 * 2.0 * m_tok * qd * wl.hidden          # Q, dA, dX, dW_Q, dW_O^T per shard
    exec1 = D * (gemm1 + (2 + 1.5) * core)            # with the kept A and lse
    exec1_re = exec1 + D * core                        # plus the forward recomputation
    alg1 = D * (4 * 2.0 * m_tok * qd * wl.hidden + 2.5 * core)  # without Q, S, A recompute
    flops2 = D * 4 * 2.0 * m_tok * kd * wl.hidden      # dX (K, V) and dW_K, dW_V per shard
    blocks["attn_bwd"] = {
        "ms": round(ms_ab1 + ms_ab2, 4), "stage1_ms": round(ms_ab1, 4),
        "stage2_ms": round(ms_ab2, 4),
        "flops_executed": exec1 + flops2, "flops_backward": alg1 + flops2,
        "tflops_executed": round((exec1 + flops2) / ((ms_ab1 + ms_ab2) * 1e-3) / 1e12, 2),
        "tflops_backward": round((alg1 + flops2) / ((ms_ab1 + ms_ab2) * 1e-3) / 1e12, 2),
        "flops_note": "stage one from the forward's kept A and log-sum-exp "
                      "(tsp_attn_rank_bwd_saved); executed: with the Q recomputation and the "
                      "two flash backward kernels' repeated score and dP products (3.5x the "
                      "forward core); backward: 2.5x the forward core plus the gradient "
                      "products",
        "recompute": {"stage1_ms": round(ms_ab1_re, 4), "ms": round(ms_ab1_re + ms_ab2, 4),
                      "tflops_executed": round((exec1_re + flops2) /
                                               ((ms_ab1_re + ms_ab2) * 1e-3) / 1e12, 2),
                      "tflops_backward": round((alg1 + flops2) /
                                               ((ms_ab1_re + ms_ab2) * 1e-3) / 1e12, 2),
                      "note": "tsp_attn_rank_bwd: A and the log-sum-exp recomputed (4.5x)"},
        "kernels": ab1_kernels}
    del dy, dkl, dvl
    return finish(args, wl, x_bits, w_bits, ms, ms_prof, rf, tflops, roofline, kernels, blocks)


def finish(args, wl, x_bits, w_bits, ms, ms_prof, rf, tflops, roofline, kernels, blocks):
    """Prints the JSON line (with the rank sweep and the CPU baseline when asked for)."""
    from paper_2604_26294_amd import tsp as T
    from paper_2604_26294_amd.flops import paper_layer_flops, rank_algorithmic_bytes
    group = min(args.group_steps or T.GROUP_STEPS_MAX, wl.degree)
    nbytes = rank_algorithmic_bytes(wl)
    hbm = {"algorithmic_bytes": nbytes, "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
           "frac_of_peak": round(nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
           "note": "all D weight shards + K/V prefix once + x (bf16) + Y (fp32), per step"}

    out = {
        "metric": METRIC, "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "seq": wl.seq, "hidden": wl.hidden,
                   "ffn": wl.ffn, "n_heads": wl.n_heads, "n_kv_heads": wl.n_kv_heads,
                   "head_dim": wl.head_dim, "degree": wl.degree, "rank": wl.rank,
                   "layout": wl.layout_name, "group_steps": group},
        "pct_of_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "flops_per_step": rf.total,
        "paper_flops_per_rank_noncausal": paper_layer_flops(wl) / wl.degree,
        "roofline": roofline,
        "kernels": kernels,
        "kernels_pass_ms_per_step": round(ms_prof, 4),
        "blocks": blocks,
        "hbm": hbm,
        "cpu_baseline": None,
    }
    if args.rank_sweep:
        out["rank_sweep"] = rank_sweep(wl, x_bits, w_bits, max(3, args.steps // 4), 2,
                                       args.group_steps)
    if not args.no_cpu_baseline and wl.layout == 0:  # the sampled oracle leg is contiguous-only
        out["cpu_baseline"] = cpu_baseline(wl, x_bits, w_bits, args.cpu_rows)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
