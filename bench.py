#!/usr/bin/env python3
"""Benchmark of one MoE layer (the LAEP hot path) on one MI355X.

Default workload ("balanced"): T=8192 tokens, d_model=2048, 64 experts,
top-8 renormalised softmax gating, SwiGLU d_ff=1024, bf16 with fp32
accumulation.  One step = one forward pass of the whole layer:
route -> expert counts -> permute -> grouped SwiGLU FFN -> combine.

Prints ONE JSON line:
  value      = tokens/s of the layer forward (inputs resident in HBM)
  roofline   = the grouped SwiGLU FFN (its two bf16 MFMA GEMM launches) against
               the bf16 dense MFMA peak, timed with HIP events on its stream
  cpu_baseline = the CPU oracle timed on a bounded token sample
Other workloads (--workload skewed | skewed_mild | shard | shard_bwd) are for
profiling; the shard workloads report routed rows/s.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def _cpu_baseline(w, c, budget_s: float):
    """Time the plain float64 oracle on a token sample of the same workload."""
    import numpy as np
    import oracle.moe as om

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1

    def run(n):
        t0 = time.perf_counter()
        if w.routed:
            om.layer_forward(c["x"][:n], c["w_router"], c["w_gate_up"], c["w_down"], w.k,
                             bias=c.get("bias"), renorm=w.renorm, dtype="bf16")
        else:
            idx = c["topk_idx"][:n]
            counts, offsets, dest = om.expert_counts(idx, w.E)
            xp = om.permute(c["x"][:n], dest, 1)
            y, act = om.grouped_ffn_fwd(xp, c["w_gate_up"], c["w_down"], offsets, dtype="bf16")
            om.combine(y, c["topk_gate"][:n], dest, 1, dtype="bf16")
        return time.perf_counter() - t0

    # grow the sample until one run costs about half the budget (or is whole)
    n = min(256, w.T)
    dt = run(n)
    for _ in range(4):
        if dt >= budget_s / 2 or n >= w.T:
            break
        n = int(min(w.T, max(2 * n, n * (budget_s * 0.6) / max(dt, 1e-3))))
        dt = run(n)
    unit = "tokens/s" if w.routed else "rows/s"
    return {"value": n / dt, "unit": unit, "cores": threads, "kind": "oracle",
            "sample": f"{n} of {w.T} {'tokens' if w.routed else 'rows'} of the same workload, "
                      f"full layer forward in float64 NumPy ({dt:.1f} s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="balanced")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the multi-GPU "
              f"expert-parallel path is not part of this build.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2601_14327_amd as laep
    from workloads import WORKLOADS, cached

    w = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    c = cached(w.name)
    bf = torch.bfloat16
    to = lambda a, dt=bf: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)

    # three input sets rotated per step so activations are not cache-resident
    n_sets = 3
    rng = np.random.default_rng(0)
    xs = [to(c["x"])] + [to(c["x"][rng.permutation(w.T)]) for _ in range(n_sets - 1)]
    wgu, wd = to(c["w_gate_up"]), to(c["w_down"])
    plan = laep.MoELayerPlan(w.T, w.d_model, w.E, w.k, w.d_ff, dtype=bf, device=dev,
                             backward=w.backward)
    if w.routed:
        wr = to(c["w_router"])
        bias = to(c["bias"], torch.float32) if "bias" in c else None

        def step(i):
            return plan.forward(xs[i % n_sets], wr, wgu, wd, bias=bias, renorm=w.renorm,
                                prune_beta=w.prune_beta, prune_alpha=w.prune_alpha)
    else:
        idx = to(c["topk_idx"], torch.int32)
        gate = to(c["topk_gate"], torch.float32)
        dout = to(c["dout"]) if w.backward else None

        def step(i):
            plan.forward_given_routing(xs[i % n_sets], idx, gate, wgu, wd)
            if w.backward:
                plan.backward(dout, wgu, wd)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = wall * 1e3 / args.steps

    # ---- the dominant kernel: grouped SwiGLU FFN, HIP events on its stream ----
    stream = torch.cuda.current_stream(dev)
    n_ev = max(10, args.steps)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n_ev)]
    for i in range(n_ev):
        s, e = evs[i]
        s.record(stream)
        laep.moe_grouped_ffn_fwd(plan.x_perm, wgu, wd, plan.offsets, ws=plan.ws_ffn,
                                 y_perm=plan.y_perm, act_save=plan.act_save)
        e.record(stream)
    torch.cuda.synchronize()
    ffn_ms = sorted(s.elapsed_time(e) for s, e in evs)
    ffn_ms_avg = sum(ffn_ms) / len(ffn_ms)
    R = w.T * w.k
    ffn_flops = 6.0 * R * w.d_model * w.d_ff
    achieved = ffn_flops / (ffn_ms_avg * 1e-3) / 1e12

    # ---- per-step breakdown (events around each call) -------------------------
    breakdown = {}
    if w.routed:
        x0 = xs[0]
        parts = [("route", lambda: plan.route(x0, wr, bias=bias, renorm=w.renorm)),
                 ("counts", lambda: plan.count()),
                 ("permute", lambda: laep.moe_permute(x0, plan.dest_row, w.k, R,
                                                      out=plan.x_perm)),
                 ("combine", lambda: laep.moe_combine(plan.y_perm, plan.topk_gate,
                                                      plan.dest_row, out=plan.out))]
        for name, fn in parts:
            es = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(10)]
            for s, e in es:
                s.record(stream)
                fn()
                e.record(stream)
            torch.cuda.synchronize()
            breakdown[name + "_us"] = round(1e3 * sum(s.elapsed_time(e) for s, e in es) / 10, 2)
        elem = 2
        bytes_route = w.T * w.d_model * elem + w.E * w.d_model * elem + 2 * w.T * w.k * 4
        bytes_perm = w.T * w.d_model * elem + R * w.d_model * elem + R * 4
        breakdown["route_GBs"] = round(bytes_route / (breakdown["route_us"] * 1e-6) / 1e9, 1)
        breakdown["permute_GBs"] = round(bytes_perm / (breakdown["permute_us"] * 1e-6) / 1e9, 1)
        breakdown["combine_GBs"] = round(
            (R * w.d_model * elem + w.T * w.d_model * elem + R * 8)
            / (breakdown["combine_us"] * 1e-6) / 1e9, 1)
    breakdown["ffn_us"] = round(ffn_ms_avg * 1e3, 2)
    breakdown["ffn_TFLOPs"] = round(achieved, 1)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = _cpu_baseline(w, c, args.cpu_budget)

    unit = "tokens/s" if w.routed else "rows/s"
    per_step = w.T
    metric = ("MoE-layer tokens/s at 1 GPU; grouped-GEMM TFLOP/s as % bf16 MFMA peak"
              if w.routed else "MoE expert-shard routed rows/s at 1 GPU (fwd" +
              ("+bwd" if w.backward else "") + ")")
    line = {
        "metric": metric,
        "value": per_step / (ms * 1e-3),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; random-init weights)",
        "config": {"workload": f"{w.name}: T={w.T} d_model={w.d_model} E={w.E} k={w.k} "
                               f"d_ff={w.d_ff} bf16" + (" fwd+bwd" if w.backward else " fwd"),
                   "tokens": w.T, "experts": w.E, "top_k": w.k, "d_model": w.d_model,
                   "d_ff": w.d_ff},
        "roofline": {"bound": "mfma", "kernel": "grouped SwiGLU FFN fwd (gate/up + down GEMMs)",
                     "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None},
        "cpu_baseline": cpu,
        "breakdown": breakdown,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
