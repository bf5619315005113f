#!/usr/bin/env python3
"""Benchmark of one MoE layer (the LAEP hot path) on one MI355X.

Default workload ("balanced"): T=8192 tokens, d_model=2048, 64 experts,
top-8 renormalised softmax gating, SwiGLU d_ff=1024, bf16 with fp32
accumulation.  One step = one forward pass of the whole layer:
route + expert counts (one call) -> dispatch + grouped SwiGLU FFN (one call, the
dispatch folded into the FFN's operand loads) -> combine, every call a kernel
of the C-ABI library; input sets rotate over the steps (at least three, and
together more than twice the 256 MB MALL) so the activations are not
cache-resident.  With one slot per token (shard,
shard_bwd) the combine folds into the FFN call as well (the down projection
writes each row, times its gate, to its token row).  Training steps write no
x_perm and no dy_perm: the weight gradient gathers the token rows through
row_src as well, and the expert backward forms dY = g * dout on load.

Prints ONE JSON line:
  value        tokens/s of the whole step (wall clock over the timed steps,
               inputs resident in HBM)
  roofline     the dominant call (the grouped FFN) against the bf16 dense MFMA
               peak; its duration comes from HIP events recorded around it on
               its stream in every timed step.  `traffic` is the HBM bytes per
               call from the committed rocprofv3 counter summary, reported only
               while the kernel sources still match the ones it was taken on.
  breakdown    every call: mean / median / p10 / p90 microseconds over a second
               pass of the same steps with events around every call, and its rate
               on algorithmic bytes or flops (the timed pass brackets only the
               dominant call, since each event marker costs the GPU a few us)
  attainable   what a plain copy kernel and a bf16 MFMA loop reach on this GPU
  supplementary  moe_expert_counts at T x {1, 8, 64} tokens; route, counts, the
               two back to back, and the fused moe_route_count, each timed alone
  cpu_baseline the float64 CPU oracle timed on a bounded token sample (all BLAS
               threads, and one thread on a smaller sample)
  warm         the step with the same input set every step
  settle       untimed steps run before the warmup until the step time is
               steady (the GPU's clocks ramp up over the first ~1 s of load)
  placement    expert rearrangement (Algorithm 2, laep_rearrange) of the
               per-expert loads the last step counted, into 8 device groups:
               group sums of the greedy and of the contiguous placement, the
               straggler factor max/mean of each, a lower bound and, for at
               most 16 experts, the exact optimum
  padding      rows of the FFN's 256-row tiles beyond the routed rows
               (sum over experts of ceil(M_e / 256) * 256 - R)

Other workloads: skewed, skewed_mild (routed, pruned every step), shard (16
experts, given Zipf routing), shard_bwd (shard forward + backward),
balanced_bwd (balanced forward + backward through the combine, FFN, dispatch
and router), mild_pruned (Algorithm 1 over a window of batches before the
timed steps, pruned experts removed; the steps run the compact layer, and
`pruning` reports the parameter reduction and the one-time repack).

Profiling helpers (used by the commands recorded under profiles/):
  --profile-target ffn|copy   run only that call a few times (for --pmc runs);
                              route_feed: moe_route_count beside a blocked read of
                              the same x bytes in the router's launch shape
  --library-ref               the grouped FFN and its backward on 64 equal experts
                              of 1024 rows beside torch.matmul / torch.bmm
                              (hipBLASLt) on the same products (context, not the
                              metric)
  --summarize-pmc DIR         turn FETCH_SIZE / WRITE_SIZE counter CSVs into the
                              traffic summary (--out FILE)
  --summarize-trace DIR       turn a --kernel-trace --stats run into a summary
                              (--append-log FILE adds the run's JSON result line)
  --summarize-counters DIR    turn --pmc runs of SQ / GRBM counters on one call
                              into a per-kernel summary (MFMA busy, LDS, waits,
                              clock)
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
CSRC = os.path.join(ROOT, "paper_2601_14327_amd", "csrc")
# sources of the forward FFN's kernels (traffic counts are valid for these bits only)
FFN_FWD_SOURCES = ["gemm_bf16.hip", "gemm_common.hpp", "tiles.hpp", "common.hpp"]
FFN_BWD_SOURCES = ["gemm_bwd.hip", "gemm_common.hpp", "tiles.hpp", "common.hpp"]
COPY_CALIB_BYTES = 1 << 32
MALL_BYTES = 256 << 20   # MI355X last-level (Infinity) cache
PROFILE_CALLS = 5
PROFILES = os.path.join(ROOT, "profiles")


def sources_sha(names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(CSRC, n), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------------------------------
# CPU oracle baseline
# ---------------------------------------------------------------------------------------
def _cpu_baseline(w, c, budget_s: float, keep=None):
    """Time the plain float64 oracle on a token sample of the same workload
    (``keep``: the surviving experts of a pruned layer)."""
    import oracle.moe as om

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1

    def run(n):
        t0 = time.perf_counter()
        sel = slice(None) if keep is None else keep
        wgu, wd = c["w_gate_up"][sel], c["w_down"][sel]
        if w.routed:
            bias = c.get("bias")
            f = om.layer_forward(c["x"][:n], c["w_router"][sel], wgu, wd, w.k,
                                 bias=None if bias is None else bias[sel], renorm=w.renorm,
                                 dtype="bf16")
        else:
            idx = c["topk_idx"][:n]
            counts, offsets, dest = om.expert_counts(idx, w.E)
            xp = om.permute(c["x"][:n], dest, 1)
            y, act = om.grouped_ffn_fwd(xp, wgu, wd, offsets, dtype="bf16")
            gate = c["topk_gate"][:n]
            om.combine(y, gate, dest, 1, dtype="bf16")
            f = dict(idx=idx, gate=gate, offsets=offsets, dest_row=dest, x_perm=xp, y_perm=y,
                     act_save=act)
        if w.backward:   # the training step's backward, the same chain the GPU step runs
            dy, dgate = om.combine_bwd(c["dout"][:n], f["y_perm"], f["gate"], f["dest_row"], w.k)
            dxp, dA, hb = om.grouped_ffn_dgrad(dy, f["act_save"], wgu, wd, f["offsets"])
            om.grouped_ffn_wgrad(dy, f["x_perm"], dA, hb, f["offsets"], wgu.shape[0])
            dx = om.permute_bwd(dxp, f["dest_row"], w.k)
            if w.routed:
                om.route_bwd(dgate, f["idx"], f["gate"], c["x"][:n], c["w_router"][sel],
                             logits=f["logits"], renorm=w.renorm, dx_in=dx)
        return time.perf_counter() - t0

    # grow the sample until one run costs about half the budget (or is whole)
    n = min(256, w.T)
    dt = run(n)
    for _ in range(4):
        if dt >= budget_s / 2 or n >= w.T:
            break
        n = int(min(w.T, max(2 * n, n * (budget_s * 0.6) / max(dt, 1e-3))))
        dt = run(n)
    # the same oracle with its BLAS held to one thread, on a smaller sample
    n1 = max(16, min(n, int(n * (budget_s * 0.25) / max(dt * threads, 1e-3))))
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            dt1 = run(n1)
        one = {"value": n1 / dt1, "sample": f"{n1} {'tokens' if w.routed else 'rows'} ({dt1:.1f} s)"}
    except Exception as e:  # pragma: no cover
        one = {"error": str(e)}
    unit = "tokens/s" if w.routed else "rows/s"
    return {"value": n / dt, "unit": unit, "cores": threads, "kind": "oracle",
            "sample": f"{n} of {w.T} {'tokens' if w.routed else 'rows'} of the same workload, "
                      f"layer {'forward + backward' if w.backward else 'forward'} in float64 "
                      f"NumPy ({dt:.1f} s)",
            "one_thread": one}


# ---------------------------------------------------------------------------------------
# the layer step, call by call
# ---------------------------------------------------------------------------------------
class Setup:
    def __init__(self, w, dev):
        import numpy as np
        import torch

        import paper_2601_14327_amd as laep
        from workloads import cached

        self.w, self.dev = w, dev
        c = cached(w.name)
        self.c = c
        bf = torch.bfloat16
        to = lambda a, dt=bf: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
        rng = np.random.default_rng(0)
        # enough x sets that together they exceed twice the 256 MB MALL, so
        # no set is still cached when its turn comes again
        x_bytes = w.T * w.d_model * 2
        self.n_sets = max(3, -(-2 * MALL_BYTES // x_bytes))
        self.xs = [to(c["x"])] + [to(c["x"][rng.permutation(w.T)]) for _ in range(self.n_sets - 1)]
        self.wgu, self.wd = to(c["w_gate_up"]), to(c["w_down"])
        self.plan = laep.MoELayerPlan(w.T, w.d_model, w.E, w.k, w.d_ff, dtype=bf, device=dev,
                                      backward=w.backward)
        if w.routed:
            self.wr = to(c["w_router"])
            self.bias = to(c["bias"], torch.float32) if "bias" in c else None
        else:
            self.idx = to(c["topk_idx"], torch.int32)
            self.gate = to(c["topk_gate"], torch.float32)
        self.dout = to(c["dout"]) if w.backward else None
        self.laep = laep
        self.E = w.E
        self.keep = None
        self.pruning = None
        if w.prune_window:
            self._prune_and_compact()

    def _prune_and_compact(self):
        """Algorithm 1 over a window of routed batches, then the pruned experts
        leave the layer: router rows, bias and FFN weights are repacked and the
        timed steps run the compact layer."""
        import torch

        w, L = self.w, self.laep
        pruner = L.ExpertPruner(w.prune_window, 1, w.E, w.T, w.k, alpha=w.prune_alpha,
                                beta=w.prune_beta, device=self.dev)
        for it in range(w.prune_window):
            idx, _ = L.moe_route(self.xs[it % self.n_sets], self.wr, w.k, bias=self.bias,
                                 renorm=w.renorm)
            L.moe_expert_counts(idx, w.E, etn_accum=pruner.slot(it, 0))
        alive, n_pruned, _ = pruner.decide()
        alive = alive[0].contiguous()
        big = sum(t.numel() * t.element_size() for t in (self.wr, self.wgu, self.wd))
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        small = L.compact_layer(alive, w_router=self.wr, w_gate_up=self.wgu, w_down=self.wd,
                                bias=self.bias)
        # time the repack alone (the slot map is already known)
        s.record()
        L.laep_repack_experts(small["expert_map"], small["n_alive"], w_router=self.wr,
                              bias=self.bias, w_gate_up=self.wgu, w_down=self.wd,
                              out={k: small[k] for k in ("w_router", "bias", "w_gate_up",
                                                         "w_down") if small.get(k) is not None})
        e.record()
        torch.cuda.synchronize()
        self.wr, self.wgu, self.wd = small["w_router"], small["w_gate_up"], small["w_down"]
        self.bias = small.get("bias")
        self.E = small["n_alive"]
        self.keep = alive.cpu().numpy().astype(bool).nonzero()[0]
        kept = sum(t.numel() * t.element_size() for t in (self.wr, self.wgu, self.wd))
        us = s.elapsed_time(e) * 1e3
        self.pruning = {"window_iters": w.prune_window, "alpha": w.prune_alpha,
                        "beta": w.prune_beta, "experts_before": w.E, "experts_after": self.E,
                        "weight_bytes_before": big, "weight_bytes_after": kept,
                        "param_reduction": round(1 - kept / big, 4),
                        "repack_us": round(us, 1),
                        "repack_GBs": round(2 * kept / (us * 1e-6) / 1e9, 1)}
        self.plan = L.MoELayerPlan(w.T, w.d_model, self.E, w.k, w.d_ff, dtype=torch.bfloat16,
                                   device=self.dev, backward=w.backward)

    def calls(self, i):
        """(name, fn) for every call of step i, in order."""
        w, p, L = self.w, self.plan, self.laep
        x = self.xs[i % self.n_sets]
        R = w.T * w.k
        out = []
        if w.routed:   # routing and expert counts: one call (the router writes the count masks)
            rc = lambda alive=None: p.route_count(x, self.wr, bias=self.bias, alive=alive,
                                                  renorm=w.renorm)
            out += [("route_count", rc)]
            if w.prune_beta is not None and not w.prune_window:
                out += [("prune", lambda: p.prune(w.prune_beta, w.prune_alpha)),
                        ("route_count_masked", lambda: rc(p.alive))]
            gate = p.topk_gate
        else:
            out += [("counts", lambda: L.moe_expert_counts(self.idx, w.E, ws=p.ws_counts,
                                                           counts=p.counts, offsets=p.offsets,
                                                           dest_row=p.dest_row,
                                                           row_src=p.row_src))]
            gate = self.gate
        if p.fused_combine:   # one slot per token: dispatch and combine folded into the FFN
            out += [("ffn_fwd", lambda: L.moe_grouped_ffn_fwd_gather_combine(
                x, p.row_src, gate, self.wgu, self.wd, p.offsets, rows=R, ws=p.ws_ffn,
                out=p.out, keep_y=p.y_perm is not None, y_perm=p.y_perm,
                save_act=p.act_save is not None, act_save=p.act_save, x_perm_out=p.x_perm))]
        elif p.fused:   # dispatch folded into the FFN's operand loads
            if p.x_perm is not None:   # kept for inspection: the token-major permute
                out += [("permute", lambda: L.moe_permute(x, p.dest_row, w.k, R, out=p.x_perm))]
            out += [("ffn_fwd", lambda: L.moe_grouped_ffn_fwd_gather(
                x, p.row_src, w.k, self.wgu, self.wd, p.offsets, rows=R, ws=p.ws_ffn,
                y_perm=p.y_perm, save_act=p.act_save is not None, act_save=p.act_save))]
        else:
            out += [("permute", lambda: L.moe_permute(x, p.dest_row, w.k, R, out=p.x_perm)),
                    ("ffn_fwd", lambda: L.moe_grouped_ffn_fwd(
                        p.x_perm, self.wgu, self.wd, p.offsets, ws=p.ws_ffn, y_perm=p.y_perm,
                        save_act=p.act_save is not None, act_save=p.act_save))]
        if not p.fused_combine:
            out += [("combine", lambda: L.moe_combine(p.y_perm, gate, p.dest_row, out=p.out))]
        if w.backward:
            if p.dw_gate_up is None:
                import torch
                p.dw_gate_up = torch.empty(self.wgu.shape, dtype=torch.float32, device=self.dev)
                p.dw_down = torch.empty(self.wd.shape, dtype=torch.float32, device=self.dev)
            out += [("combine_bwd", lambda: L.moe_combine_bwd(
                self.dout, p.y_perm, gate, p.dest_row, dy_perm=p.dy_perm, dgate=p.dgate,
                want_dy=p.dy_perm is not None))]
            if w.routed:   # the router's weight gradients on a side stream, beside the FFN's
                out += [("route_bwd_w", lambda: p.route_backward_weights_async(x, self.wr))]
            out += [("ffn_bwd", lambda: L.moe_grouped_ffn_bwd_gather(
                        None, x, p.row_src, w.k, p.act_save, self.wgu, self.wd,
                        p.offsets, dout=self.dout, topk_gate=gate,
                        h_fwd=L.ffn_fwd_h_view(p.ws_ffn, R, w.d_ff, p.dtype),
                        dw_gate_up=p.dw_gate_up, dw_down=p.dw_down, ws=p.ws_bwd,
                        dx_perm=p.dx_perm) if p.fused else L.moe_grouped_ffn_bwd(
                        p.dy_perm, p.x_perm, p.act_save, self.wgu, self.wd, p.offsets,
                        h_fwd=L.ffn_fwd_h_view(p.ws_ffn, R, w.d_ff, p.dtype),
                        dw_gate_up=p.dw_gate_up, dw_down=p.dw_down, ws=p.ws_bwd,
                        dx_perm=p.dx_perm)),
                    ("permute_bwd", lambda: L.moe_permute_bwd(p.dx_perm, p.dest_row, w.T, w.k,
                                                              out=p.dx))]
            if w.routed:   # router's dx, accumulated onto dx; then wait for route_bwd_w
                out += [("route_bwd_dx", lambda: p.route_backward_data(x, self.wr))]
        return out

    def algorithmic(self):
        """Algorithmic bytes (HBM-bound calls) or flops (matrix-core calls) per call."""
        w = self.w
        T, d, E, k, f = w.T, w.d_model, self.E, w.k, w.d_ff
        R = T * k
        e = 2  # bf16
        by = {
            "route": T * d * e + E * d * e + 2 * T * k * 4,
            "counts": T * k * 4 + 2 * (E + 1) * 4 + R * 4,
            "permute": T * d * e + R * d * e + R * 4,
            "combine": R * d * e + T * d * e + 2 * R * 4,
            # dout and y_perm read, gates and dest rows read, dgate written; dy_perm
            # written only when the plan keeps it (the fused backward forms dY
            # on load instead)
            "combine_bwd": T * d * e + R * d * e + 3 * R * 4
            + (R * d * e if getattr(self.plan, "dy_perm", None) is not None else 0),
            "permute_bwd": R * d * e + T * d * e + R * 4,
            # dx read + written, W_r once, x once (summed into dW_r), dgate/gates/ids, dW_r
            "route_bwd": 2 * T * d * e + E * d * e + T * d * e + 3 * T * k * 4 + E * d * 4,
        }
        by["route_count"] = by["route"] + by["counts"]
        by["route_count_masked"] = by["route_count"]
        fl = {"ffn_fwd": 6.0 * R * d * f, "ffn_bwd": 12.0 * R * d * f}
        return by, fl


def _settle(su, min_s=1.0, max_s=6.0, batch=10, tol=0.01):
    """Untimed steps until the step time is steady: batches of `batch` steps,
    at least `min_s` seconds, until two consecutive batch means agree within
    `tol` (or `max_s` seconds).  Returns (steps, seconds)."""
    import torch

    t_start = time.perf_counter()
    prev, n = None, 0
    while True:
        t0 = time.perf_counter()
        for i in range(batch):
            for _, fn in su.calls(n + i):
                fn()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / batch
        n += batch
        el = time.perf_counter() - t_start
        if el >= max_s or (el >= min_s and prev is not None and abs(dt - prev) <= tol * prev):
            return n, round(el, 2)
        prev = dt


def _placement(su, n_groups=8):
    """Algorithm 2 on the loads the last step counted (alive experts only)."""
    import numpy as np

    counts = su.plan.counts.cpu().numpy().astype(np.float64)
    ids = np.arange(counts.shape[0])
    if getattr(su.plan, "alive", None) is not None and su.w.prune_beta is not None \
            and not su.w.prune_window:
        ids = np.nonzero(su.plan.alive.cpu().numpy().astype(bool))[0]
    elif su.keep is not None:       # compact layer: name the survivors by their old ids
        ids = np.asarray(su.keep)
    loads = counts[:len(ids)] if su.keep is not None else counts[ids]
    rep = su.laep.placement_report(loads, n_groups, expert_ids=ids)
    rep["source"] = "per-expert routed rows counted by the last step (moe counts)"
    return rep


def _padding(su, bm=256):
    import numpy as np

    counts = su.plan.counts.cpu().numpy().astype(np.int64)
    R = int(counts.sum())
    padded = int((-(-counts // bm) * bm).sum())
    return {"tile_rows": bm, "routed_rows": R, "padded_rows": padded,
            "waste_rows": padded - R, "waste_frac": round((padded - R) / max(padded, 1), 4),
            "experts_with_rows": int((counts > 0).sum())}


def _stats(v):
    v = sorted(v)
    n = len(v)
    pick = lambda q: v[min(n - 1, max(0, int(round(q * (n - 1)))))]
    return {"mean_us": round(1e3 * sum(v) / n, 2), "median_us": round(1e3 * pick(0.5), 2),
            "p10_us": round(1e3 * pick(0.1), 2), "p90_us": round(1e3 * pick(0.9), 2)}


def _attainable(dev):
    """A plain copy kernel and a bf16 MFMA loop, timed with events."""
    import torch

    import paper_2601_14327_amd as laep
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty(n, dtype=torch.uint8, device=dev)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    laep.laep_calib_copy(src, dst)
    times = []
    for _ in range(10):
        s.record()
        laep.laep_calib_copy(src, dst)
        e.record()
        torch.cuda.synchronize()
        times.append(s.elapsed_time(e))
    copy_gbs = 2 * n / (sorted(times)[len(times) // 2] * 1e-3) / 1e9
    del src, dst
    wg, iters = 256 * 4, 4096
    out = torch.empty(wg * 512, dtype=torch.float32, device=dev)
    laep.laep_calib_mfma(wg, 64, out)
    s.record()
    laep.laep_calib_mfma(wg, iters, out)
    e.record()
    torch.cuda.synchronize()
    tf = wg * 8 * iters * 8 * 32768 / (s.elapsed_time(e) * 1e-3) / 1e12
    return {"copy_GBs": round(copy_gbs, 1), "mfma_bf16_TFLOPs": round(tf, 1),
            "copy_frac_of_peak": round(copy_gbs / PEAK_HBM_GBS, 3),
            "mfma_frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 3)}


def library_ref(args):
    """The grouped FFN on 64 equal experts of 1024 rows (no ragged tiles, the
    `balanced` layer's d and f), beside the platform BLAS (hipBLASLt, through
    torch.matmul) on the same two products as dense matrices of the same
    flops: [R, d] x [d, 2f] and [R, f] x [f, d]; and the grouped backward
    beside its four products as bf16 batched GEMMs over the experts
    (torch.bmm; the library writes the weight gradients in fp32, the batched
    GEMMs in bf16).  Context for the GEMM core, not the metric: the library's
    products fuse SwiGLU and its backward, the vendor's do neither."""
    import torch

    import paper_2601_14327_amd as laep
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    E, rows, d, f = 64, 1024, 2048, 1024
    R = E * rows
    g = torch.Generator(device=dev).manual_seed(7)
    bf = torch.bfloat16
    x = torch.randn(R, d, device=dev, generator=g).to(bf)
    wgu = (torch.randn(E, 2 * f, d, device=dev, generator=g) * d ** -0.5).to(bf)
    wd = (torch.randn(E, d, f, device=dev, generator=g) * f ** -0.5).to(bf)
    offsets = torch.arange(0, R + 1, rows, dtype=torch.int32, device=dev)
    y = torch.empty(R, d, dtype=bf, device=dev)
    # dense operands, [K, N] contiguous (no transposed views)
    b1 = wgu[0].t().contiguous()
    h = torch.randn(R, f, device=dev, generator=g).to(bf)
    b2 = wd[0].t().contiguous()
    c1 = torch.empty(R, 2 * f, dtype=bf, device=dev)
    c2 = torch.empty(R, d, dtype=bf, device=dev)
    # backward: the library's call (dY given, H_b from act_save) beside the four
    # products as bf16 batched GEMMs over the experts (torch.bmm, every operand
    # contiguous: the transposed ones are copies, never views)
    _, act = laep.moe_grouped_ffn_fwd(x, wgu, wd, offsets, save_act=True)
    dy = torch.randn(R, d, device=dev, generator=g).to(bf)
    dx = torch.empty_like(x)
    dwgu = torch.empty(wgu.shape, dtype=torch.float32, device=dev)
    dwd = torch.empty(wd.shape, dtype=torch.float32, device=dev)
    ws_b = torch.empty(laep.workspace_bytes(laep.LAEP_CALL_FFN_BWD, R, 1, E, d, f),
                       dtype=torch.uint8, device=dev)
    dy3 = dy.view(E, rows, d)
    da3 = torch.randn(E, rows, 2 * f, device=dev, generator=g).to(bf)
    x3, h3 = x.view(E, rows, d), h.view(E, rows, f)
    dy3t = dy3.transpose(1, 2).contiguous()
    da3t = da3.transpose(1, 2).contiguous()
    o_dh = torch.empty(E, rows, f, dtype=bf, device=dev)
    o_dx = torch.empty(E, rows, d, dtype=bf, device=dev)
    o_dwd = torch.empty(E, d, f, dtype=bf, device=dev)
    o_dwgu = torch.empty(E, 2 * f, d, dtype=bf, device=dev)
    calls = {
        "laep_grouped_ffn_fwd": lambda: laep.moe_grouped_ffn_fwd(x, wgu, wd, offsets,
                                                                 save_act=False, y_perm=y),
        "torch_matmul_gate_up": lambda: torch.matmul(x, b1, out=c1),
        "torch_matmul_down": lambda: torch.matmul(h, b2, out=c2),
        "laep_grouped_ffn_bwd": lambda: laep.moe_grouped_ffn_bwd(
            dy, x, act, wgu, wd, offsets, dw_gate_up=dwgu, dw_down=dwd, ws=ws_b, dx_perm=dx),
        "torch_bmm_dgrad_dH": lambda: torch.bmm(dy3, wd, out=o_dh),
        "torch_bmm_dgrad_dX": lambda: torch.bmm(da3, wgu, out=o_dx),
        "torch_bmm_wgrad_dWd": lambda: torch.bmm(dy3t, h3, out=o_dwd),
        "torch_bmm_wgrad_dWgu": lambda: torch.bmm(da3t, x3, out=o_dwgu),
    }
    # the weight gradients with fp32 outputs, as the library writes them (where
    # this PyTorch build offers bf16 x bf16 -> fp32 batched products)
    try:
        torch.bmm(dy3t[:1], h3[:1], out_dtype=torch.float32)
        calls["torch_bmm_wgrad_dWd_f32out"] = lambda: torch.bmm(dy3t, h3, out_dtype=torch.float32)
        calls["torch_bmm_wgrad_dWgu_f32out"] = lambda: torch.bmm(da3t, x3, out_dtype=torch.float32)
    except (RuntimeError, NotImplementedError, TypeError):
        pass
    flops = {"torch_bmm_wgrad_dWd_f32out": 2.0 * R * d * f,
             "torch_bmm_wgrad_dWgu_f32out": 4.0 * R * d * f,
             "laep_grouped_ffn_fwd": 6.0 * R * d * f, "torch_matmul_gate_up": 4.0 * R * d * f,
             "torch_matmul_down": 2.0 * R * d * f, "laep_grouped_ffn_bwd": 12.0 * R * d * f,
             "torch_bmm_dgrad_dH": 2.0 * R * d * f, "torch_bmm_dgrad_dX": 4.0 * R * d * f,
             "torch_bmm_wgrad_dWd": 2.0 * R * d * f, "torch_bmm_wgrad_dWgu": 4.0 * R * d * f}
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 3.0:   # clocks up
        for fn in calls.values():
            fn()
        torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {}
    for name, fn in calls.items():
        ts = []
        for _ in range(args.steps):
            s.record()
            fn()
            e.record()
            torch.cuda.synchronize()
            ts.append(s.elapsed_time(e) * 1e3)
        med = sorted(ts)[len(ts) // 2]
        out[name] = {"median_us": round(med, 1),
                     "TFLOPs": round(flops[name] / (med * 1e-6) / 1e12, 1)}
    dense_us = out["torch_matmul_gate_up"]["median_us"] + out["torch_matmul_down"]["median_us"]
    out["torch_matmul_both"] = {"median_us": round(dense_us, 1),
                                "TFLOPs": round(6.0 * R * d * f / (dense_us * 1e-6) / 1e12, 1)}
    bmm_us = sum(out[k]["median_us"] for k in ("torch_bmm_dgrad_dH", "torch_bmm_dgrad_dX",
                                                "torch_bmm_wgrad_dWd", "torch_bmm_wgrad_dWgu"))
    out["torch_bmm_backward_all"] = {"median_us": round(bmm_us, 1),
                                     "TFLOPs": round(12.0 * R * d * f / (bmm_us * 1e-6) / 1e12, 1)}
    print(json.dumps({"library_ref": out, "shape": {"experts": E, "rows_per_expert": rows,
                                                    "d_model": d, "d_ff": f}}), flush=True)


def _supplementary(w, su, dev, reps=20):
    """Latency-bound calls at other sizes: moe_expert_counts over T x {1, 8, 64}
    (random distinct expert ids, the workload's E and k), and route followed
    by counts as one event pair (the two calls the routing front end makes)."""
    import numpy as np
    import torch

    L = su.laep
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(fn):
        fn()
        ts = []
        for _ in range(reps):
            s.record()
            fn()
            e.record()
            torch.cuda.synchronize()
            ts.append(s.elapsed_time(e) * 1e3)
        return round(sorted(ts)[len(ts) // 2], 2)

    rng = np.random.default_rng(0)
    sweep = []
    for mult in (1, 8, 64):
        T = w.T * mult
        ids = np.argsort(rng.random((T, su.E)), axis=1)[:, :w.k].astype(np.int32)
        idx = torch.from_numpy(ids).to(dev)
        ws = torch.empty(max(1, L.workspace_bytes(1, T, w.k, su.E)), dtype=torch.uint8,
                         device=dev)
        bufs = dict(counts=torch.empty(su.E, dtype=torch.int32, device=dev),
                    offsets=torch.empty(su.E + 1, dtype=torch.int32, device=dev),
                    dest_row=torch.empty(T * w.k, dtype=torch.int32, device=dev))
        us = timed(lambda: L.moe_expert_counts(idx, su.E, ws=ws, **bufs))
        nbytes = T * w.k * 4 * 2 + 2 * (su.E + 1) * 4
        sweep.append({"tokens": T, "median_us": us, "GBs": round(nbytes / (us * 1e-6) / 1e9, 1)})
        del idx, ws, bufs
    out = {"counts_T_sweep": sweep}
    if w.routed:
        p, x = su.plan, su.xs[0]
        out["route_us"] = timed(lambda: L.moe_route(x, su.wr, w.k, bias=su.bias, renorm=w.renorm,
                                                    topk_idx=p.topk_idx, topk_gate=p.topk_gate))
        out["counts_us"] = timed(p.count)
        out["route_then_counts_us"] = timed(lambda: (
            L.moe_route(x, su.wr, w.k, bias=su.bias, renorm=w.renorm, topk_idx=p.topk_idx,
                        topk_gate=p.topk_gate), p.count()))
        out["route_count_fused_us"] = timed(lambda: p.route_count(x, su.wr, bias=su.bias,
                                                                  renorm=w.renorm))
    return out


def _traffic(name, sources):
    """HBM bytes per call from the committed counter summary, if still valid."""
    path = os.path.join(PROFILES, f"{name}_traffic.md")
    if not os.path.exists(path):
        return None, "no counter summary"
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), flags=re.S)
    if not m:
        return None, "summary has no data block"
    rec = json.loads(m.group(1))
    if rec.get("kernel_sources_sha256") != sources_sha(sources):
        return None, "kernel changed since the counters were taken"
    return rec["traffic_bytes_per_call"], os.path.relpath(path, ROOT)


# ---------------------------------------------------------------------------------------
# profiling helpers
# ---------------------------------------------------------------------------------------
def profile_target(args):
    import torch

    from workloads import WORKLOADS
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.profile_target == "copy":
        import paper_2601_14327_amd as laep
        src = torch.empty(COPY_CALIB_BYTES, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty(COPY_CALIB_BYTES, dtype=torch.uint8, device=dev)
        for _ in range(PROFILE_CALLS):
            laep.laep_calib_copy(src, dst)
        torch.cuda.synchronize()
        print(f"profile target: laep_calib_copy of {COPY_CALIB_BYTES} bytes x {PROFILE_CALLS}",
              flush=True)
        return
    import paper_2601_14327_amd as laep
    su = Setup(WORKLOADS[args.workload], dev)
    calls = dict(su.calls(0))
    for name, fn in su.calls(0):       # one full step prepares every input
        fn()
    # marker dispatch: the counters of every dispatch after it belong to the target
    marker = torch.empty(512, dtype=torch.float32, device=dev)
    laep.laep_calib_mfma(1, 1, marker)
    if args.profile_target == "route_feed":
        # the router's feed bound: moe_route_count beside a blocked read of the
        # same x bytes in the router's launch shape (32 token rows per
        # 512-thread workgroup), both over the rotating x sets, after a settle
        w = su.w
        block = 32 * w.d_model * 2
        out = torch.empty(w.T // 32 * 512, dtype=torch.float32, device=dev)
        _settle(su)
        n = su.n_sets
        for i in range(200):
            dict(su.calls(i))["route_count"]()
            laep.laep_calib_read(su.xs[(i + n // 2) % n], block, out)
        torch.cuda.synchronize()
        print(f"profile target: route_count and laep_calib_read ({block} B blocks) x 200 on "
              f"{args.workload}", flush=True)
        return
    for _ in range(PROFILE_CALLS):
        calls[args.profile_target]()
    torch.cuda.synchronize()
    print(f"profile target: {args.profile_target} x {PROFILE_CALLS} on {args.workload}",
          flush=True)


def _read_counters(d):
    """[(dispatch id, kernel, counter, value)] from rocprofv3 counter CSVs."""
    import csv
    out = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], r["Counter_Name"],
                        float(r["Counter_Value"])))
    return out


def _per_call(d, counter):
    """Counter total per target call (dispatches after the marker) and per kernel."""
    rows = [r for r in _read_counters(d) if r[2] == counter]
    mark = max(r[0] for r in rows if "mfma_loop_kernel" in r[1])
    tot, per_k = 0.0, {}
    for did, k, _, v in rows:
        if did > mark:
            tot += v
            name = re.sub(r"\(.*", "", k.replace("(anonymous namespace)::", ""))
            per_k[name] = per_k.get(name, 0.0) + v / PROFILE_CALLS
    return tot / PROFILE_CALLS, per_k


def _per_copy(d, counter):
    vals = [r[3] for r in _read_counters(d) if r[2] == counter and "copy_kernel" in r[1]]
    return sum(vals) / len(vals)


def summarize_pmc(args):
    """Traffic summary of one call from four counter runs: DIR/call_fetch,
    DIR/call_write (the call, PROFILE_CALLS times after a marker dispatch),
    DIR/copy_fetch, DIR/copy_write (the calibration copy of COPY_CALIB_BYTES)."""
    d = args.summarize_pmc
    call = args.profile_call
    srcs = FFN_FWD_SOURCES if call == "ffn_fwd" else FFN_BWD_SOURCES
    copy_f = _per_copy(os.path.join(d, "copy_fetch"), "FETCH_SIZE")
    copy_w = _per_copy(os.path.join(d, "copy_write"), "WRITE_SIZE")
    k_fetch = COPY_CALIB_BYTES / copy_f     # bytes per counter unit, reads
    k_write = COPY_CALIB_BYTES / copy_w     # bytes per counter unit, writes
    ff, ffk = _per_call(os.path.join(d, "call_fetch"), "FETCH_SIZE")
    fw, fwk = _per_call(os.path.join(d, "call_write"), "WRITE_SIZE")
    fetch, write = ff * k_fetch, fw * k_write
    rec = {"call": call, "workload": args.workload,
           "kernel_sources_sha256": sources_sha(srcs),
           "copy_calibration": {"bytes_read_and_written": COPY_CALIB_BYTES,
                                "FETCH_SIZE": copy_f, "WRITE_SIZE": copy_w,
                                "bytes_per_fetch_unit": k_fetch, "bytes_per_write_unit": k_write},
           "FETCH_SIZE_per_call_by_kernel": ffk, "WRITE_SIZE_per_call_by_kernel": fwk,
           "fetch_bytes_per_call": fetch, "write_bytes_per_call": write,
           "traffic_bytes_per_call": fetch + write}
    cmd = args.command_note or ""
    text = (f"# HBM traffic of `{call}` on workload `{args.workload}`\n\n"
            f"rocprofv3 counters FETCH_SIZE and WRITE_SIZE (one --pmc pass each), summed over "
            f"the call's dispatches, each scaled by what the same counter reads for the "
            f"library's plain copy kernel moving {COPY_CALIB_BYTES} bytes.\n\n"
            f"- fetched: {fetch / 1e6:.1f} MB per call\n- written: {write / 1e6:.1f} MB per call\n"
            f"- calibration: {k_fetch:.1f} bytes per FETCH_SIZE unit, {k_write:.1f} bytes per "
            f"WRITE_SIZE unit\n\nCommands:\n\n```\n{cmd}\n```\n\n```json\n"
            f"{json.dumps(rec, indent=1)}\n```\n")
    with open(args.out, "w") as fh:
        fh.write(text)
    print(text)


def summarize_counters(args):
    """Per-kernel averages per dispatch of every counter in the --pmc runs under
    DIR (one subdirectory per pass, each of the call PROFILE_CALLS times after
    the marker dispatch), and the ratios derived from them:
      clock        GRBM_GUI_ACTIVE / dispatch duration (the GPU clock while busy)
      mfma_busy    SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x SQ_BUSY_CU_CYCLES): share of
                   the CUs' busy cycles in which a SIMD's matrix core was busy
      mfma_cycles  SQ_VALU_MFMA_BUSY_CYCLES / SQ_INSTS_MFMA (cycles per MFMA)
      lds_conflict SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE
      wait_any, wait_inst, wait_lds  SQ_WAIT_ANY, SQ_WAIT_INST_ANY,
                   SQ_WAIT_INST_LDS over SQ_WAVE_CYCLES (shares of wave time)"""
    import csv
    d = args.summarize_counters
    per = {}      # kernel -> counter -> [values]
    dur = {}      # kernel -> [ns]
    for sub_dir in sorted(glob.glob(os.path.join(d, "*"))):
        rows = []
        for f in glob.glob(os.path.join(sub_dir, "**", "*counter_collection.csv"), recursive=True):
            rows += list(csv.DictReader(open(f)))
        if not rows:
            continue
        mark = max(int(r["Dispatch_Id"]) for r in rows if "mfma_loop_kernel" in r["Kernel_Name"])
        seen = set()
        for r in rows:
            did = int(r["Dispatch_Id"])
            if did <= mark:
                continue
            k = re.sub(r"\(.*", "", r["Kernel_Name"].replace("(anonymous namespace)::", ""))
            per.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            if (sub_dir, did) not in seen:
                seen.add((sub_dir, did))
                dur.setdefault(k, []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    rec = {"call": args.profile_call, "workload": args.workload, "kernels": {}}
    lines = [f"# Counters of `{args.profile_call}` on workload `{args.workload}`\n",
             "rocprofv3 --pmc passes (at most 8 SQ and 2 GRBM counters each), averaged per "
             "dispatch over the call's dispatches. Ratios: clock = GRBM_GUI_ACTIVE / duration; "
             "mfma_busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 x SQ_BUSY_CU_CYCLES); mfma_cycles = "
             "SQ_VALU_MFMA_BUSY_CYCLES / SQ_INSTS_MFMA; lds_conflict = SQ_LDS_BANK_CONFLICT / "
             "SQ_LDS_IDX_ACTIVE; wait_* = SQ_WAIT_ANY, SQ_WAIT_INST_ANY, SQ_WAIT_INST_LDS over "
             "SQ_WAVE_CYCLES. Durations are those of the counter runs.\n",
             "Commands:\n", f"```\n{args.command_note or ''}\n```\n"]
    for k, cs in per.items():
        avg = {c: sum(v) / len(v) for c, v in cs.items()}
        dns = sum(dur[k]) / len(dur[k])
        g = lambda c: avg.get(c)
        ratio = lambda a, b, f=1.0: (g(a) / (f * g(b))) if g(a) is not None and g(b) else None
        der = {"duration_us": dns / 1e3,
               "clock_ghz": (g("GRBM_GUI_ACTIVE") / dns) if g("GRBM_GUI_ACTIVE") else None,
               "mfma_busy": ratio("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CU_CYCLES", 4.0),
               "mfma_cycles": ratio("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_MFMA"),
               "lds_conflict": ratio("SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE"),
               "wait_any": ratio("SQ_WAIT_ANY", "SQ_WAVE_CYCLES"),
               "wait_inst": ratio("SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES"),
               "wait_lds": ratio("SQ_WAIT_INST_LDS", "SQ_WAVE_CYCLES")}
        rec["kernels"][k] = {"counters": avg, "derived": der}
        lines.append(f"## `{k[:110]}`\n")
        lines.append("| derived | value |\n|---|---:|")
        for n, v in der.items():
            lines.append(f"| {n} | {'' if v is None else f'{v:.4g}'} |")
        lines.append("\n| counter | per dispatch |\n|---|---:|")
        for c in sorted(avg):
            lines.append(f"| {c} | {avg[c]:.6g} |")
        lines.append("")
    text = "\n".join(lines) + f"\n```json\n{json.dumps(rec, indent=1)}\n```\n"
    with open(args.out, "w") as fh:
        fh.write(text)
    print(text)


def summarize_trace(args):
    import csv
    f = glob.glob(os.path.join(args.summarize_trace, "**", "*kernel_stats.csv"), recursive=True)[0]
    rows = list(csv.DictReader(open(f)))
    lines = [f"# Kernel time: {args.workload}\n", "rocprofv3 --kernel-trace --stats.\n",
             "Commands:\n", f"```\n{args.command_note or ''}\n```\n",
             "| kernel | calls | average (us) | min (us) | max (us) | share |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in rows:
        name = re.sub(r"\(.*", "", r["Name"].replace("(anonymous namespace)::", ""))
        lines.append(f"| `{name[:110]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.2f}% |")
    lines += _feed_loop_lines(args)
    if args.append_log:   # the run's own result line
        last = [ln for ln in open(args.append_log).read().splitlines() if ln.startswith("{")][-1]
        lines += ["", "## Result line of the same command (HIP events, medians)", "",
                  "```json", json.dumps(json.loads(last), indent=1), "```"]
    text = "\n".join(lines) + "\n"
    with open(args.out, "w") as fh:
        fh.write(text)
    print(text)


def _feed_loop_lines(args):
    """For a route_feed trace: each blocked read beside the router launch and
    the counting launch issued just before it, and the read's rate on x."""
    import csv
    import statistics
    f = glob.glob(os.path.join(args.summarize_trace, "**", "*kernel_trace.csv"), recursive=True)
    if not f:
        return []
    rows = sorted(csv.DictReader(open(f[0])), key=lambda r: int(r["Start_Timestamp"]))
    reads = [i for i, r in enumerate(rows) if "read_kernel" in r["Kernel_Name"]]
    if not reads:
        return []
    from workloads import WORKLOADS
    w = WORKLOADS[args.workload]
    x_bytes = w.T * w.d_model * 2

    def dur(r):
        return (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3

    def before(i, key):
        for j in range(i - 1, max(-1, i - 4), -1):
            if key in rows[j]["Kernel_Name"]:
                return dur(rows[j])
        raise ValueError(f"no {key} dispatch before read dispatch {i}")

    series = [("`read_kernel` (x bytes only)", [dur(rows[i]) for i in reads]),
              ("`route_kernel`", [before(i, "route_kernel") for i in reads]),
              ("`count_scan_scatter_kernel`", [before(i, "count_scan_scatter") for i in reads])]
    g = rows[reads[0]]
    rd = statistics.mean(series[0][1])
    ro = statistics.mean(series[1][1])
    out = ["", "## Feed loop",
           f"Each of the {len(reads)} iterations: `moe_route_count` on one x set, then "
           f"`laep_calib_read` on another ({int(g['Grid_Size_X']) // int(g['Workgroup_Size_X'])} "
           f"workgroups of {g['Workgroup_Size_X']} threads, 32 token rows each: the router's "
           f"launch shape), x {x_bytes / 1e6:.1f} MB.\n",
           "| dispatch | calls | average (us) | median (us) | min (us) | max (us) |",
           "|---|---:|---:|---:|---:|---:|"]
    for name, v in series:
        out.append(f"| {name} | {len(v)} | {statistics.mean(v):.2f} | {statistics.median(v):.2f} "
                   f"| {min(v):.2f} | {max(v):.2f} |")
    out += ["", f"Read rate on x: {x_bytes / rd / 1e3:.0f} GB/s. The router takes "
                f"{ro / rd:.2f}x the read ({ro - rd:.2f} us above its feed bound)."]
    return out


# ---------------------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="balanced")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-attainable", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--profile-target", choices=["ffn_fwd", "ffn_bwd", "copy", "route_count",
                                                 "permute", "combine", "counts", "route_feed"])
    ap.add_argument("--library-ref", action="store_true")
    ap.add_argument("--summarize-pmc")
    ap.add_argument("--summarize-trace")
    ap.add_argument("--summarize-counters")
    ap.add_argument("--profile-call", default="ffn_fwd")
    ap.add_argument("--command-note")
    ap.add_argument("--append-log")
    ap.add_argument("--out")
    args = ap.parse_args()
    if args.summarize_pmc:
        return summarize_pmc(args)
    if args.summarize_trace:
        return summarize_trace(args)
    if args.summarize_counters:
        return summarize_counters(args)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the library has no "
              f"multi-GPU expert-parallel path.", file=sys.stderr)
        sys.exit(2)
    if args.profile_target:
        return profile_target(args)
    if args.library_ref:
        return library_ref(args)

    import torch

    from workloads import WORKLOADS

    w = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    su = Setup(w, dev)
    stream = torch.cuda.current_stream(dev)

    settle_steps, settle_s = _settle(su)
    for i in range(args.warmup):
        for _, fn in su.calls(i):
            fn()
    torch.cuda.synchronize()
    names = [n for n, _ in su.calls(0)]
    dom = "ffn_bwd" if w.backward else "ffn_fwd"   # the dominant call
    # Timed region: wall clock over the steps gives `value`; HIP events on the
    # calls' stream bracket the dominant call only (an event marker between
    # two calls costs the GPU about 5 us, so events around every call would
    # inflate the step time).
    dom_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        for n, fn in su.calls(i):
            if n == dom:
                dom_ev[i][0].record(stream)
                fn()
                dom_ev[i][1].record(stream)
            else:
                fn()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = wall * 1e3 / args.steps

    # Per-call breakdown: the same steps again, with events around every call
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in names] for _ in range(args.steps)]
    for i in range(args.steps):
        for j, (_, fn) in enumerate(su.calls(i)):
            ev[i][j][0].record(stream)
            fn()
            ev[i][j][1].record(stream)
    torch.cuda.synchronize()

    # warm: the same input set every step (x can stay in the caches between
    # steps); reported beside the primary, rotating-input number
    for _, fn in su.calls(0):
        fn()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(args.steps):
        for _, fn in su.calls(0):
            fn()
    torch.cuda.synchronize()
    warm_ms = (time.perf_counter() - t1) * 1e3 / args.steps

    placement = _placement(su)
    padding = _padding(su)
    by, fl = su.algorithmic()
    breakdown = {}
    for j, n in enumerate(names):
        st = _stats([ev[i][j][0].elapsed_time(ev[i][j][1]) for i in range(args.steps)])
        if n in by:
            st["GBs"] = round(by[n] / (st["mean_us"] * 1e-6) / 1e9, 1)
            st["frac_hbm_peak"] = round(st["GBs"] / PEAK_HBM_GBS, 3)
        if n in fl:
            st["TFLOPs"] = round(fl[n] / (st["mean_us"] * 1e-6) / 1e12, 1)
            st["frac_mfma_peak"] = round(st["TFLOPs"] / PEAK_BF16_TFLOPS, 3)
        breakdown[n] = st

    # the dominant call (the grouped FFN, backward when the step has one), timed
    # inside the timed region
    dom_st = _stats([dom_ev[i][0].elapsed_time(dom_ev[i][1]) for i in range(args.steps)])
    dom_us = dom_st["mean_us"]
    achieved = fl[dom] / (dom_us * 1e-6) / 1e12
    traffic, traffic_src = _traffic(f"{dom}_{w.name}",
                                    FFN_BWD_SOURCES if dom == "ffn_bwd" else FFN_FWD_SOURCES)
    attain = None if args.no_attainable else _attainable(dev)
    supp = None if args.no_attainable else _supplementary(w, su, dev)
    cpu = None if args.no_cpu_baseline else _cpu_baseline(w, su.c, args.cpu_budget, su.keep)

    unit = "tokens/s" if w.routed else "rows/s"
    metric = ("MoE-layer tokens/s at 1 GPU; grouped-GEMM TFLOP/s as % bf16 MFMA peak"
              if w.routed else "MoE expert-shard routed rows/s at 1 GPU (fwd" +
              ("+bwd" if w.backward else "") + ")")
    line = {
        "metric": metric,
        "value": w.T / (ms * 1e-3),
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
        "config": {"workload": f"{w.name}: T={w.T} d_model={w.d_model} E={w.E}"
                               + (f" (pruned to {su.E})" if su.E != w.E else "") + f" k={w.k} "
                               f"d_ff={w.d_ff} bf16" + (" fwd+bwd" if w.backward else " fwd"),
                   "tokens": w.T, "experts": w.E, "top_k": w.k, "d_model": w.d_model,
                   "d_ff": w.d_ff},
        "roofline": {"bound": "mfma",
                     "kernel": f"{dom}: grouped SwiGLU FFN "
                               f"({'dgrad + wgrad GEMMs' if dom == 'ffn_bwd' else 'gate/up + down GEMMs'}"
                               f" and tile-table build), one C-ABI call",
                     "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
                     "traffic_source": traffic_src,
                     "algorithmic_flops_per_call": fl[dom], "mean_call_us": dom_us,
                     "call_us_stats": dom_st},
        "cpu_baseline": cpu,
        "attainable": attain,
        "warm": {"ms_per_step": warm_ms, "value": w.T / (warm_ms * 1e-3),
                 "note": "same input set every step"},
        "pruning": su.pruning,
        "settle": {"steps": settle_steps, "seconds": settle_s},
        "placement": placement,
        "padding": padding,
        "supplementary": supp,
        "breakdown": breakdown,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
