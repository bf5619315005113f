"""Seeded synthetic inputs for the MoE-layer workloads.

This module only draws random numbers.  It holds none of the layer's
arithmetic (no routing, no FFN, no rounding points of the method), so both
the CPU oracle and the GPU path may read from it.

Every array is returned as a NumPy float32 array.  For bf16 workloads the
values are drawn in float32 and rounded to bf16 (round-to-nearest-even, done
by torch's CPU conversion), so the float32 array holds bf16-exact values.
The GPU side converts them to ``torch.bfloat16`` without loss; the oracle
widens them to float64 without loss.

The workloads follow the stable-phase MoE-layer shapes used to measure the
LAEP hot path:

* ``tiny``      T=256, d=128, E=8, k=2, f=256, fp32, plain top-2 of a softmax
* ``balanced``  T=8192, d=2048, E=64, k=8, f=1024, bf16, renormalised top-8
* ``skewed``    as ``balanced`` plus a per-expert router bias ~N(0, 2)
* ``skewed_mild`` as ``balanced`` plus a per-expert router bias ~N(0, 0.5)
* ``shard``     one device's expert shard: 16 experts, d=4096, f=2048,
                32768 routed rows whose expert ids follow Zipf(s=1.1)
* ``shard_bwd`` ``shard`` plus an upstream gradient ~N(0, 1)
* ``balanced_bwd`` ``balanced`` plus an upstream gradient (routed training step)
* ``mild_pruned`` ``skewed_mild``'s draws; the layer after Algorithm 1 has
                removed its pruned experts

The paper's own pre-training corpus and trained weights are not available;
these seeded inputs stand in for its stable-phase expert loads (a few
experts carry most tokens, the least-loaded ones orders of magnitude fewer).
"""
from __future__ import annotations

import dataclasses
import functools
import math
from typing import Dict, Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    T: int            # tokens (for the shard workloads: routed rows, k = 1)
    d_model: int
    E: int
    k: int
    d_ff: int
    dtype: str        # "f32" or "bf16"
    renorm: bool      # renormalise the gates over the selected k
    bias_std: float = 0.0       # per-expert router bias ~N(0, bias_std); 0 = none
    routed: bool = True         # False: expert ids are given (Zipf), no router
    zipf_s: float = 0.0
    backward: bool = False
    prune_beta: Optional[float] = None
    prune_alpha: float = math.inf
    weight_std: float = 0.02
    # > 0: before the timed steps, Algorithm 1 runs over a window of this
    # many routed batches and the pruned experts are removed (compact layer)
    prune_window: int = 0

    @property
    def rows(self) -> int:
        return self.T * self.k


WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("tiny", 1001, T=256, d_model=128, E=8, k=2, d_ff=256,
                 dtype="f32", renorm=False),
        Workload("balanced", 1002, T=8192, d_model=2048, E=64, k=8, d_ff=1024,
                 dtype="bf16", renorm=True),
        Workload("skewed", 1003, T=8192, d_model=2048, E=64, k=8, d_ff=1024,
                 dtype="bf16", renorm=True, bias_std=2.0, prune_beta=0.05),
        Workload("skewed_mild", 1013, T=8192, d_model=2048, E=64, k=8,
                 d_ff=1024, dtype="bf16", renorm=True, bias_std=0.5,
                 prune_beta=0.05),
        Workload("shard", 1004, T=32768, d_model=4096, E=16, k=1, d_ff=2048,
                 dtype="bf16", renorm=False, routed=False, zipf_s=1.1),
        Workload("shard_bwd", 1005, T=32768, d_model=4096, E=16, k=1,
                 d_ff=2048, dtype="bf16", renorm=False, routed=False,
                 zipf_s=1.1, backward=True),
        # steady state after pruning: the skewed_mild generator, Algorithm 1 over
        # a window of 3 batches with a middle layer's setting of the paper's
        # pre-training run (alpha = 0.4, beta = 0.1), pruned experts removed
        Workload("mild_pruned", 1013, T=8192, d_model=2048, E=64, k=8, d_ff=1024,
                 dtype="bf16", renorm=True, bias_std=0.5, prune_beta=0.1,
                 prune_alpha=0.4, prune_window=3),
        # routed pre-training step: balanced forward, then backward through the
        # combine, the expert FFN, the dispatch and the router
        Workload("balanced_bwd", 1006, T=8192, d_model=2048, E=64, k=8, d_ff=1024,
                 dtype="bf16", renorm=True, backward=True),
    ]
}


def to_bf16_exact(a: np.ndarray) -> np.ndarray:
    """Round float32 draws to bf16 (RNE) and return them as float32."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _draw(rng: np.random.Generator, shape, std: float, bf16: bool) -> np.ndarray:
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return to_bf16_exact(a) if bf16 else a


def zipf_expert_ids(rng: np.random.Generator, rows: int, E: int, s: float):
    """Expert id per row: rank r (1..E) drawn with p_r ~ r^-s, ranks mapped
    to experts by a seeded permutation."""
    ranks = np.arange(1, E + 1, dtype=np.float64)
    p = ranks ** (-s)
    p /= p.sum()
    rank_of_row = rng.choice(E, size=rows, p=p)
    expert_of_rank = rng.permutation(E)
    return expert_of_rank[rank_of_row].astype(np.int32)


def generate(w: Workload, T: Optional[int] = None, seed: Optional[int] = None,
             with_weights: bool = True) -> Dict[str, np.ndarray]:
    """Draw one workload's inputs.  ``T`` overrides the token / row count
    (for reduced-size parity cases); ``seed`` overrides the seed.

    Draw order: x, W_r, bias, W_gu, W_d, then (given-routing workloads) the
    expert ids and gates, then (backward) dout.
    """
    T = w.T if T is None else T
    rng = np.random.default_rng(w.seed if seed is None else seed)
    bf16 = w.dtype == "bf16"
    out: Dict[str, np.ndarray] = {}
    out["x"] = _draw(rng, (T, w.d_model), 1.0, bf16)
    if w.routed:
        out["w_router"] = _draw(rng, (w.E, w.d_model), w.weight_std, bf16)
        if w.bias_std > 0:
            out["bias"] = rng.standard_normal(w.E, dtype=np.float32) * np.float32(w.bias_std)
    if with_weights:
        out["w_gate_up"] = _draw(rng, (w.E, 2 * w.d_ff, w.d_model), w.weight_std, bf16)
        out["w_down"] = _draw(rng, (w.E, w.d_model, w.d_ff), w.weight_std, bf16)
    if not w.routed:
        out["topk_idx"] = zipf_expert_ids(rng, T, w.E, w.zipf_s).reshape(T, 1)
        out["topk_gate"] = rng.uniform(0.05, 1.0, size=(T, 1)).astype(np.float32)
    if w.backward:
        out["dout"] = _draw(rng, (T, w.d_model), 1.0, bf16)
    return out


@functools.lru_cache(maxsize=4)
def cached(name: str, T: Optional[int] = None, seed: Optional[int] = None):
    """In-process cache of :func:`generate` (arrays must not be mutated)."""
    arrs = generate(WORKLOADS[name], T=T, seed=seed)
    for a in arrs.values():
        a.setflags(write=False)
    return arrs


def random_case(seed: int, T: int, d_model: int, E: int, k: int, d_ff: int,
                dtype: str = "bf16", bias_std: float = 0.0,
                weight_std: float = 0.02) -> Dict[str, np.ndarray]:
    """A small seeded case of arbitrary shape (fuzz and edge-case tests)."""
    w = Workload("case", seed, T=T, d_model=d_model, E=E, k=k, d_ff=d_ff,
                 dtype=dtype, renorm=True, bias_std=bias_std,
                 weight_std=weight_std)
    return generate(w)
