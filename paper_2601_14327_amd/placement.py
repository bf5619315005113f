"""Placement report of expert rearrangement (Section 3.3; Appendix
Algorithm 2): how the greedy placement of `laep_rearrange` balances measured
per-expert loads over device groups, next to the placement without
rearrangement.

Host-side reporting, not on the hot path.  The greedy placement itself comes
from the C ABI (`laep_rearrange`); this module only summarises it:

  greedy       laep_rearrange's groups (descending loads, least-loaded group
               with room, capacity ceil(n / n_groups))
  contiguous   experts in index order, ceil(n / n_groups) per group: expert e
               on group e // capacity, the placement an expert-parallel
               layout has before any rearrangement
  lower_bound  max(total / n_groups, largest load): no placement's largest
               group can be below it
  optimum      for n <= `exact_max_n`, the smallest possible largest group
               sum under the same capacity, found by branch and bound

The largest group sum is what sets the step time of an expert-parallel layer
(every device waits for the most loaded one); `max_over_mean` is that
straggler factor.
"""
from __future__ import annotations

import math

import numpy as np

from .api import laep_rearrange


def _summary(sums):
    sums = np.asarray(sums, dtype=np.float64)
    mean = float(sums.mean()) if sums.size else 0.0
    mx = float(sums.max()) if sums.size else 0.0
    return {"group_sums": [float(v) for v in sums], "max": mx, "mean": mean,
            "max_over_mean": (mx / mean) if mean > 0 else None}


def contiguous_sums(loads, n_groups: int):
    """Group sums of the placement without rearrangement: expert e on group
    e // ceil(n / n_groups)."""
    loads = np.asarray(loads, dtype=np.float64)
    n = loads.shape[0]
    cap = -(-n // n_groups) if n else 1
    sums = np.zeros(n_groups)
    for e in range(n):
        sums[e // cap] += loads[e]
    return sums


def optimal_max_group(loads, n_groups: int, bound: float = math.inf, max_nodes: int = 2_000_000):
    """Smallest achievable largest group sum with at most ceil(n / n_groups)
    experts per group (branch and bound over the loads in descending order;
    groups with equal (sum, size) are interchangeable, so only one of them is
    tried).  ``bound``: a known feasible value (e.g. the greedy's) to prune
    with; the result is then min(optimum, bound).  Exponential in n: returns
    None when the search visits more than ``max_nodes`` nodes."""
    loads = np.sort(np.asarray(loads, dtype=np.float64))[::-1]
    n = loads.shape[0]
    if n == 0:
        return 0.0
    cap = -(-n // n_groups)
    lb = max(float(loads.sum()) / n_groups, float(loads[0]))
    best = [bound if math.isfinite(bound) else math.inf]
    sums = [0.0] * n_groups
    sizes = [0] * n_groups
    nodes = [0]

    class _Budget(Exception):
        pass

    def rec(i, cur_max):
        nodes[0] += 1
        if nodes[0] > max_nodes:
            raise _Budget
        if cur_max >= best[0] or best[0] <= lb:
            return
        if i == n:
            best[0] = cur_max
            return
        seen = set()
        for g in range(n_groups):
            key = (sums[g], sizes[g])
            if sizes[g] >= cap or key in seen:
                continue
            seen.add(key)
            s = sums[g] + loads[i]
            if s >= best[0]:
                continue
            sums[g] = s
            sizes[g] += 1
            rec(i + 1, max(cur_max, s))
            sums[g] -= loads[i]
            sizes[g] -= 1

    try:
        rec(0, 0.0)
    except _Budget:
        return None
    return best[0]


def placement_report(loads, n_groups: int, expert_ids=None, exact_max_n: int = 16):
    """Summary of the greedy placement of measured loads into n_groups
    groups, beside the contiguous placement, a lower bound and (small n) the
    optimum.  ``expert_ids`` names the placed experts (e.g. the survivors
    of pruning) in the report."""
    loads = np.asarray(loads, dtype=np.float64)
    n = int(loads.shape[0])
    g = laep_rearrange(loads, n_groups)
    greedy = _summary(g["sums"])
    ids = list(range(n)) if expert_ids is None else [int(e) for e in expert_ids]
    greedy["groups"] = [[ids[e] for e in np.nonzero(g["group_of"] == k)[0]]
                        for k in range(n_groups)]
    contig = _summary(contiguous_sums(loads, n_groups))
    lb = max(float(loads.sum()) / n_groups, float(loads.max()) if n else 0.0)
    rep = {"n_experts": n, "n_groups": n_groups,
           "capacity": -(-n // n_groups) if n else 0,
           "total_load": float(loads.sum()),
           "greedy": greedy, "contiguous": contig,
           "contiguous_max_over_greedy_max": (contig["max"] / greedy["max"]
                                              if greedy["max"] > 0 else None),
           "lower_bound": lb,
           "greedy_gap_to_lower_bound": (greedy["max"] / lb - 1) if lb > 0 else 0.0}
    if n <= exact_max_n:
        # bound slightly above the greedy's so that an optimum equal to it is found
        opt = optimal_max_group(loads, n_groups, bound=greedy["max"] * (1 + 1e-12) + 1e-9)
        if opt is not None:
            opt = min(opt, greedy["max"])
            rep["optimum_max"] = opt
            rep["greedy_gap_to_optimum"] = (greedy["max"] / opt - 1) if opt > 0 else 0.0
    return rep
