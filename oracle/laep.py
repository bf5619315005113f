"""Oracle of LAEP's pruning rule and expert rearrangement (float64 / ints).

Test infrastructure only; see the package docstring.

Pruning (Section 3.2, Eqs. (1)-(2); Appendix, Algorithm 1).  Experts are
ranked by load, smallest first.  Walking that order, the running sum of
loads is accumulated *including* the current expert, and the expert is
marked when

    running_sum < S * topK * beta      (cumulative-load criterion, Eq. (2))
and load        < S * topK * alpha / E (individual-load criterion, Eq. (1))

The equations print "<=", while Algorithm 1 and the prose use a strict "<";
the strict form is taken here (two of three sources).  Equal loads are
ordered by expert index (a stable sort).  alpha = inf disables Eq. (1).
Both thresholds are evaluated in IEEE double in the operation order
(total * beta) and (total * alpha) / E, total = S * topK.

Because loads are ascending and the running sum is non-decreasing, once an
expert fails either test every later one does too: the marked set is a
prefix of the ascending order.

Rearrangement (Section 3.3; Appendix, Algorithm 2).  Experts are visited in
descending load order and each goes to the group with the smallest running
sum that still has room.  The printed group size floor(n / n_g) leaves too
little room when n_g does not divide n (the loop could not place the last
experts); the capacity here is ceil(n / n_g).  Ties in the minimum go to the
lowest group index and equal loads keep index order.  Full groups are set
to +inf in the running sums as in the algorithm; the reported sums are
recomputed from the group lists.
"""
from __future__ import annotations

import math

import numpy as np


# --------------------------------------------------------------------------
# Algorithm 1 for one iteration and one layer
# --------------------------------------------------------------------------
def prune_mask(counts, total: int, alpha: float = math.inf, beta: float = 0.0):
    """One (iteration, layer) pass of Algorithm 1's marking step.

    counts: per-expert loads (ETN row); total = S * topK.
    Returns (alive [E] bool, n_pruned, order) where ``order`` is the
    ascending (load, index) ranking.
    """
    counts = np.asarray(counts, dtype=np.int64)
    E = counts.shape[0]
    order = np.argsort(counts, kind="stable")      # ascending, ties by index
    beta_thr = float(total) * float(beta)
    alpha_thr = (float(total) * float(alpha)) / float(E)
    running = 0
    alive = np.ones(E, dtype=bool)
    n_pruned = 0
    for pos in range(E):
        e = int(order[pos])
        load = int(counts[e])
        running += load                            # inclusive running sum
        if float(running) < beta_thr and float(load) < alpha_thr:
            alive[e] = False
            n_pruned += 1
    return alive, n_pruned, order


def expert_pruning(etn, S: int, topK: int, alpha, beta: float, return_marker: bool = False):
    """Algorithm 1 over a window of ITER iterations and L layers.

    etn: [ITER, L, E] token counts (Step 1).  alpha: scalar or per-layer
    sequence (the layer-adaptive schedule).  Step 2 marks, per iteration and
    layer, the experts Eqs. (1)-(2) select and counts them (Exp_dis).
    Step 3 prunes, per layer, the N most-marked experts.

    Readings where the printed algorithm is ambiguous:
    * Marker is indexed by expert id (the printed index is the rank
      position, which would make Step 3 return ranks, not experts);
    * N = round(Exp_dis / ITER), the mean number marked per iteration
      (Exp_dis accumulates over ITER but is used as a per-layer count);
    * Marker ties go to the lower mean load, then to the lower index;
    * the running sum restarts at 0 for every (iteration, layer).
    Returns a list of L int arrays, the pruned expert ids per layer (and the
    Marker array [L, E] when return_marker).
    """
    etn = np.asarray(etn, dtype=np.int64)
    ITER, L, E = etn.shape
    alphas = [alpha] * L if np.isscalar(alpha) else list(alpha)
    total = int(S) * int(topK)
    exp_dis = np.zeros(L, dtype=np.int64)
    marker = np.zeros((L, E), dtype=np.int64)
    for it in range(ITER):
        for layer in range(L):
            alive, n, _ = prune_mask(etn[it, layer], total, alphas[layer], beta)
            exp_dis[layer] += n
            marker[layer] += (~alive).astype(np.int64)
    pruned = []
    mean_load = etn.mean(axis=0)
    for layer in range(L):
        n_dis = int(np.floor(exp_dis[layer] / ITER + 0.5))
        # most-marked first; ties: lower mean load, then lower index
        order = np.lexsort((np.arange(E), mean_load[layer], -marker[layer]))
        pruned.append(np.sort(order[:n_dis]).astype(np.int64))
    return (pruned, marker) if return_marker else pruned


# --------------------------------------------------------------------------
# Layer-adaptive alpha and the removal of pruned experts
# --------------------------------------------------------------------------
def hybrid_alpha(n_layers: int, edge: float = 0.2, middle: float = 0.4):
    """The per-layer alpha of the Section 3.4 ablation and the Section 4
    run: ``edge`` for the first and the last sixth of the layers, ``middle``
    for the two thirds between.  Reading: a sixth of L layers is L / 6
    rounded to the nearest integer, halves up (the paper's models have L a
    multiple of 6 or say nothing)."""
    n_edge = int(math.floor(n_layers / 6 + 0.5))
    return [edge if (l < n_edge or l >= n_layers - n_edge) else middle
            for l in range(n_layers)]


def compact(alive):
    """Slots of the surviving experts (Section 3.2: pruned experts leave the
    model).  Survivors keep their order: slot = number of alive experts with
    a lower index; pruned experts map to -1.  Returns (expert_map, n_alive)."""
    alive = np.asarray(alive).astype(bool)
    expert_map = np.full(alive.shape[0], -1, dtype=np.int64)
    slot = 0
    for e in range(alive.shape[0]):
        if alive[e]:
            expert_map[e] = slot
            slot += 1
    return expert_map, slot


# --------------------------------------------------------------------------
# Algorithm 2: expert rearrangement
# --------------------------------------------------------------------------
def rearrange(loads, n_groups: int):
    """Greedy placement of experts into n_groups device groups.

    Returns dict(groups=list of expert-id lists, group_of=[n] int,
    order=In_flat [n] int, reordered=D_r [n], sums=[n_groups] float).
    """
    loads = np.asarray(loads, dtype=np.float64)
    n = loads.shape[0]
    if n_groups < 1:
        raise ValueError("n_groups must be >= 1")
    cap = -(-n // n_groups)                        # ceil(n / n_g)
    order = np.argsort(-loads, kind="stable")      # descending, ties by index
    groups = [[] for _ in range(n_groups)]
    running = [0.0] * n_groups
    for idx in order:
        idx = int(idx)
        while True:
            g = min(range(n_groups), key=lambda i: (running[i], i))
            if len(groups[g]) < cap:
                groups[g].append(idx)
                running[g] += loads[idx]
                break
            running[g] = math.inf                  # mark the group full
    group_of = np.empty(n, dtype=np.int64)
    for g, members in enumerate(groups):
        for e in members:
            group_of[e] = g
    flat = np.array([e for members in groups for e in members], dtype=np.int64)
    sums = np.array([float(loads[m].sum()) if m else 0.0 for m in groups])
    return dict(groups=groups, group_of=group_of, order=flat,
                reordered=loads[flat], sums=sums, capacity=cap)


def best_partition_spread(loads, n_groups: int):
    """Brute force over all capacity-respecting assignments (tiny n only):
    the smallest possible max-group-sum.  Used to report the greedy's gap;
    the greedy is a heuristic, so its optimality is parity unpinned."""
    loads = np.asarray(loads, dtype=np.float64)
    n = loads.shape[0]
    cap = -(-n // n_groups)
    best = math.inf

    def rec(i, sums, sizes):
        nonlocal best
        if max(sums) >= best:
            return
        if i == n:
            best = max(sums)
            return
        seen = set()
        for g in range(n_groups):
            if sizes[g] < cap and (sums[g], sizes[g]) not in seen:
                seen.add((sums[g], sizes[g]))
                sums[g] += loads[i]
                sizes[g] += 1
                rec(i + 1, sums, sizes)
                sums[g] -= loads[i]
                sizes[g] -= 1

    rec(0, [0.0] * n_groups, [0] * n_groups)
    return best
