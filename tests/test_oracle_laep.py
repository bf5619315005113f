"""Pins of the oracle's LAEP prune rule and expert rearrangement (CPU)."""
import math
import os

import numpy as np
import pytest

from oracle import laep

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                yield [c.strip() for c in line.split(";")]


def _ints(s):
    return [] if s == "-" else [int(v) for v in s.split(",")]


PRUNE = list(_rows("prune_examples.txt"))
REARR = list(_rows("rearrange_examples.txt"))


@pytest.mark.parametrize("row", PRUNE, ids=[r[0] + "/" + r[2] + "/" + r[3] for r in PRUNE])
def test_prune_worked_examples(row):
    counts, total, alpha, beta, want = row
    alive, n, _ = laep.prune_mask(_ints(counts), int(total), float(alpha), float(beta))
    pruned = sorted(np.nonzero(~alive)[0].tolist())
    assert pruned == _ints(want)
    assert n == len(pruned)


def _brute_prune(counts, total, alpha, beta):
    """Each expert checked at its own rank, independently of the others."""
    E = len(counts)
    rank = sorted(range(E), key=lambda e: (counts[e], e))
    pruned = set()
    for pos, e in enumerate(rank):
        cum = sum(counts[rank[i]] for i in range(pos + 1))
        if cum < total * beta and counts[e] < total * alpha / E:
            pruned.add(e)
    return pruned


def test_prune_invariants_random():
    rng = np.random.default_rng(11)
    for trial in range(300):
        E = int(rng.integers(1, 65))
        counts = (rng.pareto(1.0, E) * 50).astype(np.int64)
        total = max(int(counts.sum()), 1)
        beta = float(rng.choice([0.0, 0.01, 0.05, 0.1, 0.2, 0.5, 1.0]))
        alpha = float(rng.choice([math.inf, 0.1, 0.2, 0.4, 1.0, 3.0]))
        alive, n, order = laep.prune_mask(counts, total, alpha, beta)
        pruned = set(np.nonzero(~alive)[0].tolist())
        assert pruned == _brute_prune(counts.tolist(), total, alpha, beta)
        # the pruned set is a prefix of the ascending order
        assert set(order[:n].tolist()) == pruned
        # monotone in beta and alpha
        a2, _, _ = laep.prune_mask(counts, total, alpha, min(1.0, beta * 2 + 0.01))
        assert pruned <= set(np.nonzero(~a2)[0].tolist())
        a3, _, _ = laep.prune_mask(counts, total, alpha * 2, beta)
        assert pruned <= set(np.nonzero(~a3)[0].tolist())


def test_prune_is_strict_not_leq():
    # running sum hits beta*total exactly at the 2nd expert
    alive, n, _ = laep.prune_mask([5, 5, 90], 100, math.inf, 0.1)
    assert n == 1 and not alive[0] and alive[1]


def test_algorithm1_window_reduces_to_single_pass():
    rng = np.random.default_rng(2)
    etn = rng.integers(0, 200, size=(1, 3, 16))
    S, topK = int(etn[0, 0].sum()), 1
    pruned = laep.expert_pruning(etn, S, topK, alpha=[0.2, 0.4, 0.2], beta=0.1)
    for layer, a in enumerate([0.2, 0.4, 0.2]):
        alive, _, _ = laep.prune_mask(etn[0, layer], S * topK, a, 0.1)
        assert pruned[layer].tolist() == np.nonzero(~alive)[0].tolist()


def test_algorithm1_window_hand_example():
    # 3 iterations, 1 layer, 4 experts; S*topK = 100, beta = 0.1, alpha = inf.
    # iter 0 loads [1, 50, 4, 45] -> ascending e0(1), e2(4), e3, e1: cum 1, 5, 50 -> marks {0, 2}
    # iter 1 loads [8, 50, 1, 41] -> e2(1), e0(8): cum 1, 9, 50 -> marks {2, 0}
    # iter 2 loads [2, 40, 9, 49] -> e0(2), e2(9): cum 2, 11 -> marks {0}
    # Exp_dis = 5 -> N = round(5/3) = 2; markers e0: 3, e2: 2 -> pruned {0, 2}
    etn = np.array([[[1, 50, 4, 45]], [[8, 50, 1, 41]], [[2, 40, 9, 49]]])
    pruned = laep.expert_pruning(etn, 100, 1, alpha=math.inf, beta=0.1)
    assert pruned[0].tolist() == [0, 2]


@pytest.mark.parametrize("row", REARR, ids=[r[0] for r in REARR])
def test_rearrange_worked_examples(row):
    loads, n_g, groups, sums = row
    res = laep.rearrange([float(v) for v in loads.split(",")], int(n_g))
    want_groups = [_ints(g) for g in groups.split("|")]
    assert res["groups"] == want_groups
    np.testing.assert_array_equal(res["sums"], [float(v) for v in sums.split(",")])
    flat = [e for g in want_groups for e in g]
    assert res["order"].tolist() == flat
    loads_a = np.array([float(v) for v in loads.split(",")])
    np.testing.assert_array_equal(res["reordered"], loads_a[flat])


def test_rearrange_invariants_and_gap_report():
    rng = np.random.default_rng(4)
    for trial in range(60):
        n = int(rng.integers(1, 10))
        n_g = int(rng.integers(1, n + 1))
        loads = rng.integers(0, 100, size=n).astype(float)
        res = laep.rearrange(loads, n_g)
        cap = -(-n // n_g)
        members = sorted(e for g in res["groups"] for e in g)
        assert members == list(range(n))                   # a partition
        assert all(len(g) <= cap for g in res["groups"])   # capacity
        assert abs(res["sums"].sum() - loads.sum()) < 1e-9
        for g, m in enumerate(res["groups"]):
            assert all(res["group_of"][e] == g for e in m)
        # the greedy is a heuristic; its gap to the optimum is reported only
        best = laep.best_partition_spread(loads, n_g)
        assert res["sums"].max() >= best - 1e-9
