"""The rearrangement placement report (paper_2601_14327_amd/placement.py):
the greedy groups come from the C ABI's laep_rearrange; the contiguous
placement, the lower bound and the exact optimum are checked against worked
examples and against the oracle's brute force (CPU)."""
import itertools

import numpy as np
import pytest

from oracle import laep as olaep


@pytest.fixture(scope="module")
def P():
    import paper_2601_14327_amd as laep

    return laep


def test_worked_examples(P):
    # the worked example of Algorithm 2 (tests/golden/rearrange_examples.txt)
    r = P.placement_report([40, 30, 20, 10, 5, 5], 2)
    assert r["capacity"] == 3
    assert r["greedy"]["group_sums"] == [55.0, 55.0]
    assert r["greedy"]["groups"] == [[0, 3, 4], [1, 2, 5]]
    assert r["contiguous"]["group_sums"] == [90.0, 20.0]        # {0,1,2} and {3,4,5}
    assert r["contiguous_max_over_greedy_max"] == pytest.approx(90 / 55)
    assert r["optimum_max"] == 55.0 and r["greedy_gap_to_optimum"] == 0.0
    assert r["lower_bound"] == 55.0
    # one dominant expert: every placement's largest group holds it
    r = P.placement_report([100, 1, 1, 1], 2)
    assert r["greedy"]["group_sums"] == [101.0, 2.0]
    assert r["contiguous"]["group_sums"] == [101.0, 2.0]
    assert r["optimum_max"] == 101.0 and r["lower_bound"] == 100.0
    # expert ids name the placed experts (e.g. the survivors of pruning)
    r = P.placement_report([3.0, 9.0, 1.0], 3, expert_ids=[4, 10, 20])
    assert sorted(sum(r["greedy"]["groups"], [])) == [4, 10, 20]


def test_contiguous_placement_by_definition(P):
    from paper_2601_14327_amd.placement import contiguous_sums

    rng = np.random.default_rng(2)
    for _ in range(50):
        n = int(rng.integers(1, 70))
        g = int(rng.integers(1, n + 1))
        loads = rng.integers(0, 100, n).astype(float)
        cap = -(-n // g)
        want = [sum(loads[e] for e in range(n) if e // cap == q) for q in range(g)]
        np.testing.assert_array_equal(contiguous_sums(loads, g), want)


def test_optimum_against_oracle_brute_force(P):
    from paper_2601_14327_amd.placement import optimal_max_group

    rng = np.random.default_rng(3)
    for _ in range(120):
        n = int(rng.integers(1, 10))
        g = int(rng.integers(1, n + 1))
        loads = rng.integers(0, 50, n).astype(float)
        want = olaep.best_partition_spread(loads, g)
        assert optimal_max_group(loads, g) == want
        r = P.placement_report(loads, g)
        assert r["optimum_max"] == want
        assert r["lower_bound"] <= want <= r["greedy"]["max"]
        assert r["greedy"]["group_sums"] == olaep.rearrange(loads, g)["sums"].tolist()


def test_two_per_group_optimum_is_extremes_paired(P):
    # capacity 2 with every slot filled: pairing the largest with the
    # smallest load is optimal (exchange argument)
    from paper_2601_14327_amd.placement import optimal_max_group

    rng = np.random.default_rng(4)
    for _ in range(20):
        loads = np.sort(rng.integers(1, 1000, 16).astype(float))
        want = max(loads[i] + loads[15 - i] for i in range(8))
        assert optimal_max_group(rng.permutation(loads), 8) == want


def test_search_budget(P):
    from paper_2601_14327_amd.placement import optimal_max_group

    assert optimal_max_group(np.arange(1, 31, dtype=float) ** 1.5, 3, max_nodes=100) is None
