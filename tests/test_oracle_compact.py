"""Pins of the oracle's layer-adaptive alpha (oracle.laep.hybrid_alpha) and
expert compaction (oracle.laep.compact): the schedule the paper states in
words, and the property that removing pruned experts leaves the layer's
function unchanged (a layer routed with an alive mask over E experts equals
the layer built from the survivors alone)."""
import numpy as np
import pytest

import oracle.laep as laep
import oracle.moe as om


def test_hybrid_alpha_matches_the_stated_split():
    # Section 3.4: alpha = 20 % on the first and last 1/6 of the layers,
    # 40 % on the middle 2/3.
    assert laep.hybrid_alpha(6) == [0.2, 0.4, 0.4, 0.4, 0.4, 0.2]
    assert laep.hybrid_alpha(12) == [0.2] * 2 + [0.4] * 8 + [0.2] * 2
    for L in range(6, 121, 6):
        a = laep.hybrid_alpha(L)
        assert a[: L // 6] == [0.2] * (L // 6) and a[L - L // 6:] == [0.2] * (L // 6)
        assert a[L // 6: L - L // 6] == [0.4] * (2 * L // 3)
    # reading for L not divisible by 6: round(L / 6), halves up
    assert laep.hybrid_alpha(103).count(0.2) == 2 * 17
    assert laep.hybrid_alpha(9).count(0.2) == 2 * 2          # 1.5 -> 2
    assert laep.hybrid_alpha(1) == [0.4]                      # 1/6 rounds to 0
    assert laep.hybrid_alpha(4, 0.1, 0.7) == [0.1, 0.7, 0.7, 0.1]


def test_compact_is_a_monotone_bijection_onto_the_slots():
    rng = np.random.default_rng(3)
    for _ in range(50):
        E = int(rng.integers(1, 70))
        alive = rng.random(E) < rng.random()
        m, n = laep.compact(alive)
        assert n == int(alive.sum())
        assert np.all(m[~alive] == -1)
        assert sorted(m[alive].tolist()) == list(range(n))     # onto 0..n-1
        assert np.all(np.diff(m[alive]) == 1)                  # order kept


@pytest.mark.parametrize("renorm", [True, False])
def test_compacted_layer_equals_the_masked_layer(renorm):
    rng = np.random.default_rng(11)
    T, d, E, k, f = 48, 32, 12, 3, 16
    x = rng.standard_normal((T, d))
    w_r = rng.standard_normal((E, d)) * 0.3
    bias = rng.standard_normal(E)
    w_gu = rng.standard_normal((E, 2 * f, d)) * 0.1
    w_d = rng.standard_normal((E, d, f)) * 0.1
    alive = np.ones(E, bool)
    alive[[1, 4, 5, 9]] = False
    m, n = laep.compact(alive)
    keep = np.nonzero(alive)[0]
    full = om.layer_forward(x, w_r, w_gu, w_d, k, bias=bias, alive=alive, renorm=renorm,
                            dtype="f64")
    small = om.layer_forward(x, w_r[keep], w_gu[keep], w_d[keep], k, bias=bias[keep],
                             renorm=renorm, dtype="f64")
    assert full["margin"].min() > 1e-9
    # the survivors' ids map through the slot map; gates and outputs agree
    np.testing.assert_array_equal(m[full["idx"]], small["idx"])
    np.testing.assert_allclose(small["gate"], full["gate"], rtol=1e-6, atol=0)
    np.testing.assert_allclose(small["out"], full["out"], rtol=1e-6, atol=1e-12)
    # the grouped FFN over the full weights through the map is the same layer
    y_map, _ = om.grouped_ffn_fwd(full["x_perm"], w_gu[keep], w_d[keep], full["offsets"],
                                  expert_map=m, dtype="f64")
    np.testing.assert_array_equal(y_map, full["y_perm"])


def test_compact_with_nothing_pruned_or_all_pruned():
    m, n = laep.compact(np.ones(7, bool))
    assert n == 7 and m.tolist() == list(range(7))
    m, n = laep.compact(np.zeros(5, bool))
    assert n == 0 and m.tolist() == [-1] * 5
