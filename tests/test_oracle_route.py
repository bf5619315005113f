"""Pins of the oracle's router, top-k gating and expert histogram (CPU)."""
import itertools

import numpy as np
import pytest
import scipy.special

from oracle import moe
from oracle.numerics import round_f32


def _brute_topk(l, k, alive):
    """All C(E_alive, k) subsets; the best maximises the sum of logits."""
    cand = [e for e in range(len(l)) if alive[e]]
    best, best_sum, second = None, -np.inf, -np.inf
    for sub in itertools.combinations(cand, k):
        s = sum(l[e] for e in sub)
        if s > best_sum:
            second, best_sum, best = best_sum, s, sub
        elif s > second:
            second = s
    return set(best), best_sum, second


@pytest.mark.parametrize("E,k", [(8, 1), (8, 2), (6, 3), (5, 5), (4, 2)])
@pytest.mark.parametrize("masked", [False, True])
def test_topk_brute_force(E, k, masked):
    rng = np.random.default_rng(E * 10 + k + 100 * masked)
    T = 200
    logits = rng.standard_normal((T, E))
    alive = np.ones(E, bool)
    if masked:
        alive[rng.choice(E, size=max(0, E - k - 1), replace=False)] = False
        alive[:k] = True
    idx, gate, margin = moe.topk_gating(logits, k, alive=alive, renorm=True)
    lf = round_f32(logits)
    for t in range(T):
        sel, s, second = _brute_topk(lf[t], k, alive)
        assert set(idx[t].tolist()) == sel
        # slots in descending logit order
        vals = lf[t, idx[t]]
        assert np.all(np.diff(vals) <= 0)
        # unique best subset iff the k-th and (k+1)-th logits differ
        if alive.sum() > k:
            assert (margin[t] > 0) == (s > second)


def test_topk_ties_go_to_lower_index_and_k_equals_E_is_full_sort():
    l = np.array([[1.0, 3.0, 3.0, 2.0, 3.0]])
    idx, _, margin = moe.topk_gating(l, 2)
    assert idx.tolist() == [[1, 2]] and margin[0] == 0.0
    idx, _, _ = moe.topk_gating(l, 5)
    assert idx.tolist() == [[1, 2, 4, 3, 0]]


def test_gates_against_library_softmax():
    rng = np.random.default_rng(7)
    T, E, k = 64, 8, 3
    logits = rng.standard_normal((T, E)) * 3
    alive = np.array([1, 1, 0, 1, 1, 1, 0, 1], bool)
    lf = round_f32(logits)
    idx, g1, _ = moe.topk_gating(logits, k, alive=alive, renorm=True)
    idx0, g0, _ = moe.topk_gating(logits, k, alive=alive, renorm=False)
    assert np.array_equal(idx, idx0)
    for t in range(T):
        sm_sel = scipy.special.softmax(lf[t, idx[t]])
        np.testing.assert_allclose(g1[t], sm_sel, rtol=1e-7)
        full = np.full(E, -np.inf)
        full[alive] = lf[t, alive]
        sm_all = scipy.special.softmax(full)
        np.testing.assert_allclose(g0[t], sm_all[idx[t]], rtol=1e-7)
        assert abs(g1[t].sum() - 1) < 1e-6
        assert np.all(np.diff(g1[t]) <= 0)
        assert not np.any(np.isin(idx[t], np.nonzero(~alive)[0]))
    # gates are float32 values
    assert np.array_equal(g1, g1.astype(np.float32).astype(np.float64))


def test_k1_renorm_gate_is_one_and_fewer_alive_than_k():
    rng = np.random.default_rng(3)
    logits = rng.standard_normal((10, 6))
    _, g, _ = moe.topk_gating(logits, 1, renorm=True)
    assert np.all(g == 1.0)
    alive = np.array([0, 1, 0, 0, 1, 0], bool)
    idx, g, margin = moe.topk_gating(logits, 3, alive=alive)
    assert np.all(idx[:, 2] == -1) and np.all(g[:, 2] == 0)
    assert np.all(np.sort(idx[:, :2], axis=1) == [1, 4])
    assert np.all(np.isinf(margin))


def test_router_logits_against_explicit_sum():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((7, 12))
    w = rng.standard_normal((4, 12))
    b = rng.standard_normal(4)
    want = np.array([[sum(x[t, c] * w[e, c] for c in range(12)) + b[e]
                      for e in range(4)] for t in range(7)])
    np.testing.assert_allclose(moe.router_logits(x, w, b), want, rtol=1e-13)


@pytest.mark.parametrize("T,E,k", [(1, 1, 1), (50, 8, 2), (300, 64, 8), (33, 5, 5)])
def test_counts_invariants_and_brute_force(T, E, k):
    rng = np.random.default_rng(T + E + k)
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts, offsets, dest = moe.expert_counts(idx, E)
    assert counts.sum() == T * k and offsets[E] == T * k and offsets[0] == 0
    np.testing.assert_array_equal(counts, np.bincount(idx.reshape(-1), minlength=E))
    assert sorted(dest.tolist()) == list(range(T * k))          # bijection
    # brute force: rank among earlier tokens with the same expert
    for t in range(T):
        for j in range(k):
            e = idx[t, j]
            earlier = sum(1 for t2 in range(t) for j2 in range(k) if idx[t2, j2] == e)
            assert dest[t * k + j] == offsets[e] + earlier
    # inside a group, rows are ordered by token
    src_tok = np.empty(T * k, np.int64)
    src_tok[dest] = np.arange(T * k) // k
    for e in range(E):
        seg = src_tok[offsets[e]:offsets[e + 1]]
        assert np.all(np.diff(seg) > 0)


def test_counts_skip_unrouted_slots():
    idx = np.array([[0, -1], [1, -1], [0, -1]], np.int32)
    counts, offsets, dest = moe.expert_counts(idx, 3)
    assert counts.tolist() == [2, 1, 0] and offsets.tolist() == [0, 2, 3, 3]
    assert dest.tolist() == [0, -1, 2, -1, 1, -1]


def test_selection_gates_of_any_selection_against_library_softmax():
    """Gates of an arbitrary selection (not the top-k, in any slot order,
    with empty slots): scipy's softmax over the selected logits (renorm) or
    over all alive logits taken at the selected experts (full softmax)."""
    rng = np.random.default_rng(11)
    T, E, k = 40, 9, 4
    logits = rng.standard_normal((T, E)) * 2
    alive = np.array([1, 0, 1, 1, 1, 1, 0, 1, 1], bool)
    lf = round_f32(logits)
    live = np.nonzero(alive)[0]
    idx = np.stack([rng.permutation(live)[:k] for _ in range(T)]).astype(np.int32)
    idx[::5, 3] = -1                            # an empty slot in some rows
    for renorm in (True, False):
        g = moe.selection_gates(logits, idx, alive=alive, renorm=renorm)
        for t in range(T):
            used = idx[t] >= 0
            if renorm:
                want = scipy.special.softmax(lf[t, idx[t][used]])
            else:
                full = np.full(E, -np.inf)
                full[alive] = lf[t, alive]
                want = scipy.special.softmax(full)[idx[t][used]]
            np.testing.assert_allclose(g[t][used], want, rtol=1e-7)
            assert np.all(g[t][~used] == 0)
        # the gates follow the experts, not the slots
        perm = idx[:, ::-1].copy()
        np.testing.assert_array_equal(moe.selection_gates(logits, perm, alive=alive,
                                                          renorm=renorm), g[:, ::-1])
    # with the top-k selection they are topk_gating's gates
    ti, tg, _ = moe.topk_gating(logits, k, alive=alive, renorm=True)
    np.testing.assert_array_equal(moe.selection_gates(logits, ti, alive=alive), tg)
    # no slot filled: all gates zero
    assert np.all(moe.selection_gates(logits[:2], np.full((2, k), -1, np.int32)) == 0)
