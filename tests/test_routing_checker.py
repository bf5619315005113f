"""The routing checker of the GPU tests (tests/_gpu.py::check_routing), run on
the CPU against planted routings: genuine near-tie alternatives pass, and
each plausible device mistake is rejected."""
import numpy as np
import pytest

from oracle import moe
import _gpu
from _gpu import NEAR_TIE, check_routing

T, E, K = 2000, 16, 8     # 16000 routings: the mismatch budget allows one


@pytest.fixture(autouse=True)
def _keep_records_clean():
    # planted cases are not device results: keep them out of the session's
    # near-tie summary
    n = len(_gpu.ROUTING_RECORDS)
    yield
    del _gpu.ROUTING_RECORDS[n:]


def _case():
    rng = np.random.default_rng(21)
    logits = rng.standard_normal((T, E))
    # token 0: the top k nearly equal, and a boundary near-tie with expert k+1
    o = np.argsort(-logits[0], kind="stable")
    logits[0, o[:K]] = 2.0 + 1e-3 * np.arange(K)[::-1]
    logits[0, o[K]] = 2.0 - 0.9 * NEAR_TIE
    # token 1: an inner near-tie between its slots 1 and 2
    o1 = np.argsort(-logits[1], kind="stable")
    logits[1, o1[2]] = logits[1, o1[1]] - 0.3 * NEAR_TIE
    # token 2: its first two logits far apart
    o2 = np.argsort(-logits[2], kind="stable")
    logits[2, o2[1]] = logits[2, o2[0]] - 0.5
    # token 3: a second boundary near-tie
    o3 = np.argsort(-logits[3], kind="stable")
    logits[3, o3[K]] = logits[3, o3[K - 1]] - 0.5 * NEAR_TIE
    idx, gate, margin = moe.topk_gating(logits, K)
    assert margin[0] < NEAR_TIE and margin[3] < NEAR_TIE
    return logits, idx, gate


def _swap_boundary(logits, idx, t):
    o = np.argsort(-logits[t], kind="stable")
    out = idx.copy()
    out[t, K - 1] = o[K]
    return out


def _regate(logits, idx, gate, toks):
    g = gate.copy()
    g[toks] = moe.selection_gates(logits[toks], idx[toks])
    return g


def test_identical_routing_passes():
    logits, idx, gate = _case()
    n, err = check_routing(idx, gate, idx, gate, logits, K, label="planted: identical")
    assert n == 0 and err == 0


def test_boundary_near_tie_alternative_passes():
    logits, idx, gate = _case()
    alt = _swap_boundary(logits, idx, 0)
    n, _ = check_routing(alt, _regate(logits, alt, gate, [0]), idx, gate, logits, K,
                         label="planted: boundary near-tie")
    assert n == 1


def test_inner_near_tie_slot_order_passes():
    logits, idx, gate = _case()
    alt, g = idx.copy(), gate.copy()
    alt[1, [1, 2]] = alt[1, [2, 1]]
    g[1, [1, 2]] = g[1, [2, 1]]
    n, _ = check_routing(alt, g, idx, gate, logits, K, label="planted: inner near-tie")
    assert n == 1


def test_far_expert_swapped_in_at_a_near_tie_is_rejected():
    logits, idx, gate = _case()
    alt = idx.copy()
    alt[0, K - 1] = int(np.argmin(logits[0]))          # the lowest logit, far away
    with pytest.raises(AssertionError, match="away from a near-tie"):
        check_routing(alt, _regate(logits, alt, gate, [0]), idx, gate, logits, K)


def test_reordered_non_tied_pair_is_rejected():
    logits, idx, gate = _case()
    alt, g = idx.copy(), gate.copy()
    alt[2, [0, 1]] = alt[2, [1, 0]]
    g[2, [0, 1]] = g[2, [1, 0]]
    with pytest.raises(AssertionError, match="away from a near-tie"):
        check_routing(alt, g, idx, gate, logits, K)


def test_near_tie_alternative_with_the_oracles_gates_is_rejected():
    # the device chose the tied expert but kept the gates of the other set
    logits, idx, gate = _case()
    alt = _swap_boundary(logits, idx, 0)
    with pytest.raises(AssertionError, match="differ from their own selection"):
        check_routing(alt, gate, idx, gate, logits, K)


@pytest.mark.parametrize("mistake", ["scaled", "full_softmax"])
def test_wrong_gates_at_a_near_tie_are_rejected(mistake):
    logits, idx, gate = _case()
    alt = _swap_boundary(logits, idx, 0)
    g = _regate(logits, alt, gate, [0])
    if mistake == "scaled":
        g[0] *= 0.5
    else:   # gates of the full softmax where the call asked for renormalised ones
        g[0] = moe.selection_gates(logits[:1], alt[:1], renorm=False)[0]
    with pytest.raises(AssertionError, match="differ from their own selection"):
        check_routing(alt, g, idx, gate, logits, K)


def test_gate_error_on_a_matching_token_is_rejected():
    logits, idx, gate = _case()
    g = gate.copy()
    g[7, 0] *= 1 + 1e-4
    with pytest.raises(AssertionError, match="routed as the oracle"):
        check_routing(idx, g, idx, gate, logits, K)


def test_repeated_or_dead_expert_is_rejected():
    logits, idx, gate = _case()
    alt = idx.copy()
    alt[9, 1] = alt[9, 0]
    with pytest.raises(AssertionError, match="repeats"):
        check_routing(alt, gate, idx, gate, logits, K)
    alive = np.ones(E, bool)
    alive[int(idx[4, 0])] = False
    ridx, rgate, _ = moe.topk_gating(logits, K, alive=alive)
    bad = ridx.copy()
    bad[4, K - 1] = idx[4, 0]                           # the dead expert
    with pytest.raises(AssertionError, match="dead expert"):
        check_routing(bad, rgate, ridx, rgate, logits, K, alive)


def test_mismatch_budget_is_enforced():
    # two genuine near-tie swaps are two differing routings: over the budget
    logits, idx, gate = _case()
    alt = _swap_boundary(logits, _swap_boundary(logits, idx, 0), 3)
    with pytest.raises(AssertionError, match="mismatched routings"):
        check_routing(alt, _regate(logits, alt, gate, [0, 3]), idx, gate, logits, K)
