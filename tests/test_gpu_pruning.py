"""GPU parity of Algorithm 1 over a recorded window (laep_expert_pruning), the
ETN recording through moe_expert_counts, and physical expert compaction
(laep_compact_experts, laep_repack_experts) against the oracle."""
import math

import numpy as np
import pytest
import torch

import oracle.laep as ol
import oracle.moe as om
import paper_2601_14327_amd as laep
from workloads import random_case
from _gpu import TOL_BF16, case, check_routing, dev, host, rownorm_err

pytestmark = pytest.mark.gpu


def _window(rng, iters, L, E, total, skew):
    """Loads per (iteration, layer): a multinomial split of ``total`` over
    experts with Pareto-skewed preferences that drift a little per iteration."""
    etn = np.zeros((iters, L, E), np.int64)
    for l in range(L):
        pref = rng.pareto(skew, E) + 1e-3
        for it in range(iters):
            p = pref * rng.uniform(0.7, 1.3, E)
            etn[it, l] = rng.multinomial(total, p / p.sum())
    return etn


def _check_pruning(etn, total, alpha, beta):
    iters, L, E = etn.shape
    alive, n, marker = laep.laep_expert_pruning(dev(etn, torch.int64), total, alpha, beta,
                                                want_marker=True)
    torch.cuda.synchronize()
    pruned, ref_marker = ol.expert_pruning(etn, total, 1, alpha, beta, return_marker=True)
    a = host(alive).astype(bool)
    for l in range(L):
        assert np.nonzero(~a[l])[0].tolist() == pruned[l].tolist(), f"layer {l}"
        assert int(host(n)[l]) == len(pruned[l])
    np.testing.assert_array_equal(host(marker), ref_marker)


def test_expert_pruning_window_parity():
    rng = np.random.default_rng(41)
    cases = 0
    for iters, L, E in [(1, 1, 8), (3, 4, 16), (8, 12, 64), (5, 2, 256), (2, 6, 1), (16, 3, 64)]:
        for skew in (0.6, 1.5):
            total = int(rng.integers(1000, 100000))
            etn = _window(rng, iters, L, E, total, skew)
            for alpha, beta in [(math.inf, 0.05), (ol.hybrid_alpha(L), 0.1),
                                (0.4, 0.3), (0.2, 1.0)]:
                case(f"expert_pruning ITER={iters} L={L} E={E} skew={skew} beta={beta}")
                _check_pruning(etn, total, alpha, beta)
                cases += 1
    assert cases == 48


def test_expert_pruning_ties_and_hand_window():
    # the worked window of the oracle's pins (3 iterations, 4 experts)
    etn = np.array([[[1, 50, 4, 45]], [[8, 50, 1, 41]], [[2, 40, 9, 49]]], np.int64)
    case("expert_pruning hand window")
    _check_pruning(etn, 100, math.inf, 0.1)
    # equal loads everywhere: ranks by index, markers tie, window sums tie
    etn = np.full((4, 2, 10), 7, np.int64)
    _check_pruning(etn, 70, math.inf, 0.35)
    # zero loads (dead experts) and an all-zero layer
    etn = np.zeros((3, 2, 12), np.int64)
    etn[:, 0, :6] = 40
    _check_pruning(etn, 240, 1.0, 0.5)


def test_etn_window_recorded_by_counts():
    rng = np.random.default_rng(5)
    iters, L, E, T, k = 3, 2, 16, 300, 4
    pruner = laep.ExpertPruner(iters, L, E, T, k, alpha=ol.hybrid_alpha(L), beta=0.1)
    ref = np.zeros((iters, L, E), np.int64)
    case("etn window recording")
    for it in range(iters):
        for l in range(L):
            pref = rng.pareto(1.0, E) + 0.05
            idx = np.stack([rng.choice(E, k, replace=False, p=pref / pref.sum())
                            for _ in range(T)]).astype(np.int32)
            laep.moe_expert_counts(dev(idx, torch.int32), E, etn_accum=pruner.slot(it, l))
            ref[it, l] = np.bincount(idx.ravel(), minlength=E)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(pruner.etn), ref)
    alive, n, _ = pruner.decide()
    pruned = ol.expert_pruning(ref, T, k, ol.hybrid_alpha(L), 0.1)
    a = host(alive).astype(bool)
    for l in range(L):
        assert np.nonzero(~a[l])[0].tolist() == pruned[l].tolist()


def test_compact_map_parity():
    rng = np.random.default_rng(8)
    for L, E in [(1, 1), (3, 8), (12, 64), (2, 256), (4, 200)]:
        alive = (rng.random((L, E)) < rng.random((L, 1))).astype(np.uint8)
        alive[0, :] = 1
        if L > 1:
            alive[1, :] = 0
        case(f"compact map L={L} E={E}")
        m, n = laep.laep_compact_experts(dev(alive, torch.uint8))
        torch.cuda.synchronize()
        for l in range(L):
            rm, rn = ol.compact(alive[l])
            np.testing.assert_array_equal(host(m)[l], rm)
            assert int(host(n)[l]) == rn


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_repack_parity(dtype):
    rng = np.random.default_rng(9)
    td = {"bf16": torch.bfloat16, "f32": torch.float32}[dtype]
    E, d, f = 16, 64, 96
    c = random_case(77, T=8, d_model=d, E=E, k=2, d_ff=f, dtype=dtype, bias_std=1.0)
    alive = np.ones(E, np.uint8)
    alive[[0, 3, 4, 10, 15]] = 0
    rm, rn = ol.compact(alive)
    keep = np.nonzero(alive)[0]
    w_r, w_gu, w_d = (dev(c[n], td) for n in ("w_router", "w_gate_up", "w_down"))
    bias = dev(c["bias"], torch.float32)
    state = dev(rng.standard_normal((E, 2 * f, d)).astype(np.float32), torch.float32)
    case(f"repack {dtype}")
    m, n = laep.laep_compact_experts(dev(alive, torch.uint8))
    out = laep.laep_repack_experts(m, rn, w_router=w_r, bias=bias, w_gate_up=w_gu, w_down=w_d)
    st = laep.laep_repack_experts(m, rn, w_gate_up=state)
    torch.cuda.synchronize()
    assert int(host(n)[0]) == rn
    for name, src in (("w_router", w_r), ("bias", bias), ("w_gate_up", w_gu), ("w_down", w_d)):
        assert torch.equal(out[name].cpu(), src.cpu()[torch.from_numpy(keep)]), name
    assert torch.equal(st["w_gate_up"].cpu(), state.cpu()[torch.from_numpy(keep)])
    # fewer slots than survivors: only slots < n_out are written
    sentinel = torch.full((4, d), 3.0, dtype=td, device="cuda")
    laep.laep_repack_experts(m, 3, w_router=w_r, out={"w_router": sentinel})
    torch.cuda.synchronize()
    assert torch.equal(sentinel[:3].cpu(), w_r.cpu()[torch.from_numpy(keep[:3])])
    assert torch.all(sentinel[3].float().cpu() == 3.0)


def _layer(x, w_r, bias, w_gu, w_d, k, alive=None):
    idx, gate, logits = laep.moe_route(x, w_r, k, bias=bias, alive=alive, want_logits=True)
    counts, offsets, dest = laep.moe_expert_counts(idx, w_r.shape[0])
    xp = laep.moe_permute(x, dest, k)
    y, _ = laep.moe_grouped_ffn_fwd(xp, w_gu, w_d, offsets, save_act=False)
    out = laep.moe_combine(y, gate, dest)
    return dict(idx=idx, gate=gate, logits=logits, offsets=offsets, dest=dest, y=y, out=out)


def test_pruned_and_compacted_layer_end_to_end():
    """Record a window of skewed routing, prune with Algorithm 1, remove the
    pruned experts, and run the compact layer: it routes like the masked layer
    and matches the oracle of the survivors."""
    T, d, E, k, f = 512, 256, 16, 4, 128
    c = random_case(123, T=T, d_model=d, E=E, k=k, d_ff=f, dtype="bf16", bias_std=1.5)
    x, w_r, w_gu, w_d = (dev(c[n], torch.bfloat16) for n in ("x", "w_router", "w_gate_up",
                                                               "w_down"))
    bias = dev(c["bias"], torch.float32)
    rng = np.random.default_rng(6)
    iters = 4
    pruner = laep.ExpertPruner(iters, 1, E, T, k, alpha=math.inf, beta=0.1)
    case("pruned layer: window")
    for it in range(iters):
        xi = dev(c["x"][rng.permutation(T)], torch.bfloat16)
        idx, _ = laep.moe_route(xi, w_r, k, bias=bias)
        laep.moe_expert_counts(idx, E, etn_accum=pruner.slot(it, 0))
    alive, n_pruned, _ = pruner.decide()
    torch.cuda.synchronize()
    pruned = ol.expert_pruning(host(pruner.etn), T, k, math.inf, 0.1)[0]
    a = host(alive)[0].astype(bool)
    assert np.nonzero(~a)[0].tolist() == pruned.tolist()
    assert 0 < len(pruned) < E - k, f"pruned {len(pruned)} of {E}: the case should prune some"
    case("pruned layer: compact and run")
    small = laep.compact_layer(alive[0].contiguous(), w_router=w_r, w_gate_up=w_gu, w_down=w_d,
                               bias=bias)
    n_alive = small["n_alive"]
    assert n_alive == E - len(pruned)
    masked = _layer(x, w_r, bias, w_gu, w_d, k, alive=alive[0].contiguous())
    comp = _layer(x, small["w_router"], small["bias"], small["w_gate_up"], small["w_down"], k)
    torch.cuda.synchronize()
    # the compact layer's expert ids are the masked layer's, through the slot map
    rm, _ = ol.compact(a)
    keep = np.nonzero(a)[0]
    # both device routings are checked against the oracle: the compact layer
    # against the oracle of the survivors, the masked layer against the
    # oracle over all experts with the alive mask
    ref = om.route(c["x"], c["w_router"][keep], k, bias=c["bias"][keep])
    check_routing(host(comp["idx"]), host(comp["gate"]), ref[0], ref[1], ref[3], k,
                  label="pruned layer, compact")
    refm = om.route(c["x"], c["w_router"], k, bias=c["bias"], alive=a)
    check_routing(host(masked["idx"]), host(masked["gate"]), refm[0], refm[1], refm[3], k, a,
                  label="pruned layer, masked")
    # the compact layer's ids are the masked layer's through the slot map
    # (up to the near-ties both checks allow)
    same = np.all(rm[host(masked["idx"])] == host(comp["idx"]), axis=1)
    np.testing.assert_array_equal(rm[refm[0]], ref[0])
    # identical routing gives identical expert rows and outputs
    if same.all():
        assert torch.equal(masked["y"], comp["y"])
    ref_out = om.layer_forward(c["x"], c["w_router"][keep], c["w_gate_up"][keep],
                               c["w_down"][keep], k, bias=c["bias"][keep])["out"]
    err = rownorm_err(host(comp["out"]), ref_out)
    assert err <= TOL_BF16, err
    # the parameter reduction: the compact tensors hold only the survivors
    assert small["w_gate_up"].shape[0] == n_alive and small["w_router"].shape[0] == n_alive
