"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (MoELayerPlan).  Integer outputs are checked completely;
floating-point outputs on rows the oracle computes one by one (rows are
independent, so a row subset is exact): one row from every 32-row block of
every 256-row tile of every expert, and for the weight gradients whole
256 x 256 output tiles."""
import numpy as np
import pytest
import torch

import oracle.laep as ol
import oracle.moe as om
import paper_2601_14327_amd as laep
from workloads import WORKLOADS, cached
from _gpu import TOL_BF16, TOL_F32, case, check_routing, dev, rownorm_err

pytestmark = pytest.mark.gpu
BF = torch.bfloat16


def h32(t):
    return t.detach().float().cpu().numpy()


def hint(t):
    return t.detach().cpu().numpy()


def _block_rows(offsets, block=32, seed=0):
    """One random row from every `block`-row block of every expert's rows
    (blocks start at the expert's first row, as its row tiles do), plus
    each expert's last row."""
    rng = np.random.default_rng(seed)
    rows = []
    for e in range(len(offsets) - 1):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        for b in range(lo, hi, block):
            rows.append(int(rng.integers(b, min(b + block, hi))))
        if hi > lo:
            rows.append(hi - 1)
    return np.unique(np.array(rows, np.int64))


def _expert_of_rows(rows, offsets):
    return np.searchsorted(offsets, rows, side="right") - 1


def _check_ffn_rows(plan, c, rows, w_gu_h, w_d_h):
    offsets = hint(plan.offsets).astype(np.int64)
    xp = h32(plan.x_perm[torch.from_numpy(rows).cuda()])
    y = h32(plan.y_perm[torch.from_numpy(rows).cuda()])
    act = h32(plan.act_save[torch.from_numpy(rows).cuda()])
    ex = _expert_of_rows(rows, offsets)
    ry = np.zeros_like(y, dtype=np.float64)
    ract = np.zeros_like(act, dtype=np.float64)
    for e in np.unique(ex):
        sel = ex == e
        ry[sel], ract[sel], _ = om.expert_ffn(xp[sel], w_gu_h[e], w_d_h[e], "bf16")
    assert rownorm_err(y, ry) <= TOL_BF16
    assert rownorm_err(act, ract) <= TOL_BF16


def _check_combine_tokens(plan, toks):
    k = plan.k
    dest = hint(plan.dest_row).reshape(-1, k)[toks]
    gate = hint(plan.topk_gate)[toks]
    rows = np.unique(dest[dest >= 0]).astype(np.int64)
    remap = {int(r): i for i, r in enumerate(rows)}
    y = h32(plan.y_perm[torch.from_numpy(rows).cuda()])
    dloc = np.vectorize(lambda r: remap.get(int(r), -1))(dest).reshape(-1)
    ref = om.combine(y, gate, dloc, k, dtype="bf16")
    assert rownorm_err(h32(plan.out)[toks], ref) <= TOL_BF16


def _routed_plan(name):
    w = WORKLOADS[name]
    c = cached(name)
    plan = laep.MoELayerPlan(w.T, w.d_model, w.E, w.k, w.d_ff, dtype=BF, device="cuda",
                             save_act=True)
    x, wr = dev(c["x"], BF), dev(c["w_router"], BF)
    wgu, wd = dev(c["w_gate_up"], BF), dev(c["w_down"], BF)
    bias = dev(c["bias"], torch.float32) if "bias" in c else None
    return w, c, plan, x, wr, wgu, wd, bias


@pytest.mark.parametrize("name", ["balanced", "skewed", "skewed_mild"])
def test_router_layer_full_size(name):
    w, c, plan, x, wr, wgu, wd, bias = _routed_plan(name)
    case(f"full-size layer {name}: first routing pass")
    plan.route(x, wr, bias=bias, renorm=w.renorm)
    plan.count()
    torch.cuda.synchronize()
    ridx, rgate, margin, rlog = om.route(c["x"], c["w_router"], w.k, bias=c.get("bias"),
                                        renorm=w.renorm)
    idx = hint(plan.topk_idx)
    n_diff, _ = check_routing(idx, hint(plan.topk_gate), ridx, rgate, rlog, w.k,
                              renorm=w.renorm, label=f"full-size {name}, first pass")
    print(f"  near-tie tokens routed differently: {n_diff} of {w.T}")
    rc, ro, rd = om.expert_counts(idx, w.E)
    np.testing.assert_array_equal(hint(plan.counts), rc)
    np.testing.assert_array_equal(hint(plan.offsets), ro)
    np.testing.assert_array_equal(hint(plan.dest_row), rd)
    alive = None
    if w.prune_beta is not None:
        case(f"full-size layer {name}: prune + second routing pass")
        plan.prune(w.prune_beta, w.prune_alpha)
        plan.route(x, wr, bias=bias, alive=plan.alive, renorm=w.renorm)
        plan.count()
        torch.cuda.synchronize()
        ra, rn, _ = ol.prune_mask(rc, w.T * w.k, w.prune_alpha, w.prune_beta)
        alive = hint(plan.alive).astype(bool)
        np.testing.assert_array_equal(alive, ra)
        assert int(hint(plan.n_pruned)[0]) == rn
        print(f"  pruned {rn} of {w.E} experts (beta={w.prune_beta})")
        ridx, rgate, margin, rlog = om.route(c["x"], c["w_router"], w.k, bias=c.get("bias"),
                                            alive=alive, renorm=w.renorm)
        idx = hint(plan.topk_idx)
        check_routing(idx, hint(plan.topk_gate), ridx, rgate, rlog, w.k, alive,
                      renorm=w.renorm, label=f"full-size {name}, after pruning")
        rc, ro, rd = om.expert_counts(idx, w.E)
        np.testing.assert_array_equal(hint(plan.counts), rc)
        np.testing.assert_array_equal(hint(plan.dest_row), rd)
        assert np.all(rc[~alive] == 0)
    case(f"full-size layer {name}: permute / FFN / combine")
    plan.experts_and_combine(x, wgu, wd)
    torch.cuda.synchronize()
    # permute is a copy: check every row
    src = np.empty(w.T * w.k, np.int64)
    src[rd] = np.arange(w.T * w.k) // w.k
    xp = plan.x_perm.view(torch.int16).cpu().numpy()
    xs = x.view(torch.int16).cpu().numpy()
    assert np.array_equal(xp, xs[src])
    rows = _block_rows(ro)
    _check_ffn_rows(plan, c, rows, c["w_gate_up"], c["w_down"])
    toks = np.random.default_rng(1).choice(w.T, 2048, replace=False)
    _check_combine_tokens(plan, toks)


def _shard_plan(name, backward=False):
    w = WORKLOADS[name]
    c = cached(name)
    plan = laep.MoELayerPlan(w.T, w.d_model, w.E, w.k, w.d_ff, dtype=BF, device="cuda",
                             backward=backward, save_act=True)
    x = dev(c["x"], BF)
    wgu, wd = dev(c["w_gate_up"], BF), dev(c["w_down"], BF)
    idx = dev(c["topk_idx"], torch.int32)
    gate = dev(c["topk_gate"], torch.float32)
    return w, c, plan, x, wgu, wd, idx, gate


def test_shard_forward_full_size():
    w, c, plan, x, wgu, wd, idx, gate = _shard_plan("shard")
    case("full-size expert shard forward (16 experts, d=4096, f=2048, 32768 rows)")
    plan.forward_given_routing(x, idx, gate, wgu, wd)
    torch.cuda.synchronize()
    rc, ro, rd = om.expert_counts(c["topk_idx"], w.E)
    np.testing.assert_array_equal(hint(plan.counts), rc)
    np.testing.assert_array_equal(hint(plan.dest_row), rd)
    print(f"  rows per expert: {sorted(rc.tolist())}")
    rows = _block_rows(ro, seed=3)
    _check_ffn_rows(plan, c, rows, c["w_gate_up"], c["w_down"])
    toks = np.random.default_rng(2).choice(w.T, 2048, replace=False)
    _check_combine_tokens(plan, toks)


def test_shard_backward_full_size():
    w, c, plan, x, wgu, wd, idx, gate = _shard_plan("shard_bwd", backward=True)
    case("full-size expert shard forward + backward")
    out_fwd = plan.forward_given_routing(x, idx, gate, wgu, wd).clone()
    # k = 1: the combine is folded into the FFN call; it must equal moe_combine
    assert plan.fused_combine and plan.y_perm is not None
    ref_out = laep.moe_combine(plan.y_perm, plan.topk_gate, plan.dest_row)
    dout = dev(c["dout"], BF)
    plan.backward(dout, wgu, wd)
    torch.cuda.synchronize()
    assert torch.equal(out_fwd, ref_out)
    R, d, f = w.T, w.d_model, w.d_ff
    offsets = hint(plan.offsets).astype(np.int64)
    dest = hint(plan.dest_row)
    g = hint(plan.topk_gate)[:, 0].astype(np.float64)
    rng = np.random.default_rng(5)
    # combine backward on sampled routed rows
    toks = rng.choice(R, 512, replace=False)
    rows = dest[toks].astype(np.int64)
    tr = torch.from_numpy(rows).cuda()
    y = h32(plan.y_perm[tr]).astype(np.float64)
    dq = h32(dout[torch.from_numpy(toks).cuda()]).astype(np.float64)
    ref_dg = np.einsum("ij,ij->i", dq, y)
    cond = np.abs(dq * y).sum(1)
    assert np.all(np.abs(hint(plan.dgate)[toks, 0] - ref_dg) <= TOL_F32 * cond)
    from oracle.numerics import round_bf16
    # the plan keeps no dy_perm (the expert backward forms dY on load): the
    # combine backward's dY, for the checks, from a separate call
    assert plan.dy_perm is None
    dyp, _ = laep.moe_combine_bwd(dout, plan.y_perm, plan.topk_gate, plan.dest_row)
    assert rownorm_err(h32(dyp[tr]), round_bf16(g[toks, None] * dq)) <= TOL_BF16
    # dgrad on sampled rows, teacher-forced on the GPU's act_save / dY / dA; the
    # plan hands the backward the forward's H, so the H_b buffer keeps dH
    dA_ws, dh_ws = laep.ffn_bwd_ws_views(plan.ws_bwd, R, f, BF)
    h_fwd = laep.ffn_fwd_h_view(plan.ws_ffn, R, f, BF)
    # the plan keeps no x_perm (the weight gradient gathers the token rows):
    # the dispatched rows, for the checks, by indexing here
    assert plan.x_perm is None
    xg = x[(plan.row_src.long() // w.k)]
    srows = _block_rows(offsets, seed=6)
    ts = torch.from_numpy(srows).cuda()
    ex = _expert_of_rows(srows, offsets)
    dy_s, act_s = h32(dyp[ts]), h32(plan.act_save[ts])
    dA_s, dh_s, dx_s = h32(dA_ws[ts]), h32(dh_ws[ts]), h32(plan.dx_perm[ts])
    xp_s, h_s = h32(xg[ts]), h32(h_fwd[ts])
    for e in np.unique(ex):
        sel = ex == e
        dH = dy_s[sel].astype(np.float64) @ c["w_down"][e].astype(np.float64)
        assert rownorm_err(dh_s[sel], round_bf16(dH)) <= TOL_BF16
        rdA, _ = om.swiglu_bwd(dH, act_s[sel], "bf16")
        assert rownorm_err(dA_s[sel], rdA) <= TOL_BF16
        rdx = round_bf16(dA_s[sel].astype(np.float64) @ c["w_gate_up"][e].astype(np.float64))
        assert rownorm_err(dx_s[sel], rdx) <= TOL_BF16
        _, _, rh = om.expert_ffn(xp_s[sel], c["w_gate_up"][e], c["w_down"][e], "bf16")
        assert rownorm_err(h_s[sel], rh) <= TOL_BF16
    # wgrad, teacher-forced on the GPU's dA / forward H: per expert one whole
    # 256 x 256 output tile of dW_gu and of dW_d, and three full output rows
    case("full-size wgrad checks")
    dwgu, dwd = plan.dw_gate_up, plan.dw_down
    TB = 256
    for e in range(w.E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi == lo:
            continue
        i0, j0 = TB * int(rng.integers(2 * f // TB)), TB * int(rng.integers(d // TB))
        dA_t = h32(dA_ws[lo:hi, i0:i0 + TB]).astype(np.float64)
        x_t = h32(xg[lo:hi, j0:j0 + TB]).astype(np.float64)
        assert rownorm_err(h32(dwgu[e, i0:i0 + TB, j0:j0 + TB]), dA_t.T @ x_t) <= TOL_F32, e
        i0, j0 = TB * int(rng.integers(d // TB)), TB * int(rng.integers(f // TB))
        dy_t = h32(dyp[lo:hi, i0:i0 + TB]).astype(np.float64)
        h_t = h32(h_fwd[lo:hi, j0:j0 + TB]).astype(np.float64)
        assert rownorm_err(h32(dwd[e, i0:i0 + TB, j0:j0 + TB]), dy_t.T @ h_t) <= TOL_F32, e
        tr = torch.arange(lo, hi, device="cuda")
        i_d = rng.choice(d, 3, replace=False)
        i_g = rng.choice(2 * f, 3, replace=False)
        dy_e = h32(dyp[tr][:, torch.from_numpy(i_d).cuda()]).astype(np.float64)
        h_e = h32(h_fwd[tr]).astype(np.float64)
        ref_d = dy_e.T @ h_e
        assert rownorm_err(h32(dwd[e][torch.from_numpy(i_d).cuda()]), ref_d) <= TOL_F32
        dA_e = h32(dA_ws[tr][:, torch.from_numpy(i_g).cuda()]).astype(np.float64)
        x_e = h32(xg[tr]).astype(np.float64)
        ref_g = dA_e.T @ x_e
        assert rownorm_err(h32(dwgu[e][torch.from_numpy(i_g).cuda()]), ref_g) <= TOL_F32
    # permute backward (k = 1: a gather back to token order)
    dx_tok = h32(plan.dx[torch.from_numpy(toks).cuda()])
    assert np.array_equal(dx_tok, h32(plan.dx_perm[torch.from_numpy(rows).cuda()]))
    # the fused backward (gathered X, dY on load) equals the unfused chain bit for bit
    case("full-size fused backward vs the unfused chain (shard_bwd)")
    dxp_u, dwgu_u, dwd_u = laep.moe_grouped_ffn_bwd(dyp, xg, plan.act_save, wgu, wd,
                                                    plan.offsets, h_fwd=h_fwd)
    torch.cuda.synchronize()
    assert torch.equal(dxp_u, plan.dx_perm)
    assert torch.equal(dwgu_u, plan.dw_gate_up) and torch.equal(dwd_u, plan.dw_down)


@pytest.mark.parametrize("name", ["balanced", "shard"])
def test_fused_dispatch_matches_unfused_full_size(name):
    """The forward-only plan folds the dispatch into the FFN's operand loads
    (and, with one slot per token, the combine into its epilogue); its outputs
    must equal the permute + FFN + combine chain's bit for bit."""
    w = WORKLOADS[name]
    c = cached(name)
    x = dev(c["x"], BF)
    wgu, wd = dev(c["w_gate_up"], BF), dev(c["w_down"], BF)
    pf = laep.MoELayerPlan(w.T, w.d_model, w.E, w.k, w.d_ff, dtype=BF, device="cuda")
    pu = laep.MoELayerPlan(w.T, w.d_model, w.E, w.k, w.d_ff, dtype=BF, device="cuda",
                           fused_dispatch=False)
    assert pf.fused and not pu.fused
    case(f"full-size fused vs unfused dispatch ({name})")
    if w.routed:
        wr = dev(c["w_router"], BF)
        of = pf.forward(x, wr, wgu, wd, renorm=w.renorm)
        ou = pu.forward(x, wr, wgu, wd, renorm=w.renorm)
    else:
        idx = dev(c["topk_idx"], torch.int32)
        gate = dev(c["topk_gate"], torch.float32)
        of = pf.forward_given_routing(x, idx, gate, wgu, wd)
        ou = pu.forward_given_routing(x, idx, gate, wgu, wd)
    torch.cuda.synchronize()
    if pf.fused_combine:   # k = 1: the combine is folded in too, y_perm never written
        assert pf.y_perm is None
    else:
        assert torch.equal(pf.y_perm, pu.y_perm)
    assert torch.equal(of, ou)


def test_routed_training_step_full_size():
    """balanced_bwd: forward, the expert backward, then the router backward
    accumulated onto dx; the router part is checked against the oracle,
    teacher-forced on the GPU's routing, gate gradient and expert-path dx."""
    w = WORKLOADS["balanced_bwd"]
    c = cached("balanced_bwd")
    x, wr = dev(c["x"], BF), dev(c["w_router"], BF)
    wgu, wd = dev(c["w_gate_up"], BF), dev(c["w_down"], BF)
    dout = dev(c["dout"], BF)
    plan = laep.MoELayerPlan(w.T, w.d_model, w.E, w.k, w.d_ff, dtype=BF, device="cuda",
                             backward=True)
    case("full-size routed training step (balanced_bwd)")
    plan.forward(x, wr, wgu, wd, renorm=w.renorm)
    assert plan.x_perm is None      # the weight gradient gathers the token rows
    plan.backward(dout, wgu, wd)
    torch.cuda.synchronize()
    dx_expert = h32(plan.dx)
    # the gathered backward equals the permute + unfused backward bit for bit
    case("full-size fused backward (gathered X, dY on load) vs permute + combine_bwd's dY + "
         "unfused backward (balanced_bwd)")
    xp = laep.moe_permute(x, plan.dest_row, w.k, plan.R)
    h_fwd = laep.ffn_fwd_h_view(plan.ws_ffn, plan.R, w.d_ff, BF)
    dyp, _ = laep.moe_combine_bwd(dout, plan.y_perm, plan.topk_gate, plan.dest_row)
    dxp, dwgu_u, dwd_u = laep.moe_grouped_ffn_bwd(dyp, xp, plan.act_save, wgu, wd,
                                                  plan.offsets, h_fwd=h_fwd)
    torch.cuda.synchronize()
    assert torch.equal(dxp, plan.dx_perm)
    assert torch.equal(dwgu_u, plan.dw_gate_up) and torch.equal(dwd_u, plan.dw_down)
    del xp, dyp, dxp, dwgu_u, dwd_u
    plan.route_backward(x, wr, renorm=w.renorm, want_dbias=True)
    torch.cuda.synchronize()
    rl, rw, rb, rx = om.route_bwd(hint(plan.dgate).astype(np.float64), hint(plan.topk_idx),
                                  hint(plan.topk_gate).astype(np.float64), c["x"], c["w_router"],
                                  renorm=True, dtype="bf16", dx_in=dx_expert)
    assert rownorm_err(hint(plan.dw_router), rw) <= TOL_F32
    assert rownorm_err(hint(plan.dbias), rb) <= TOL_F32
    assert rownorm_err(h32(plan.dx), rx) <= TOL_BF16
    # the training step with the router's weight gradients on a side stream,
    # beside the expert backward: the same bits
    dx_seq, dw_seq, db_seq = plan.dx.clone(), plan.dw_router.clone(), plan.dbias.clone()
    dwd_seq = plan.dw_down.clone()
    case("full-size routed training step, router weight gradients beside the expert backward")
    plan.forward(x, wr, wgu, wd, renorm=w.renorm)
    plan.backward(dout, wgu, wd, router=(x, wr), want_dbias=True)
    torch.cuda.synchronize()
    assert torch.equal(plan.dx, dx_seq)
    assert torch.equal(plan.dw_router, dw_seq) and torch.equal(plan.dbias, db_seq)
    assert torch.equal(plan.dw_down, dwd_seq)


def test_pruned_compact_layer_full_size():
    """mild_pruned: Algorithm 1 over a window of routed batches, the pruned
    experts removed, and the compact layer run at full size against the
    oracle of the survivors."""
    w = WORKLOADS["mild_pruned"]
    c = cached("mild_pruned")
    x, wr = dev(c["x"], BF), dev(c["w_router"], BF)
    wgu, wd = dev(c["w_gate_up"], BF), dev(c["w_down"], BF)
    bias = dev(c["bias"], torch.float32)
    rng = np.random.default_rng(0)
    perms = [np.arange(w.T)] + [rng.permutation(w.T) for _ in range(w.prune_window - 1)]
    pruner = laep.ExpertPruner(w.prune_window, 1, w.E, w.T, w.k, alpha=w.prune_alpha,
                               beta=w.prune_beta)
    case("full-size pruned layer: window")
    for it, pm in enumerate(perms):
        idx, _ = laep.moe_route(x[torch.from_numpy(pm).cuda()], wr, w.k, bias=bias)
        laep.moe_expert_counts(idx, w.E, etn_accum=pruner.slot(it, 0))
    alive, n_pruned, _ = pruner.decide()
    torch.cuda.synchronize()
    # the window's loads are the oracle's counts of the device routing of x
    idx0, _ = laep.moe_route(x, wr, w.k, bias=bias)
    rc, _, _ = om.expert_counts(hint(idx0), w.E)
    np.testing.assert_array_equal(hint(pruner.etn)[:, 0], np.stack([rc] * w.prune_window))
    pruned = ol.expert_pruning(hint(pruner.etn), w.T, w.k, w.prune_alpha, w.prune_beta)[0]
    a = hint(alive)[0].astype(bool)
    assert np.nonzero(~a)[0].tolist() == pruned.tolist()
    print(f"  pruned {len(pruned)} of {w.E} experts")
    case("full-size pruned layer: compact + forward")
    small = laep.compact_layer(alive[0].contiguous(), w_router=wr, w_gate_up=wgu, w_down=wd,
                               bias=bias)
    E2 = small["n_alive"]
    keep = np.nonzero(a)[0]
    assert E2 == len(keep)
    plan = laep.MoELayerPlan(w.T, w.d_model, E2, w.k, w.d_ff, dtype=BF, device="cuda",
                             save_act=True)
    plan.route(x, small["w_router"], bias=small["bias"], renorm=w.renorm)
    plan.count()
    plan.experts_and_combine(x, small["w_gate_up"], small["w_down"])
    torch.cuda.synchronize()
    ridx, rgate, _, rlog = om.route(c["x"], c["w_router"][keep], w.k, bias=c["bias"][keep],
                                    renorm=w.renorm)
    idx = hint(plan.topk_idx)
    check_routing(idx, hint(plan.topk_gate), ridx, rgate, rlog, w.k, renorm=w.renorm,
                  label="full-size mild_pruned, compact layer")
    rc2, ro2, rd2 = om.expert_counts(idx, E2)
    np.testing.assert_array_equal(hint(plan.counts), rc2)
    np.testing.assert_array_equal(hint(plan.dest_row), rd2)
    rows = _block_rows(ro2)
    _check_ffn_rows(plan, c, rows, c["w_gate_up"][keep], c["w_down"][keep])
    toks = np.random.default_rng(2).choice(w.T, 2048, replace=False)
    _check_combine_tokens(plan, toks)
