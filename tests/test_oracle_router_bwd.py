"""Pins of the oracle's router backward (oracle.moe.route_bwd): torch autograd
through an independent float64 forward of the router and gates, the zero-sum
property of a softmax Jacobian, special cases, and central differences."""
import numpy as np
import pytest
import torch

import oracle.moe as om
from oracle.numerics import round_f32


def _case(seed, T=37, d=24, E=9, k=3, alive=None):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, d))
    w = rng.standard_normal((E, d)) * 0.3
    b = rng.standard_normal(E) * 0.5
    dg = rng.standard_normal((T, k))
    logits = om.router_logits(x, w, b)
    idx, _, margin = om.topk_gating(logits, k, alive=alive, renorm=True)
    return x, w, b, dg, idx


def _autograd(x, w, b, dg, idx, renorm, alive=None):
    """float64 forward of the gates with the selection fixed, and autograd."""
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    logits = xt @ wt.T + bt
    logits.retain_grad()
    it = torch.tensor(np.where(idx >= 0, idx, 0), dtype=torch.long)
    ok = torch.tensor(idx >= 0)
    if renorm:
        sel = torch.gather(logits, 1, it).masked_fill(~ok, float("-inf"))
        g = torch.softmax(sel, dim=1).masked_fill(~ok, 0.0)
    else:
        a = torch.ones(w.shape[0], dtype=torch.bool) if alive is None else torch.tensor(alive)
        p = torch.softmax(logits.masked_fill(~a[None, :], float("-inf")), dim=1)
        g = torch.gather(p, 1, it).masked_fill(~ok, 0.0)
    (g * torch.tensor(dg)).sum().backward()
    return (g.detach().numpy(), logits.grad.numpy(), wt.grad.numpy(), bt.grad.numpy(),
            xt.grad.numpy())


def _close(a, b, rtol=2e-6):
    scale = max(float(np.abs(b).max()), 1e-30)
    assert float(np.abs(np.asarray(a) - np.asarray(b)).max()) <= rtol * scale


@pytest.mark.parametrize("renorm", [True, False])
@pytest.mark.parametrize("seed", [1, 2, 3])
def test_router_bwd_matches_autograd(renorm, seed):
    x, w, b, dg, idx = _case(seed)
    g, dl_ref, dw_ref, db_ref, dx_ref = _autograd(x, w, b, dg, idx, renorm)
    logits = om.router_logits(x, w, b)
    dl, dw, db, dx = om.route_bwd(dg, idx, g, x, w, logits=logits, renorm=renorm, dtype="f64")
    _close(dl, dl_ref)
    _close(dw, dw_ref)
    _close(db, db_ref)
    _close(dx, dx_ref)


def test_router_bwd_dead_experts_and_unrouted_slots():
    alive = np.ones(9, bool)
    alive[[2, 5, 6, 7, 8]] = False                   # 4 alive, k = 5: one slot unroutable
    x, w, b, dg, idx = _case(7, k=5, alive=alive)
    assert np.all(idx[:, 4] == -1)
    for renorm in (True, False):
        g, dl_ref, dw_ref, db_ref, dx_ref = _autograd(x, w, b, dg, idx, renorm, alive=alive)
        dl, dw, db, dx = om.route_bwd(dg, idx, g, x, w, logits=om.router_logits(x, w, b),
                                      alive=alive, renorm=renorm, dtype="f64")
        assert np.all(dl[:, ~alive] == 0)
        _close(dl, dl_ref)
        _close(dw, dw_ref)
        _close(dx, dx_ref)


@pytest.mark.parametrize("renorm", [True, False])
def test_softmax_jacobian_rows_sum_to_zero(renorm):
    x, w, b, dg, idx = _case(11, T=64, E=16, k=4)
    logits = om.router_logits(x, w, b)
    _, gate, _ = om.topk_gating(logits, 4, renorm=renorm)
    dl, _, db, _ = om.route_bwd(dg, idx, gate, x, w, logits=logits, renorm=renorm, dtype="f64")
    assert np.abs(dl.sum(axis=1)).max() <= 1e-6 * np.abs(dl).max()


def test_top1_renormalised_gate_is_constant():
    x, w, b, dg, idx = _case(5, k=1)
    g = np.ones((x.shape[0], 1))
    dx_in = np.random.default_rng(0).standard_normal(x.shape)
    dl, dw, db, dx = om.route_bwd(dg, idx, g, x, w, renorm=True, dtype="f64", dx_in=dx_in)
    assert np.all(dl == 0) and np.all(dw == 0) and np.all(db == 0)
    np.testing.assert_array_equal(dx, dx_in)


@pytest.mark.parametrize("renorm", [True, False])
def test_router_bwd_central_differences(renorm):
    x, w, b, dg, idx = _case(13, T=20, d=10, E=6, k=2)

    def loss(x_, w_, b_):
        l = x_ @ w_.T + b_
        if renorm:
            sel = np.take_along_axis(l, idx, axis=1)
            e = np.exp(sel - sel.max(axis=1, keepdims=True))
            g = e / e.sum(axis=1, keepdims=True)
        else:
            e = np.exp(l - l.max(axis=1, keepdims=True))
            g = np.take_along_axis(e / e.sum(axis=1, keepdims=True), idx, axis=1)
        return float((g * dg).sum())

    logits = om.router_logits(x, w, b)
    _, gate, _ = om.topk_gating(logits, 2, renorm=renorm, decide_f32=False)
    g_exact = _autograd(x, w, b, dg, idx, renorm)[0]
    dl, dw, db, dx = om.route_bwd(dg, idx, g_exact, x, w, logits=logits, renorm=renorm,
                                  dtype="f64")
    h = 1e-6
    rng = np.random.default_rng(3)
    for _ in range(6):
        e, c = rng.integers(6), rng.integers(10)
        wp, wm = w.copy(), w.copy()
        wp[e, c] += h
        wm[e, c] -= h
        fd = (loss(x, wp, b) - loss(x, wm, b)) / (2 * h)
        assert abs(fd - dw[e, c]) <= 1e-5 * max(1.0, abs(fd))
        t, c = rng.integers(20), rng.integers(10)
        xp, xm = x.copy(), x.copy()
        xp[t, c] += h
        xm[t, c] -= h
        fd = (loss(xp, w, b) - loss(xm, w, b)) / (2 * h)
        assert abs(fd - dx[t, c]) <= 1e-5 * max(1.0, abs(fd))
        e = rng.integers(6)
        bp, bm = b.copy(), b.copy()
        bp[e] += h
        bm[e] -= h
        fd = (loss(x, w, bp) - loss(x, w, bm)) / (2 * h)
        assert abs(fd - db[e]) <= 1e-5 * max(1.0, abs(fd))
