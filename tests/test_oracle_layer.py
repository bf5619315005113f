"""Pins of the oracle's permute / grouped FFN / combine and their backward.

Closed forms (shared experts reduce the layer to a dense SwiGLU FFN scaled
by the sum of gates), an independent dense evaluation in torch CPU float64,
torch autograd for the SwiGLU backward, and central finite differences of
the whole layer in float64.
"""
import numpy as np
import pytest
import torch

from oracle import moe
from oracle.numerics import round_bf16


def _dense_swiglu_torch(x, w_gu, w_d):
    """Dense SwiGLU in torch float64, written independently of the oracle."""
    x = torch.tensor(x, dtype=torch.float64)
    wg = torch.tensor(w_gu, dtype=torch.float64)
    wd = torch.tensor(w_d, dtype=torch.float64)
    f = wd.shape[1]
    gate = torch.nn.functional.linear(x, wg[:f])
    up = torch.nn.functional.linear(x, wg[f:])
    return torch.nn.functional.linear(torch.nn.functional.silu(gate) * up, wd).numpy()


def _case(seed, T=40, d=24, E=5, k=2, f=16):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, d))
    w_r = rng.standard_normal((E, d)) * 0.3
    w_gu = rng.standard_normal((E, 2 * f, d)) * 0.2
    w_d = rng.standard_normal((E, d, f)) * 0.2
    return x, w_r, w_gu, w_d


@pytest.mark.parametrize("renorm", [True, False])
def test_shared_experts_equal_dense_ffn_times_gate_sum(renorm):
    x, w_r, w_gu, w_d = _case(1)
    E, k = w_r.shape[0], 2
    w_gu[:] = w_gu[0]
    w_d[:] = w_d[0]
    res = moe.layer_forward(x, w_r, w_gu, w_d, k, renorm=renorm, dtype="f64")
    dense = _dense_swiglu_torch(x, w_gu[0], w_d[0])
    gsum = res["gate"].sum(axis=1, keepdims=True)
    np.testing.assert_allclose(res["out"], dense * gsum, rtol=1e-11, atol=1e-13)
    if renorm:
        np.testing.assert_allclose(gsum, 1.0, atol=1e-6)
    else:
        assert np.all(gsum < 1.0)       # top-2 of a softmax over 5 experts


def test_single_expert_is_dense_ffn():
    x, w_r, w_gu, w_d = _case(2, E=1)
    res = moe.layer_forward(x, w_r, w_gu, w_d, 1, renorm=True, dtype="f64")
    np.testing.assert_allclose(res["out"], _dense_swiglu_torch(x, w_gu[0], w_d[0]),
                               rtol=1e-12, atol=1e-13)


def test_per_expert_rows_use_their_own_expert():
    x, w_r, w_gu, w_d = _case(3, T=30, E=4, k=2)
    res = moe.layer_forward(x, w_r, w_gu, w_d, 2, dtype="f64")
    for t in range(30):
        want = sum(res["gate"][t, j] * _dense_swiglu_torch(x[t:t + 1], w_gu[e], w_d[e])[0]
                   for j, e in enumerate(res["idx"][t]))
        np.testing.assert_allclose(res["out"][t], want, rtol=1e-11, atol=1e-13)


def test_identity_ffn_combine_is_x_times_gate_sum():
    rng = np.random.default_rng(9)
    T, d, E, k = 25, 16, 6, 3
    x = rng.standard_normal((T, d))
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    gate = rng.uniform(0.05, 1, (T, k))
    counts, offsets, dest = moe.expert_counts(idx, E)
    xp = moe.permute(x, dest, k)
    out = moe.combine(xp, gate, dest, k, dtype="f64")
    np.testing.assert_allclose(out, x * gate.sum(1, keepdims=True), rtol=1e-14)
    # permute_bwd of the permuted rows gives k copies back
    np.testing.assert_allclose(moe.permute_bwd(xp, dest, k, dtype="f64"), k * x, rtol=1e-14)


def test_bf16_rounding_points():
    x, w_r, w_gu, w_d = _case(4)
    x, w_gu, w_d = round_bf16(x), round_bf16(w_gu), round_bf16(w_d)
    res = moe.layer_forward(x, w_r, w_gu, w_d, 2, dtype="bf16")
    for key in ("out", "y_perm", "act_save"):
        assert np.array_equal(res[key], round_bf16(res[key])), key
    ref = moe.layer_forward(x, w_r, w_gu, w_d, 2, dtype="f64")
    np.testing.assert_allclose(res["out"], ref["out"], rtol=3e-2, atol=3e-3)


def test_swiglu_bwd_against_autograd():
    rng = np.random.default_rng(6)
    act = rng.standard_normal((9, 2 * 7)) * 2
    dH = rng.standard_normal((9, 7))
    dA, Hb = moe.swiglu_bwd(dH, act, dtype="f64")
    a = torch.tensor(act, requires_grad=True)
    f = 7
    h = torch.nn.functional.silu(a[:, :f]) * a[:, f:]
    h.backward(torch.tensor(dH))
    np.testing.assert_allclose(dA, a.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(Hb, h.detach().numpy(), rtol=1e-14)


def _loss(x, gate, w_gu, w_d, dest, offsets, k, dout):
    xp = moe.permute(x, dest, k)
    y, _ = moe.grouped_ffn_fwd(xp, w_gu, w_d, offsets, dtype="f64")
    out = moe.combine(y, gate, dest, k, dtype="f64")
    return float((out * dout).sum())


def test_backward_finite_differences():
    rng = np.random.default_rng(8)
    T, d, E, k, f = 12, 8, 3, 2, 6
    x = rng.standard_normal((T, d))
    w_gu = rng.standard_normal((E, 2 * f, d)) * 0.4
    w_d = rng.standard_normal((E, d, f)) * 0.4
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    gate = rng.uniform(0.1, 1, (T, k))
    dout = rng.standard_normal((T, d))
    counts, offsets, dest = moe.expert_counts(idx, E)

    xp = moe.permute(x, dest, k)
    y, act = moe.grouped_ffn_fwd(xp, w_gu, w_d, offsets, dtype="f64")
    dy, dgate = moe.combine_bwd(dout, y, gate, dest, k, dtype="f64")
    dxp, dA, Hb = moe.grouped_ffn_dgrad(dy, act, w_gu, w_d, offsets, dtype="f64")
    dw_gu, dw_d = moe.grouped_ffn_wgrad(dy, xp, dA, Hb, offsets, E, out_f32=False)
    dx = moe.permute_bwd(dxp, dest, k, dtype="f64")

    h = 1e-6
    L = lambda **kw: _loss(**{**dict(x=x, gate=gate, w_gu=w_gu, w_d=w_d, dest=dest,
                                     offsets=offsets, k=k, dout=dout), **kw})

    def fd(name, arr, index):
        p, m = arr.copy(), arr.copy()
        p[index] += h
        m[index] -= h
        return (L(**{name: p}) - L(**{name: m})) / (2 * h)

    for index in [(0, 0), (5, 3), (11, 7)]:
        assert abs(fd("x", x, index) - dx[index]) < 1e-7
    for index in [(0, 0), (7, 1), (11, 1)]:
        assert abs(fd("gate", gate, index) - dgate[index]) < 1e-7
    for index in [(0, 0, 0), (1, 5, 3), (2, 11, 7), (1, 6, 2)]:
        assert abs(fd("w_gu", w_gu, index) - dw_gu[index]) < 1e-7
    for index in [(0, 0, 0), (1, 3, 5), (2, 7, 2)]:
        assert abs(fd("w_d", w_d, index) - dw_d[index]) < 1e-7


def test_k1_gate_gradient_identity():
    """For k = 1: sum_r dgate[r] * g[r] = <dout, out>."""
    rng = np.random.default_rng(10)
    T, d, E, f = 30, 8, 4, 6
    x = rng.standard_normal((T, d))
    w_gu = rng.standard_normal((E, 2 * f, d)) * 0.3
    w_d = rng.standard_normal((E, d, f)) * 0.3
    idx = rng.integers(0, E, size=(T, 1))
    gate = rng.uniform(0.05, 1, (T, 1))
    dout = rng.standard_normal((T, d))
    counts, offsets, dest = moe.expert_counts(idx, E)
    xp = moe.permute(x, dest, 1)
    y, _ = moe.grouped_ffn_fwd(xp, w_gu, w_d, offsets, dtype="f64")
    out = moe.combine(y, gate, dest, 1, dtype="f64")
    _, dgate = moe.combine_bwd(dout, y, gate, dest, 1, dtype="f64")
    assert abs((dgate * gate).sum() - (dout * out).sum()) < 1e-10


def test_shared_expert_weight_gradient_equals_dense_gradient():
    """Experts sharing one weight set: sum_e dW[e] is the dense gradient of
    sum_t <dout_t, sum_j g_tj FFN(x_t)>, evaluated by torch autograd."""
    rng = np.random.default_rng(12)
    T, d, E, k, f = 16, 8, 4, 2, 5
    x = rng.standard_normal((T, d))
    wg = rng.standard_normal((2 * f, d)) * 0.3
    wd = rng.standard_normal((d, f)) * 0.3
    w_gu = np.repeat(wg[None], E, 0)
    w_d = np.repeat(wd[None], E, 0)
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    gate = rng.uniform(0.1, 1, (T, k))
    dout = rng.standard_normal((T, d))
    counts, offsets, dest = moe.expert_counts(idx, E)
    xp = moe.permute(x, dest, k)
    y, act = moe.grouped_ffn_fwd(xp, w_gu, w_d, offsets, dtype="f64")
    dy, _ = moe.combine_bwd(dout, y, gate, dest, k, dtype="f64")
    dxp, dA, Hb = moe.grouped_ffn_dgrad(dy, act, w_gu, w_d, offsets, dtype="f64")
    dw_gu, dw_d = moe.grouped_ffn_wgrad(dy, xp, dA, Hb, offsets, E, out_f32=False)

    tx = torch.tensor(x)
    twg = torch.tensor(wg, requires_grad=True)
    twd = torch.tensor(wd, requires_grad=True)
    h = torch.nn.functional.silu(tx @ twg[:f].T) * (tx @ twg[f:].T)
    out = (h @ twd.T) * torch.tensor(gate.sum(1, keepdims=True))
    (out * torch.tensor(dout)).sum().backward()
    np.testing.assert_allclose(dw_gu.sum(0), twg.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dw_d.sum(0), twd.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_planted_mistakes_are_caught(monkeypatch):
    """A swapped gate/up or a dropped SiLU in the oracle fails the dense pin."""
    x, w_r, w_gu, w_d = _case(13, E=1)
    dense = _dense_swiglu_torch(x, w_gu[0], w_d[0])
    good = moe.layer_forward(x, w_r, w_gu, w_d, 1, dtype="f64")["out"]
    assert np.allclose(good, dense, rtol=1e-11)

    orig = moe.silu
    monkeypatch.setattr(moe, "silu", lambda a: np.asarray(a, np.float64))   # SiLU dropped
    bad = moe.layer_forward(x, w_r, w_gu, w_d, 1, dtype="f64")["out"]
    assert not np.allclose(bad, dense, rtol=1e-6)
    monkeypatch.setattr(moe, "silu", orig)

    swapped = np.concatenate([w_gu[:, 16:], w_gu[:, :16]], axis=1)
    bad = moe.layer_forward(x, w_r, swapped, w_d, 1, dtype="f64")["out"]
    assert not np.allclose(bad, dense, rtol=1e-6)
