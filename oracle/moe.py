"""Oracle of the MoE layer's data-parallel hot path (float64 NumPy).

Test infrastructure only; see the package docstring.

Notation (Section 3.2): E[i, j, l] = 1 iff token j of layer l is routed to
expert i.  For one layer and one batch, the load of expert i is
sum_j E[i, j, l] -- the left-hand side of Eq. (1) and the quantity recorded
as ETN in Step 1 of Algorithm 1 (Appendix).

The paper does not spell out the router, the gating function or the expert
FFN.  The readings used here:

* router: logits = x W_r^T (+ per-expert bias b when given);
* top-k: the k largest logits among the alive experts, ties to the lower
  expert index, slots in descending logit order; the decision is taken on
  logits rounded to float32 (the precision the kernels decide in);
* gates: renorm=True -> softmax over the k selected logits;
  renorm=False -> softmax over all alive experts, then the k selected;
* expert FFN: SwiGLU, y = W_d (silu(W_g x) * (W_u x)) -- three d x f
  matrices per expert, as the paper's parameter counts imply (Appendix,
  model-structure table);
* dropless routing: every token keeps its k routes, so the total load is
  S * topK as in Algorithm 1.  If fewer than k experts are alive, the
  unfillable slots hold expert -1 and gate 0 and are not routed.

Rounding points (the layer dtype "bf16" or "f32"; "f64" = none):
act_save = round(A); H = round(silu(A_g) * A_u) from the unrounded A;
Y = round(H W_d^T); out = round(sum_j g_j Y_j).  Backward: dY = round(g dout);
dH = dY W_d is kept unrounded into the SwiGLU backward; dA = round(.);
dX = round(dA W_gu).  The router backward keeps dlogits unrounded into
dW_r, db and dx.  Gates, dgate, dlogits and weight gradients are returned
as float32.
"""
from __future__ import annotations

import numpy as np

from .numerics import rounder, round_f32, round_bf16, silu, sigmoid

F64 = np.float64


# --------------------------------------------------------------------------
# Router scoring and top-k gating
# --------------------------------------------------------------------------
def router_logits(x, w_router, bias=None) -> np.ndarray:
    """logits[t, e] = sum_c x[t, c] * W_r[e, c] (+ b[e]), in float64."""
    logits = np.asarray(x, F64) @ np.asarray(w_router, F64).T
    if bias is not None:
        logits = logits + np.asarray(bias, F64)[None, :]
    return logits


def topk_gating(logits, k: int, alive=None, renorm: bool = True,
                decide_f32: bool = True):
    """Select the top-k alive experts per token and their gates.

    Returns (idx [T,k] int32, gate [T,k] float32-valued float64,
    margin [T] float64).  margin_t = l_(k) - l_(k+1) over alive experts
    (+inf when fewer than k+1 are alive); a margin near zero marks a
    near-tie, where a different but equally valid choice is possible.
    """
    logits = np.asarray(logits, F64)
    if decide_f32:
        logits = round_f32(logits)
    T, E = logits.shape
    alive = np.ones(E, bool) if alive is None else np.asarray(alive).astype(bool)
    masked = np.where(alive[None, :], logits, -np.inf)
    # stable sort of -logit: equal logits keep ascending expert order
    order = np.argsort(-masked, axis=1, kind="stable")
    n_alive = int(alive.sum())
    kk = min(k, n_alive)
    idx = np.full((T, k), -1, dtype=np.int32)
    idx[:, :kk] = order[:, :kk]
    sel = np.take_along_axis(masked, order[:, :kk], axis=1)
    gate = selection_gates(logits, idx, alive=alive, renorm=renorm, decide_f32=False)
    if n_alive > k:
        nxt = np.take_along_axis(masked, order[:, k:k + 1], axis=1)[:, 0]
        margin = sel[:, kk - 1] - nxt
    else:
        margin = np.full(T, np.inf)
    return idx, gate, margin


def selection_gates(logits, idx, alive=None, renorm: bool = True,
                    decide_f32: bool = True) -> np.ndarray:
    """Gates of a given selection idx [T, k] (slots holding -1 are empty and
    get gate 0), whether or not it is the top-k:

      renorm=True:  g_j = exp(l_j) / sum over the selected i of exp(l_i)
      renorm=False: g_j = exp(l_j) / sum over all alive e of exp(l_e)

    evaluated in float64 (shifted by the token's largest logit, which
    cancels) from the float32-rounded logits, and returned rounded to
    float32.  ``topk_gating`` takes its gates from here; a routing checker
    uses it to price an alternative selection at a near-tie.
    """
    logits = np.asarray(logits, F64)
    if decide_f32:
        logits = round_f32(logits)
    idx = np.asarray(idx)
    T, E = logits.shape
    alive = np.ones(E, bool) if alive is None else np.asarray(alive).astype(bool)
    masked = np.where(alive[None, :], logits, -np.inf)
    used = idx >= 0
    sel = np.where(used, np.take_along_axis(masked, np.where(used, idx, 0), axis=1), -np.inf)
    if renorm:
        top = np.max(sel, axis=1, keepdims=True)
        top = np.where(np.isfinite(top), top, 0.0)
        ex = np.where(used, np.exp(sel - top), 0.0)
        den = ex.sum(axis=1, keepdims=True)
    else:
        top = np.max(masked, axis=1, keepdims=True)
        top = np.where(np.isfinite(top), top, 0.0)
        ex = np.where(used, np.exp(sel - top), 0.0)
        den = np.where(alive[None, :], np.exp(masked - top), 0.0).sum(axis=1, keepdims=True)
    gate = ex / np.where(den > 0, den, 1.0)
    return round_f32(gate)


def route(x, w_router, k, bias=None, alive=None, renorm=True):
    """Router scoring followed by top-k gating; returns
    (idx, gate, margin, logits)."""
    logits = router_logits(x, w_router, bias)
    idx, gate, margin = topk_gating(logits, k, alive=alive, renorm=renorm)
    return idx, gate, margin, logits


def route_bwd(dgate, idx, gate, x, w_router, logits=None, alive=None, renorm: bool = True,
              dtype: str = "bf16", dx_in=None):
    """Backward of router scoring and gating with the selection held fixed
    (the top-k choice is piecewise constant in the logits, so no gradient
    flows through it).

    dl[t, e] = dLoss/dlogits[t, e] for dLoss/dgate[t, j] = dgate[t, j]:
      renorm:      the gates are a softmax over the k selected logits, so for
                   e = idx[t, j]:  dl = g_j (dg_j - sum_i g_i dg_i); 0 elsewhere.
      full softmax: the gates are p_e at the selected experts, p = softmax over
                   the alive logits; with q_e = dg_j at e = idx[t, j] (0 for
                   the other experts):  dl_e = p_e (q_e - sum_j g_j dg_j) for
                   alive e; 0 for dead ones.  Needs the logits.
    dW_r = dl^T x and db = sum_t dl (float32);
    dx = round_dtype(dx_in + dl W_r)  (dx_in = 0 when not given).
    Slots with idx = -1 carry no gradient.  dl enters dW_r, db and dx
    unrounded; it is returned rounded to float32 (the dlogits output).
    Returns (dl [T, E], dW_r [E, d], db [E], dx [T, d]).
    """
    dgate = np.asarray(dgate, F64)
    idx = np.asarray(idx)
    gate = np.asarray(gate, F64)
    x = np.asarray(x, F64)
    w = np.asarray(w_router, F64)
    T, k = idx.shape
    E = w.shape[0]
    ok = idx >= 0
    s = np.sum(np.where(ok, gate * dgate, 0.0), axis=1)          # sum_j g_j dg_j
    dl = np.zeros((T, E), F64)
    if renorm:
        tt, jj = np.nonzero(ok)
        dl[tt, idx[tt, jj]] = gate[tt, jj] * (dgate[tt, jj] - s[tt])
    else:
        l = round_f32(np.asarray(logits, F64))
        alive_m = np.ones(E, bool) if alive is None else np.asarray(alive).astype(bool)
        masked = np.where(alive_m[None, :], l, -np.inf)
        top = masked.max(axis=1, keepdims=True)
        ex = np.where(alive_m[None, :], np.exp(masked - top), 0.0)
        p = ex / ex.sum(axis=1, keepdims=True)
        q = np.zeros((T, E), F64)
        tt, jj = np.nonzero(ok)
        q[tt, idx[tt, jj]] = dgate[tt, jj]
        dl = np.where(alive_m[None, :], p * (q - s[:, None]), 0.0)
    dw = round_f32(dl.T @ x)
    db = round_f32(dl.sum(axis=0))
    dx = dl @ w
    if dx_in is not None:
        dx = dx + np.asarray(dx_in, F64)
    return round_f32(dl), dw, db, rounder(dtype)(dx)


# --------------------------------------------------------------------------
# Per-expert token histogram, offsets and the dispatch permutation
# --------------------------------------------------------------------------
def expert_counts(idx, E: int):
    """Expert loads and the stable counting-sort permutation.

    counts[e] = #{(t, j): idx[t, j] = e}   (sum_j E[e, j, l], Section 3.2)
    offsets   = exclusive prefix sum of counts; offsets[E] = routed rows
    dest_row[t*k + j] = offsets[e] + #{(t', j'): idx[t', j'] = e, t' < t}
    i.e. rows are grouped by expert and ordered by token inside a group.
    Unrouted slots (idx = -1) get dest_row = -1.
    """
    idx = np.asarray(idx)
    flat = idx.reshape(-1)
    counts = np.zeros(E, dtype=np.int64)
    for e in range(E):
        counts[e] = int(np.count_nonzero(flat == e))
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    dest = np.full(flat.shape[0], -1, dtype=np.int64)
    routed = np.nonzero(flat >= 0)[0]
    # flat position t*k + j increases with t; a token never repeats an
    # expert, so a stable sort by expert orders each group by token.
    order = routed[np.argsort(flat[routed], kind="stable")]
    dest[order] = np.arange(order.shape[0])
    return counts, offsets, dest


# --------------------------------------------------------------------------
# Permute / grouped SwiGLU FFN / combine
# --------------------------------------------------------------------------
def permute(x, dest_row, k: int):
    """x_perm[dest_row[t*k + j]] = x[t]  (a copy)."""
    x = np.asarray(x)
    dest_row = np.asarray(dest_row)
    R = int((dest_row >= 0).sum())
    out = np.zeros((R, x.shape[1]), dtype=x.dtype)
    for s, r in enumerate(dest_row):
        if r >= 0:
            out[r] = x[s // k]
    return out


def _phys(expert_map, e):
    return e if expert_map is None else int(expert_map[e])


def expert_ffn(x_rows, w_gu, w_d, dtype: str):
    """SwiGLU FFN of one expert on its rows.

    A = X W_gu^T (W_gu = [W_gate; W_up], shape [2f, d]); A is kept
    unrounded inside the FFN.  act_save = round(A).
    H = round(silu(A_gate) * A_up);  Y = round(H W_d^T).
    """
    rnd = rounder(dtype)
    f = w_d.shape[1]
    A = np.asarray(x_rows, F64) @ np.asarray(w_gu, F64).T
    act = rnd(A)
    H = rnd(silu(A[:, :f]) * A[:, f:])
    Y = rnd(H @ np.asarray(w_d, F64).T)
    return Y, act, H


def grouped_ffn_fwd(x_perm, w_gate_up, w_down, offsets, expert_map=None,
                    dtype: str = "bf16", return_h: bool = False):
    """Per expert e with rows [offsets[e], offsets[e+1]): the SwiGLU FFN
    with that expert's weights (physical slot expert_map[e]).
    Returns (y_perm, act_save), and H (the rounded activation the down
    projection consumes) when ``return_h``."""
    x_perm = np.asarray(x_perm)
    R, d = x_perm.shape
    f = w_down.shape[2]
    y = np.zeros((R, d), F64)
    act = np.zeros((R, 2 * f), F64)
    h = np.zeros((R, f), F64)
    E = len(offsets) - 1
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi == lo:
            continue
        p = _phys(expert_map, e)
        if p < 0:
            raise ValueError(f"expert {e} has rows but no weight slot")
        y[lo:hi], act[lo:hi], h[lo:hi] = expert_ffn(x_perm[lo:hi], w_gate_up[p],
                                                    w_down[p], dtype)
    return (y, act, h) if return_h else (y, act)


def combine(y_perm, gate, dest_row, k: int, dtype: str = "bf16"):
    """out[t] = round(sum_j g[t, j] * y[dest_row[t*k + j]]), float64 sum."""
    rnd = rounder(dtype)
    gate = np.asarray(gate, F64).reshape(-1, k)
    dest_row = np.asarray(dest_row).reshape(-1, k)
    T = gate.shape[0]
    out = np.zeros((T, y_perm.shape[1]), F64)
    for t in range(T):
        acc = np.zeros(y_perm.shape[1], F64)
        for j in range(k):
            r = dest_row[t, j]
            if r >= 0:
                acc += gate[t, j] * np.asarray(y_perm[r], F64)
        out[t] = acc
    return rnd(out)


# --------------------------------------------------------------------------
# Backward (pre-training step)
# --------------------------------------------------------------------------
def combine_bwd(dout, y_perm, gate, dest_row, k: int, dtype: str = "bf16"):
    """Backward of combine.

    dgate[t, j] = float32(<dout[t], y[row]>),
    dy[row]     = round(g[t, j] * dout[t]),   row = dest_row[t*k + j].
    """
    rnd = rounder(dtype)
    gate = np.asarray(gate, F64).reshape(-1, k)
    dest_row = np.asarray(dest_row).reshape(-1, k)
    T = gate.shape[0]
    dgate = np.zeros((T, k), F64)
    dy = np.zeros(y_perm.shape, F64)
    for t in range(T):
        d_t = np.asarray(dout[t], F64)
        for j in range(k):
            r = dest_row[t, j]
            if r < 0:
                continue
            dgate[t, j] = float(np.dot(d_t, np.asarray(y_perm[r], F64)))
            dy[r] = rnd(gate[t, j] * d_t)
    rnd_g = (lambda a: a) if dtype == "f64" else round_f32
    return dy, rnd_g(dgate)


def swiglu_bwd(dH, act_save, dtype: str = "bf16"):
    """Backward of H = silu(A_g) * A_u, evaluated at the saved A.

    With s = sigmoid(A_g):
      dA_g = dH * A_u * s * (1 + A_g * (1 - s))   (d silu / da = s(1 + a(1-s)))
      dA_u = dH * silu(A_g)
    Returns (dA = round([dA_g, dA_u]), H_b = round(silu(A_g) * A_u)); H_b is
    the H the weight gradient of W_d uses.
    """
    rnd = rounder(dtype)
    act = np.asarray(act_save, F64)
    f = act.shape[1] // 2
    ag, au = act[:, :f], act[:, f:]
    s = sigmoid(ag)
    dH = np.asarray(dH, F64)
    dAg = dH * au * s * (1.0 + ag * (1.0 - s))
    dAu = dH * silu(ag)
    dA = rnd(np.concatenate([dAg, dAu], axis=1))
    Hb = rnd(silu(ag) * au)
    return dA, Hb


def grouped_ffn_dgrad(dy_perm, act_save, w_gate_up, w_down, offsets,
                      expert_map=None, dtype: str = "bf16", dA_given=None):
    """Data gradient of the grouped FFN.

    Per expert: dH = dY W_d (unrounded); (dA, H_b) = swiglu_bwd(dH,
    act_save); dX = round(dA W_gu).  ``dA_given`` (teacher forcing) replaces
    the dA computed here as the input of dX.  Returns (dx_perm, dA, H_b).
    """
    rnd = rounder(dtype)
    R, d = dy_perm.shape
    f = w_down.shape[2]
    dx = np.zeros((R, d), F64)
    dA = np.zeros((R, 2 * f), F64)
    Hb = np.zeros((R, f), F64)
    E = len(offsets) - 1
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi == lo:
            continue
        p = _phys(expert_map, e)
        dH = np.asarray(dy_perm[lo:hi], F64) @ np.asarray(w_down[p], F64)
        dA[lo:hi], Hb[lo:hi] = swiglu_bwd(dH, act_save[lo:hi], dtype)
        src = dA[lo:hi] if dA_given is None else np.asarray(dA_given[lo:hi], F64)
        dx[lo:hi] = rnd(src @ np.asarray(w_gate_up[p], F64))
    return dx, dA, Hb


def grouped_ffn_wgrad(dy_perm, x_perm, dA, Hb, offsets, n_phys: int,
                      expert_map=None, out_f32: bool = True):
    """Weight gradients (float32): per expert with rows,
    dW_gu = dA^T X and dW_d = dY^T H over the expert's rows, where ``Hb`` is
    the H to use: the forward's (the activation the down projection
    consumed) or H_b recomputed at the saved pre-activations.
    Weight slots that receive no rows get zero gradient."""
    R, d = x_perm.shape
    f = Hb.shape[1]
    dw_gu = np.zeros((n_phys, 2 * f, d), F64)
    dw_d = np.zeros((n_phys, d, f), F64)
    E = len(offsets) - 1
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi == lo:
            continue
        p = _phys(expert_map, e)
        dw_gu[p] = np.asarray(dA[lo:hi], F64).T @ np.asarray(x_perm[lo:hi], F64)
        dw_d[p] = np.asarray(dy_perm[lo:hi], F64).T @ np.asarray(Hb[lo:hi], F64)
    if out_f32:
        return round_f32(dw_gu), round_f32(dw_d)
    return dw_gu, dw_d


def permute_bwd(dx_perm, dest_row, k: int, dtype: str = "bf16"):
    """dx[t] = round(sum_j dx_perm[dest_row[t*k + j]]), float64 sum."""
    rnd = rounder(dtype)
    dest_row = np.asarray(dest_row).reshape(-1, k)
    T = dest_row.shape[0]
    dx = np.zeros((T, dx_perm.shape[1]), F64)
    for t in range(T):
        for j in range(k):
            r = dest_row[t, j]
            if r >= 0:
                dx[t] += np.asarray(dx_perm[r], F64)
    return rnd(dx)


# --------------------------------------------------------------------------
# The whole layer (forward) -- convenience for end-to-end checks
# --------------------------------------------------------------------------
def layer_forward(x, w_router, w_gate_up, w_down, k, bias=None, alive=None,
                  renorm=True, dtype="bf16"):
    idx, gate, margin, logits = route(x, w_router, k, bias=bias, alive=alive,
                                      renorm=renorm)
    E = w_router.shape[0]
    counts, offsets, dest = expert_counts(idx, E)
    xp = permute(x, dest, k)
    y, act = grouped_ffn_fwd(xp, w_gate_up, w_down, offsets, dtype=dtype)
    out = combine(y, gate, dest, k, dtype=dtype)
    return dict(idx=idx, gate=gate, margin=margin, logits=logits,
                counts=counts, offsets=offsets, dest_row=dest, x_perm=xp,
                y_perm=y, act_save=act, out=out)


__all__ = [
    "router_logits", "topk_gating", "selection_gates", "route", "expert_counts", "permute",
    "expert_ffn", "grouped_ffn_fwd", "combine", "combine_bwd", "swiglu_bwd",
    "grouped_ffn_dgrad", "grouped_ffn_wgrad", "permute_bwd", "layer_forward",
    "round_bf16",
]
