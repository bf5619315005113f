"""Python binding of the LAEP MoE C ABI on torch tensors.

Argument marshalling only: each function checks tensor placement and
layout, allocates missing outputs with torch (device memory is PyTorch's
job), and calls the same-named C entry point on the current HIP stream.
Every step of the layer runs in the library's HIP kernels.
"""
from __future__ import annotations

import ctypes
import math
from typing import Optional, Tuple

import torch

from ._lib import (LAEP_BF16, LAEP_CALL_COUNTS, LAEP_CALL_FFN_BWD, LAEP_CALL_FFN_FWD,
                   LAEP_CALL_ROUTE_BWD, LAEP_F32, LaepError, check, lib)

_DT = {torch.float32: LAEP_F32, torch.bfloat16: LAEP_BF16}


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise LaepError(2, f"unsupported dtype {t.dtype}")
    return _DT[t.dtype]


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dev(t: torch.Tensor, name: str) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def workspace_bytes(which: int, T: int, k: int, E: int, d_model: int = 0, d_ff: int = 0) -> int:
    return int(lib().moe_workspace_bytes(which, T, k, E, d_model, d_ff))


def _workspace(ws, nbytes, device):
    if ws is None:
        return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)
    if ws.numel() * ws.element_size() < nbytes:
        raise LaepError(3, f"workspace {ws.numel() * ws.element_size()} < {nbytes} bytes")
    return ws


# ---------------------------------------------------------------------------
def moe_route(x: torch.Tensor, w_router: torch.Tensor, k: int, *, bias=None, alive=None,
              renorm: bool = True, want_logits: bool = False, topk_idx=None, topk_gate=None):
    """Router scoring + top-k gating.  Returns (topk_idx, topk_gate[, logits])."""
    _dev(x, "x"), _dev(w_router, "w_router")
    T, d = x.shape
    E = w_router.shape[0]
    dev = x.device
    if topk_idx is None:
        topk_idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    if topk_gate is None:
        topk_gate = torch.empty((T, k), dtype=torch.float32, device=dev)
    logits = torch.empty((T, E), dtype=torch.float32, device=dev) if want_logits else None
    if bias is not None:
        _dev(bias, "bias")
    if alive is not None:
        _dev(alive, "alive")
    check(lib().moe_route(_ptr(x), _ptr(w_router), _ptr(bias), _ptr(alive), _dtype_code(x), T, d,
                          E, k, int(renorm), _ptr(logits), _ptr(topk_idx), _ptr(topk_gate), None,
                          0, _stream(dev)))
    return (topk_idx, topk_gate, logits) if want_logits else (topk_idx, topk_gate)


def moe_route_bwd(dgate: torch.Tensor, topk_idx: torch.Tensor, topk_gate: torch.Tensor,
                  x: torch.Tensor, w_router: torch.Tensor, *, renorm: bool = True,
                  logits=None, alive=None, offsets=None, row_src=None, dx=None,
                  accumulate_dx: bool = False, want_dlogits: bool = False,
                  want_dbias: bool = False, dw_router=None, dlogits=None, dbias=None, ws=None,
                  data: bool = True, weights: bool = True):
    """Router/gate backward with the selection fixed.  ``data=False`` skips dx,
    ``weights=False`` skips dw_router and dbias.
    Returns (dx, dw_router, dbias, dlogits), None for what was not computed."""
    for t, n in ((dgate, "dgate"), (topk_idx, "topk_idx"), (topk_gate, "topk_gate"), (x, "x"),
                 (w_router, "w_router")):
        _dev(t, n)
    T, k = topk_idx.shape
    E, d = w_router.shape
    dev = x.device
    if data:
        dx = torch.zeros_like(x) if dx is None else dx
    else:
        dx = None
    if weights:
        dw_router = (torch.empty((E, d), dtype=torch.float32, device=dev) if dw_router is None
                     else dw_router)
        if want_dbias and dbias is None:
            dbias = torch.empty(E, dtype=torch.float32, device=dev)
    else:
        dw_router, dbias = None, None
    if want_dlogits and dlogits is None:
        dlogits = torch.empty((T, E), dtype=torch.float32, device=dev)
    ws = _workspace(ws, workspace_bytes(LAEP_CALL_ROUTE_BWD, T, k, E, d), dev)
    check(lib().moe_route_bwd(_ptr(dgate), _ptr(topk_idx), _ptr(topk_gate), _ptr(logits),
                              _ptr(alive), _ptr(x), _ptr(w_router), _ptr(offsets), _ptr(row_src),
                              _dtype_code(x), T, d, E, k, int(renorm), _ptr(dlogits),
                              _ptr(dw_router), _ptr(dbias), _ptr(dx), int(accumulate_dx),
                              _ptr(ws), ws.numel(), _stream(dev)))
    return dx, dw_router, dbias, dlogits


def moe_expert_counts(topk_idx: torch.Tensor, E: int, *, want_row_src: bool = False,
                      etn_accum=None, ws=None, counts=None, offsets=None, dest_row=None,
                      row_src=None):
    """Returns (counts [E] i32, offsets [E+1] i32, dest_row [T*k] i32[, row_src])."""
    _dev(topk_idx, "topk_idx")
    T, k = topk_idx.shape
    dev = topk_idx.device
    counts = torch.empty(E, dtype=torch.int32, device=dev) if counts is None else counts
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev) if offsets is None else offsets
    dest_row = torch.empty(T * k, dtype=torch.int32, device=dev) if dest_row is None else dest_row
    want_row_src = want_row_src or row_src is not None
    if want_row_src and row_src is None:
        row_src = torch.empty(T * k, dtype=torch.int32, device=dev)
    nbytes = workspace_bytes(LAEP_CALL_COUNTS, T, k, E)
    ws = _workspace(ws, nbytes, dev)
    check(lib().moe_expert_counts(_ptr(topk_idx), T, k, E, _ptr(counts), _ptr(offsets),
                                  _ptr(dest_row), _ptr(row_src), _ptr(etn_accum), _ptr(ws),
                                  ws.numel(), _stream(dev)))
    out = (counts, offsets, dest_row)
    return out + (row_src,) if want_row_src else out


def moe_route_count(x: torch.Tensor, w_router: torch.Tensor, k: int, *, bias=None, alive=None,
                    renorm: bool = True, want_logits: bool = False, want_row_src: bool = False,
                    etn_accum=None, ws=None, topk_idx=None, topk_gate=None, counts=None,
                    offsets=None, dest_row=None, row_src=None):
    """Routing and expert counts in one call.  Returns (topk_idx, topk_gate,
    counts, offsets, dest_row, row_src or None, logits or None)."""
    _dev(x, "x"), _dev(w_router, "w_router")
    T, d = x.shape
    E = w_router.shape[0]
    dev = x.device
    i32 = torch.int32
    topk_idx = torch.empty((T, k), dtype=i32, device=dev) if topk_idx is None else topk_idx
    topk_gate = (torch.empty((T, k), dtype=torch.float32, device=dev) if topk_gate is None
                 else topk_gate)
    counts = torch.empty(E, dtype=i32, device=dev) if counts is None else counts
    offsets = torch.empty(E + 1, dtype=i32, device=dev) if offsets is None else offsets
    dest_row = torch.empty(T * k, dtype=i32, device=dev) if dest_row is None else dest_row
    if want_row_src and row_src is None:
        row_src = torch.empty(T * k, dtype=i32, device=dev)
    logits = torch.empty((T, E), dtype=torch.float32, device=dev) if want_logits else None
    ws = _workspace(ws, workspace_bytes(LAEP_CALL_COUNTS, T, k, E), dev)
    check(lib().moe_route_count(_ptr(x), _ptr(w_router), _ptr(bias), _ptr(alive), _dtype_code(x),
                                T, d, E, k, int(renorm), _ptr(logits), _ptr(topk_idx),
                                _ptr(topk_gate), _ptr(counts), _ptr(offsets), _ptr(dest_row),
                                _ptr(row_src), _ptr(etn_accum), _ptr(ws), ws.numel(),
                                _stream(dev)))
    return topk_idx, topk_gate, counts, offsets, dest_row, row_src, logits


def moe_route_count_noalloc(x: torch.Tensor, w_router: torch.Tensor, k: int, *, bias=None,
                            alive=None, renorm: bool = True, want_logits: bool = False,
                            want_row_src: bool = False, etn_accum=None, topk_idx=None,
                            topk_gate=None, counts=None, offsets=None, dest_row=None,
                            row_src=None, logits=None):
    """moe_route_count with the library's own scratch array (no workspace;
    the C call allocates nothing).  Pass every output to keep this wrapper
    allocation-free too.  Returns as moe_route_count."""
    _dev(x, "x"), _dev(w_router, "w_router")
    T, d = x.shape
    E = w_router.shape[0]
    dev = x.device
    i32 = torch.int32
    topk_idx = torch.empty((T, k), dtype=i32, device=dev) if topk_idx is None else topk_idx
    topk_gate = (torch.empty((T, k), dtype=torch.float32, device=dev) if topk_gate is None
                 else topk_gate)
    counts = torch.empty(E, dtype=i32, device=dev) if counts is None else counts
    offsets = torch.empty(E + 1, dtype=i32, device=dev) if offsets is None else offsets
    dest_row = torch.empty(T * k, dtype=i32, device=dev) if dest_row is None else dest_row
    if want_row_src and row_src is None:
        row_src = torch.empty(T * k, dtype=i32, device=dev)
    if want_logits and logits is None:
        logits = torch.empty((T, E), dtype=torch.float32, device=dev)
    check(lib().moe_route_count_noalloc(_ptr(x), _ptr(w_router), _ptr(bias), _ptr(alive),
                                        _dtype_code(x), T, d, E, k, int(renorm), _ptr(logits),
                                        _ptr(topk_idx), _ptr(topk_gate), _ptr(counts),
                                        _ptr(offsets), _ptr(dest_row), _ptr(row_src),
                                        _ptr(etn_accum), _stream(dev)))
    return topk_idx, topk_gate, counts, offsets, dest_row, row_src, logits


def laep_prune_mask(counts: torch.Tensor, total: int, alpha: float = math.inf,
                    beta: float = 0.0, *, alive=None, n_pruned=None):
    """LAEP prune decision.  Returns (alive [E] uint8, n_pruned [1] int32)."""
    _dev(counts, "counts")
    E = counts.shape[0]
    dev = counts.device
    alive = torch.empty(E, dtype=torch.uint8, device=dev) if alive is None else alive
    n_pruned = torch.empty(1, dtype=torch.int32, device=dev) if n_pruned is None else n_pruned
    check(lib().laep_prune_mask(_ptr(counts), E, int(total), float(alpha), float(beta),
                                _ptr(alive), _ptr(n_pruned), _stream(dev)))
    return alive, n_pruned


def laep_expert_pruning(etn: torch.Tensor, total: int, alpha, beta: float, *,
                        alive=None, n_pruned=None, want_marker: bool = False):
    """Algorithm 1 over a recorded window etn [ITER, L, E] int64.  ``alpha`` is a
    float or a per-layer sequence.  Returns (alive [L, E] uint8, n_pruned [L]
    int32, marker [L, E] int32 or None)."""
    _dev(etn, "etn")
    if etn.dtype != torch.int64 or etn.dim() != 3:
        raise ValueError("etn must be an int64 tensor [ITER, L, E]")
    iters, L, E = etn.shape
    alphas = [float(alpha)] * L if isinstance(alpha, (int, float)) else [float(a) for a in alpha]
    if len(alphas) != L:
        raise ValueError(f"alpha has {len(alphas)} entries for {L} layers")
    dev = etn.device
    alive = torch.empty((L, E), dtype=torch.uint8, device=dev) if alive is None else alive
    n_pruned = torch.empty(L, dtype=torch.int32, device=dev) if n_pruned is None else n_pruned
    marker = torch.empty((L, E), dtype=torch.int32, device=dev) if want_marker else None
    a_host = (ctypes.c_double * L)(*alphas)
    check(lib().laep_expert_pruning(_ptr(etn), iters, L, E, int(total), a_host, float(beta),
                                    _ptr(alive), _ptr(n_pruned), _ptr(marker), _stream(dev)))
    return alive, n_pruned, marker


def laep_compact_experts(alive: torch.Tensor, *, expert_map=None, n_alive=None):
    """Slots of the surviving experts.  alive [E] or [L, E] uint8.
    Returns (expert_map of alive's shape int32, n_alive [L] int32)."""
    _dev(alive, "alive")
    a2 = alive.reshape(-1, alive.shape[-1])
    L, E = a2.shape
    dev = alive.device
    expert_map = (torch.empty(alive.shape, dtype=torch.int32, device=dev) if expert_map is None
                  else expert_map)
    n_alive = torch.empty(L, dtype=torch.int32, device=dev) if n_alive is None else n_alive
    check(lib().laep_compact_experts(_ptr(alive), L, E, _ptr(expert_map), _ptr(n_alive),
                                     _stream(dev)))
    return expert_map, n_alive


def laep_repack_experts(expert_map: torch.Tensor, n_out: int, *, w_router=None, bias=None,
                        w_gate_up=None, w_down=None, out=None):
    """Copy the surviving experts' parameters (one layer) into n_out slots.
    Returns a dict with the repacked tensors that were given."""
    _dev(expert_map, "expert_map")
    E = expert_map.shape[0]
    given = {n: t for n, t in (("w_router", w_router), ("bias", bias), ("w_gate_up", w_gate_up),
                               ("w_down", w_down)) if t is not None}
    mats = [t for n, t in given.items() if n != "bias"]
    dtype = mats[0].dtype if mats else torch.float32
    if any(t.dtype != dtype for t in mats):
        raise ValueError("the repacked matrices must share one dtype")
    d_model = (w_router.shape[1] if w_router is not None else
               w_gate_up.shape[2] if w_gate_up is not None else
               w_down.shape[1] if w_down is not None else 8)
    d_ff = (w_gate_up.shape[1] // 2 if w_gate_up is not None else
            w_down.shape[2] if w_down is not None else 0)
    for n, t in given.items():
        _dev(t, n)
        if t.shape[0] != E:
            raise ValueError(f"{n} has {t.shape[0]} experts, expert_map {E}")
    out = {} if out is None else dict(out)
    for n, t in given.items():
        if n not in out:
            out[n] = torch.empty((n_out, *t.shape[1:]), dtype=t.dtype, device=t.device)
    code = _dtype_code(mats[0]) if mats else LAEP_F32
    check(lib().laep_repack_experts(_ptr(expert_map), E, int(n_out), code, d_model, d_ff,
                                    _ptr(w_router), _ptr(bias), _ptr(w_gate_up), _ptr(w_down),
                                    _ptr(out.get("w_router")), _ptr(out.get("bias")),
                                    _ptr(out.get("w_gate_up")), _ptr(out.get("w_down")),
                                    _stream(expert_map.device)))
    return out


def moe_permute(x: torch.Tensor, dest_row: torch.Tensor, k: int, rows: Optional[int] = None,
                *, out=None):
    """x_perm[dest_row[t*k+j]] = x[t].  ``rows`` defaults to T*k."""
    _dev(x, "x"), _dev(dest_row, "dest_row")
    T, d = x.shape
    rows = T * k if rows is None else rows
    out = torch.empty((rows, d), dtype=x.dtype, device=x.device) if out is None else out
    check(lib().moe_permute(_ptr(x), _dtype_code(x), _ptr(dest_row), T, k, d, _ptr(out),
                            _stream(x.device)))
    return out


def moe_grouped_ffn_fwd(x_perm: torch.Tensor, w_gate_up: torch.Tensor, w_down: torch.Tensor,
                        offsets: torch.Tensor, *, expert_map=None, save_act: bool = True,
                        ws=None, y_perm=None, act_save=None):
    """Grouped SwiGLU FFN.  Returns (y_perm, act_save or None)."""
    for t, n in ((x_perm, "x_perm"), (w_gate_up, "w_gate_up"), (w_down, "w_down"),
                 (offsets, "offsets")):
        _dev(t, n)
    R, d = x_perm.shape
    f = w_down.shape[2]
    E = offsets.shape[0] - 1
    dev = x_perm.device
    y_perm = torch.empty_like(x_perm) if y_perm is None else y_perm
    if save_act and act_save is None:
        act_save = torch.empty((R, 2 * f), dtype=x_perm.dtype, device=dev)
    if not save_act:
        act_save = None
    ws = _workspace(ws, workspace_bytes(LAEP_CALL_FFN_FWD, R, 1, E, d, f), dev)
    check(lib().moe_grouped_ffn_fwd(_ptr(x_perm), _ptr(w_gate_up), _ptr(w_down), _ptr(offsets),
                                    _ptr(expert_map), _dtype_code(x_perm), E, d, f, R,
                                    _ptr(y_perm), _ptr(act_save), _ptr(ws), ws.numel(),
                                    _stream(dev)))
    return y_perm, act_save


def moe_grouped_ffn_fwd_gather(x: torch.Tensor, row_src: torch.Tensor, k: int,
                               w_gate_up: torch.Tensor, w_down: torch.Tensor,
                               offsets: torch.Tensor, *, rows: Optional[int] = None,
                               expert_map=None, save_act: bool = False, ws=None, y_perm=None,
                               act_save=None, x_perm_out=None):
    """moe_permute + moe_grouped_ffn_fwd in one pass (bf16): routed row r reads
    token row row_src[r] // k; ``x_perm_out`` [R, d] (optional) also receives
    the dispatched rows, copied beside the FFN.  Returns (y_perm, act_save or None)."""
    for t, n in ((x, "x"), (row_src, "row_src"), (w_gate_up, "w_gate_up"), (w_down, "w_down"),
                 (offsets, "offsets")):
        _dev(t, n)
    T, d = x.shape
    R = T * k if rows is None else rows
    f = w_down.shape[2]
    E = offsets.shape[0] - 1
    dev = x.device
    y_perm = torch.empty((R, d), dtype=x.dtype, device=dev) if y_perm is None else y_perm
    if save_act and act_save is None:
        act_save = torch.empty((R, 2 * f), dtype=x.dtype, device=dev)
    if not save_act:
        act_save = None
    ws = _workspace(ws, workspace_bytes(LAEP_CALL_FFN_FWD, R, 1, E, d, f), dev)
    check(lib().moe_grouped_ffn_fwd_gather(_ptr(x), _ptr(row_src), T, k, _ptr(w_gate_up),
                                           _ptr(w_down), _ptr(offsets), _ptr(expert_map),
                                           _dtype_code(x), E, d, f, R, _ptr(y_perm),
                                           _ptr(act_save), _ptr(x_perm_out), _ptr(ws), ws.numel(),
                                           _stream(dev)))
    return y_perm, act_save


def moe_grouped_ffn_fwd_gather_combine(x: torch.Tensor, row_src: torch.Tensor,
                                       topk_gate: torch.Tensor, w_gate_up: torch.Tensor,
                                       w_down: torch.Tensor, offsets: torch.Tensor, *,
                                       rows: Optional[int] = None, expert_map=None,
                                       keep_y: bool = False, save_act: bool = False, ws=None,
                                       out=None, y_perm=None, act_save=None, x_perm_out=None):
    """moe_grouped_ffn_fwd_gather + moe_combine for one slot per token (bf16):
    routed row r goes straight to token row row_src[r], times its gate.
    Returns (out, y_perm or None, act_save or None)."""
    for t, n in ((x, "x"), (row_src, "row_src"), (topk_gate, "topk_gate"),
                 (w_gate_up, "w_gate_up"), (w_down, "w_down"), (offsets, "offsets")):
        _dev(t, n)
    T, d = x.shape
    R = T if rows is None else rows
    f = w_down.shape[2]
    E = offsets.shape[0] - 1
    dev = x.device
    out = torch.empty((T, d), dtype=x.dtype, device=dev) if out is None else out
    if keep_y and y_perm is None:
        y_perm = torch.empty((R, d), dtype=x.dtype, device=dev)
    if not keep_y:
        y_perm = None
    if save_act and act_save is None:
        act_save = torch.empty((R, 2 * f), dtype=x.dtype, device=dev)
    if not save_act:
        act_save = None
    ws = _workspace(ws, workspace_bytes(LAEP_CALL_FFN_FWD, R, 1, E, d, f), dev)
    check(lib().moe_grouped_ffn_fwd_gather_combine(
        _ptr(x), _ptr(row_src), T, 1, _ptr(w_gate_up), _ptr(w_down), _ptr(offsets),
        _ptr(expert_map), _ptr(topk_gate), _dtype_code(x), E, d, f, R, _ptr(out), _ptr(y_perm),
        _ptr(act_save), _ptr(x_perm_out), _ptr(ws), ws.numel(), _stream(dev)))
    return out, y_perm, act_save


def moe_grouped_ffn_bwd(dy_perm, x_perm, act_save, w_gate_up, w_down, offsets, *,
                        h_fwd=None, expert_map=None, dw_gate_up=None, dw_down=None,
                        accumulate=False, ws=None, dx_perm=None, return_ws: bool = False):
    """Backward of the grouped FFN.  ``h_fwd``: the forward's H [R, f] (see
    ffn_fwd_h_view); dW_d then uses it, else H_b recomputed at act_save.
    Returns (dx_perm, dw_gate_up, dw_down[, ws])."""
    for t, n in ((dy_perm, "dy_perm"), (x_perm, "x_perm"), (act_save, "act_save"),
                 (w_gate_up, "w_gate_up"), (w_down, "w_down"), (offsets, "offsets")):
        _dev(t, n)
    if h_fwd is not None:
        _dev(h_fwd, "h_fwd")
    R, d = x_perm.shape
    f = w_down.shape[2]
    E = offsets.shape[0] - 1
    dev = x_perm.device
    dx_perm = torch.empty_like(x_perm) if dx_perm is None else dx_perm
    if dw_gate_up is None:
        dw_gate_up = torch.empty(w_gate_up.shape, dtype=torch.float32, device=dev)
    if dw_down is None:
        dw_down = torch.empty(w_down.shape, dtype=torch.float32, device=dev)
    ws = _workspace(ws, workspace_bytes(LAEP_CALL_FFN_BWD, R, 1, E, d, f), dev)
    check(lib().moe_grouped_ffn_bwd(_ptr(dy_perm), _ptr(x_perm), _ptr(act_save), _ptr(h_fwd),
                                    _ptr(w_gate_up), _ptr(w_down), _ptr(offsets),
                                    _ptr(expert_map), _dtype_code(x_perm), E, d, f, R,
                                    _ptr(dx_perm), _ptr(dw_gate_up), _ptr(dw_down),
                                    int(accumulate), _ptr(ws), ws.numel(), _stream(dev)))
    out = (dx_perm, dw_gate_up, dw_down)
    return out + (ws,) if return_ws else out


def moe_grouped_ffn_bwd_gather(dy_perm, x, row_src, k: int, act_save, w_gate_up, w_down,
                               offsets, *, dout=None, topk_gate=None, h_fwd=None,
                               expert_map=None, dw_gate_up=None, dw_down=None, accumulate=False,
                               ws=None, dx_perm=None, return_ws: bool = False):
    """moe_grouped_ffn_bwd with the weight gradient reading X's routed rows
    from the token rows x through row_src (no x_perm).  With dy_perm None,
    dY is formed on load from ``dout`` [T, d] and ``topk_gate`` [T, k] (no
    dy_perm).  Returns as moe_grouped_ffn_bwd."""
    for t, n in ((x, "x"), (row_src, "row_src"), (act_save, "act_save"),
                 (w_gate_up, "w_gate_up"), (w_down, "w_down"), (offsets, "offsets")):
        _dev(t, n)
    if dy_perm is None:
        if dout is None or topk_gate is None:
            raise ValueError("without dy_perm, dout and topk_gate are needed")
        _dev(dout, "dout"), _dev(topk_gate, "topk_gate")
    else:
        _dev(dy_perm, "dy_perm")
    if h_fwd is not None:
        _dev(h_fwd, "h_fwd")
    T, d = x.shape
    R = row_src.shape[0]
    f = w_down.shape[2]
    E = offsets.shape[0] - 1
    dev = x.device
    dx_perm = torch.empty((R, d), dtype=x.dtype, device=dev) if dx_perm is None else dx_perm
    if dw_gate_up is None:
        dw_gate_up = torch.empty(w_gate_up.shape, dtype=torch.float32, device=dev)
    if dw_down is None:
        dw_down = torch.empty(w_down.shape, dtype=torch.float32, device=dev)
    ws = _workspace(ws, workspace_bytes(LAEP_CALL_FFN_BWD, R, 1, E, d, f), dev)
    check(lib().moe_grouped_ffn_bwd_gather(
        _ptr(dy_perm), _ptr(dout), _ptr(topk_gate), _ptr(x), _ptr(row_src), T, k,
        _ptr(act_save), _ptr(h_fwd),
        _ptr(w_gate_up), _ptr(w_down), _ptr(offsets), _ptr(expert_map), _dtype_code(x), E, d, f,
        R, _ptr(dx_perm), _ptr(dw_gate_up), _ptr(dw_down), int(accumulate), _ptr(ws), ws.numel(),
        _stream(dev)))
    out = (dx_perm, dw_gate_up, dw_down)
    return out + (ws,) if return_ws else out


def ffn_fwd_h_view(ws: torch.Tensor, R: int, d_ff: int, dtype: torch.dtype):
    """H [R, f] as the forward leaves it in its workspace (byte offset 0)."""
    esz = torch.empty((), dtype=dtype).element_size()
    return ws.view(torch.uint8)[: R * d_ff * esz].view(dtype).view(R, d_ff)


def ffn_bwd_ws_views(ws: torch.Tensor, R: int, d_ff: int, dtype: torch.dtype):
    """dA [R, 2f] and the H_b buffer [R, f] (H_b, or dH when the backward
    used the forward's H) as left in the backward workspace."""
    code = _DT[dtype]
    esz = torch.empty((), dtype=dtype).element_size()
    off = int(lib().laep_ws_hb_offset(R, d_ff, code))
    raw = ws.view(torch.uint8)
    dA = raw[: R * 2 * d_ff * esz].view(dtype).view(R, 2 * d_ff)
    hb = raw[off: off + R * d_ff * esz].view(dtype).view(R, d_ff)
    return dA, hb


def moe_combine(y_perm: torch.Tensor, topk_gate: torch.Tensor, dest_row: torch.Tensor,
                *, out=None):
    """out[t] = sum_j g[t,j] * y_perm[dest_row[t*k+j]]."""
    _dev(y_perm, "y_perm"), _dev(topk_gate, "topk_gate"), _dev(dest_row, "dest_row")
    T, k = topk_gate.shape
    d = y_perm.shape[1]
    out = torch.empty((T, d), dtype=y_perm.dtype, device=y_perm.device) if out is None else out
    check(lib().moe_combine(_ptr(y_perm), _ptr(topk_gate), _ptr(dest_row), T, k, d,
                            _dtype_code(y_perm), _ptr(out), _stream(y_perm.device)))
    return out


def moe_combine_bwd(dout: torch.Tensor, y_perm: torch.Tensor, topk_gate: torch.Tensor,
                    dest_row: torch.Tensor, *, dy_perm=None, dgate=None, want_dy: bool = True):
    """Returns (dy_perm, dgate); with want_dy False only dgate is computed
    (dy_perm None: moe_grouped_ffn_bwd_gather forms dY itself)."""
    for t, n in ((dout, "dout"), (y_perm, "y_perm"), (topk_gate, "topk_gate"),
                 (dest_row, "dest_row")):
        _dev(t, n)
    T, k = topk_gate.shape
    d = dout.shape[1]
    dev = dout.device
    if want_dy and dy_perm is None:
        dy_perm = torch.empty_like(y_perm)
    if not want_dy:
        dy_perm = None
    dgate = torch.empty((T, k), dtype=torch.float32, device=dev) if dgate is None else dgate
    check(lib().moe_combine_bwd(_ptr(dout), _ptr(y_perm), _ptr(topk_gate), _ptr(dest_row), T, k,
                                d, _dtype_code(dout), _ptr(dy_perm), _ptr(dgate), _stream(dev)))
    return dy_perm, dgate


def moe_permute_bwd(dx_perm: torch.Tensor, dest_row: torch.Tensor, T: int, k: int, *, out=None):
    """dx[t] = sum_j dx_perm[dest_row[t*k+j]]."""
    _dev(dx_perm, "dx_perm"), _dev(dest_row, "dest_row")
    d = dx_perm.shape[1]
    out = torch.empty((T, d), dtype=dx_perm.dtype, device=dx_perm.device) if out is None else out
    check(lib().moe_permute_bwd(_ptr(dx_perm), _ptr(dest_row), T, k, d, _dtype_code(dx_perm),
                                _ptr(out), _stream(dx_perm.device)))
    return out


def laep_rearrange(loads, n_groups: int):
    """Host utility (Algorithm 2).  Returns dict(group_of, order, sums)."""
    import numpy as np

    loads = np.ascontiguousarray(loads, dtype=np.float64)
    n = loads.shape[0]
    group_of = np.empty(n, dtype=np.int32)
    order = np.empty(n, dtype=np.int32)
    sums = np.empty(max(n_groups, 1), dtype=np.float64)
    check(lib().laep_rearrange(loads.ctypes.data, n, n_groups, group_of.ctypes.data,
                               order.ctypes.data, sums.ctypes.data))
    return dict(group_of=group_of, order=order, sums=sums[:n_groups])


# ---- measurement kernels (laep_calib.h) -----------------------------------------------
def laep_calib_copy(src: torch.Tensor, dst: torch.Tensor):
    """dst <- src (raw bytes) with the library's streaming copy kernel."""
    _dev(src, "src")
    _dev(dst, "dst")
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < nbytes:
        raise ValueError("dst is smaller than src")
    check(lib().laep_calib_copy(_ptr(src), _ptr(dst), nbytes, _stream(src.device)))


def laep_calib_read(src: torch.Tensor, block_bytes: int, out: torch.Tensor):
    """Blocked streaming read of src (laep_calib_read): one 512-thread
    workgroup per block_bytes, out float32 [n_blocks * 512]."""
    _dev(src, "src")
    _dev(out, "out")
    nbytes = src.numel() * src.element_size()
    if block_bytes <= 0 or out.dtype != torch.float32 or \
            out.numel() < (nbytes // block_bytes) * 512:
        raise ValueError("out must be float32 with (src bytes / block_bytes) * 512 elements")
    check(lib().laep_calib_read(_ptr(src), nbytes, int(block_bytes), _ptr(out),
                                _stream(src.device)))


def laep_calib_mfma(n_workgroups: int, iters: int, out: torch.Tensor):
    """bf16 MFMA loop: n_workgroups x 8 waves x iters x 8 MFMA 32x32x16."""
    _dev(out, "out")
    if out.dtype != torch.float32 or out.numel() < n_workgroups * 512:
        raise ValueError("out must be float32 with n_workgroups * 512 elements")
    check(lib().laep_calib_mfma(n_workgroups, iters, _ptr(out), _stream(out.device)))
