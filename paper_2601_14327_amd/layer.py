"""One MoE layer pass as a fixed chain of C-ABI calls on preallocated buffers.

Forward (router path):
    moe_route -> moe_expert_counts
      [-> laep_prune_mask -> moe_route(alive) -> moe_expert_counts]   (pruning)
    -> moe_permute -> moe_grouped_ffn_fwd -> moe_combine
Forward (given routing, one device's expert shard with k = 1):
    moe_expert_counts -> moe_permute -> moe_grouped_ffn_fwd -> moe_combine
With fused dispatch (bf16, the default), moe_permute + moe_grouped_ffn_fwd
become one moe_grouped_ffn_fwd_gather call that reads the token rows through
row_src, and the backward reads them the same way
(moe_grouped_ffn_bwd_gather), so a training step never writes x_perm; that
call also forms dY = g * dout on load, so moe_combine_bwd writes only the
gate gradient and a training step never writes dy_perm either.  A forward
that keeps its activations for inspection (save_act without a backward)
still writes x_perm.
With one slot per token (k = 1) the combine folds in as well
(moe_grouped_ffn_fwd_gather_combine): the down projection writes each row,
times its gate, to its token row; y_perm is written only for a backward pass.
Backward:
    moe_combine_bwd -> moe_grouped_ffn_bwd[_gather] -> moe_permute_bwd
      [-> moe_route_bwd, accumulating the router's dx]   (router path)
In a training step the router's weight gradients need only the gate gradient:
backward(router=...) runs them on a side stream beside the expert backward and
takes the router's dx after moe_permute_bwd.

All buffers are allocated once, so a pass makes no allocation and no host
synchronisation; every step runs in the library's kernels on the current
stream.
"""
from __future__ import annotations

import math
from typing import Optional

import torch

from . import api
from ._lib import LAEP_CALL_COUNTS, LAEP_CALL_FFN_BWD, LAEP_CALL_FFN_FWD, LAEP_CALL_ROUTE_BWD


class MoELayerPlan:
    def __init__(self, T: int, d_model: int, E: int, k: int, d_ff: int,
                 dtype: torch.dtype = torch.bfloat16, device="cuda", backward: bool = False,
                 save_act: Optional[bool] = None, fused_dispatch: Optional[bool] = None):
        self.T, self.d, self.E, self.k, self.f = T, d_model, E, k, d_ff
        self.R = T * k
        self.dtype = dtype
        dev = torch.device(device)
        self.device = dev
        i32 = torch.int32
        R = self.R
        self.topk_idx = torch.empty((T, k), dtype=i32, device=dev)
        self.topk_gate = torch.empty((T, k), dtype=torch.float32, device=dev)
        self.counts = torch.empty(E, dtype=i32, device=dev)
        self.offsets = torch.empty(E + 1, dtype=i32, device=dev)
        self.dest_row = torch.empty(R, dtype=i32, device=dev)
        self.alive = torch.empty(E, dtype=torch.uint8, device=dev)
        self.n_pruned = torch.empty(1, dtype=i32, device=dev)
        # pre-activations are kept when a backward pass will read them (or on request)
        save_act = backward if save_act is None else save_act
        # the dispatch folds into the FFN's operand loads (bf16), forward and
        # backward; x_perm is kept only unfused, or for a forward that keeps its
        # activations without a backward (inspection)
        if fused_dispatch is None:
            fused_dispatch = dtype == torch.bfloat16
        self.fused = bool(fused_dispatch)
        self.x_perm = (None if self.fused and (backward or not save_act) else
                       torch.empty((R, d_model), dtype=dtype, device=dev))
        self.x_in = None   # the token rows of the last forward (the gathered backward reads them)
        # the dispatch order is kept when the FFN gathers through it or the
        # router backward sums dW_r over it
        self.row_src = (torch.empty(R, dtype=i32, device=dev) if self.fused or backward
                        else None)
        # one slot per token (bf16): the combine folds into the down projection's
        # epilogue; y_perm is then written only for the backward (combine_bwd) or
        # when the caller keeps the activations (save_act)
        self.fused_combine = k == 1 and self.fused
        self.y_perm = (None if self.fused_combine and not (backward or save_act) else
                       torch.empty((R, d_model), dtype=dtype, device=dev))
        self.act_save = (torch.empty((R, 2 * d_ff), dtype=dtype, device=dev) if save_act
                         else None)
        self.out = torch.empty((T, d_model), dtype=dtype, device=dev)
        self.ws_counts = torch.empty(max(1, api.workspace_bytes(LAEP_CALL_COUNTS, T, k, E)),
                                     dtype=torch.uint8, device=dev)
        self.ws_ffn = torch.empty(api.workspace_bytes(LAEP_CALL_FFN_FWD, R, 1, E, d_model, d_ff),
                                  dtype=torch.uint8, device=dev)
        if backward:
            # fused plans form dY on load in the expert backward (no dy_perm)
            self.dy_perm = (None if self.fused else
                            torch.empty((R, d_model), dtype=dtype, device=dev))
            self.dx_perm = torch.empty((R, d_model), dtype=dtype, device=dev)
            self.dgate = torch.empty((T, k), dtype=torch.float32, device=dev)
            self.dx = torch.empty((T, d_model), dtype=dtype, device=dev)
            self.ws_bwd = torch.empty(
                api.workspace_bytes(LAEP_CALL_FFN_BWD, R, 1, E, d_model, d_ff),
                dtype=torch.uint8, device=dev)
            self.dw_gate_up = None
            self.dw_down = None
            self.dw_router = None
            self.dbias = None
            rb = max(1, api.workspace_bytes(LAEP_CALL_ROUTE_BWD, T, k, E, d_model))
            self.ws_route_bwd = torch.empty(rb, dtype=torch.uint8, device=dev)
            # the router's weight gradients run on a side stream beside the expert
            # backward, with a workspace of their own
            self.ws_route_bwd_w = torch.empty(rb, dtype=torch.uint8, device=dev)
            self._side = None
            self._side_done = None

    # -- pieces --------------------------------------------------------------
    def route(self, x, w_router, bias=None, alive=None, renorm=True):
        api.moe_route(x, w_router, self.k, bias=bias, alive=alive, renorm=renorm,
                      topk_idx=self.topk_idx, topk_gate=self.topk_gate)

    def count(self, etn_accum=None):
        api.moe_expert_counts(self.topk_idx, self.E, ws=self.ws_counts, counts=self.counts,
                              offsets=self.offsets, dest_row=self.dest_row,
                              row_src=self.row_src, etn_accum=etn_accum)

    def route_count(self, x, w_router, bias=None, alive=None, renorm=True, etn_accum=None):
        """route + count in one call (the router also writes the count masks)."""
        api.moe_route_count(x, w_router, self.k, bias=bias, alive=alive, renorm=renorm,
                            etn_accum=etn_accum, ws=self.ws_counts, topk_idx=self.topk_idx,
                            topk_gate=self.topk_gate, counts=self.counts, offsets=self.offsets,
                            dest_row=self.dest_row, row_src=self.row_src)

    def prune(self, beta: float, alpha: float = math.inf):
        api.laep_prune_mask(self.counts, self.T * self.k, alpha, beta, alive=self.alive,
                            n_pruned=self.n_pruned)

    def experts_and_combine(self, x, w_gate_up, w_down, expert_map=None):
        self.x_in = x
        if self.fused_combine:
            api.moe_grouped_ffn_fwd_gather_combine(
                x, self.row_src, self.topk_gate, w_gate_up, w_down, self.offsets, rows=self.R,
                expert_map=expert_map, ws=self.ws_ffn, out=self.out,
                keep_y=self.y_perm is not None, y_perm=self.y_perm,
                save_act=self.act_save is not None, act_save=self.act_save,
                x_perm_out=self.x_perm)
            return self.out
        if self.fused:
            # x_perm (kept for inspection only) by the token-major permute, which
            # reads each token row once
            if self.x_perm is not None:
                api.moe_permute(x, self.dest_row, self.k, self.R, out=self.x_perm)
            api.moe_grouped_ffn_fwd_gather(x, self.row_src, self.k, w_gate_up, w_down,
                                           self.offsets, rows=self.R, expert_map=expert_map,
                                           ws=self.ws_ffn, y_perm=self.y_perm,
                                           save_act=self.act_save is not None,
                                           act_save=self.act_save)
        else:
            api.moe_permute(x, self.dest_row, self.k, self.R, out=self.x_perm)
            api.moe_grouped_ffn_fwd(self.x_perm, w_gate_up, w_down, self.offsets,
                                    expert_map=expert_map, ws=self.ws_ffn, y_perm=self.y_perm,
                                    save_act=self.act_save is not None, act_save=self.act_save)
        api.moe_combine(self.y_perm, self.topk_gate, self.dest_row, out=self.out)
        return self.out

    # -- whole passes ----------------------------------------------------------
    def forward(self, x, w_router, w_gate_up, w_down, bias=None, renorm=True,
                prune_beta: Optional[float] = None, prune_alpha: float = math.inf):
        self.route_count(x, w_router, bias=bias, renorm=renorm)
        if prune_beta is not None:
            self.prune(prune_beta, prune_alpha)
            self.route_count(x, w_router, bias=bias, alive=self.alive, renorm=renorm)
        return self.experts_and_combine(x, w_gate_up, w_down)

    def forward_given_routing(self, x, topk_idx, topk_gate, w_gate_up, w_down):
        self.topk_idx.copy_(topk_idx)
        self.topk_gate.copy_(topk_gate)
        self.count()
        return self.experts_and_combine(x, w_gate_up, w_down)

    def route_backward(self, x, w_router, renorm=True, want_dbias=False):
        """Router / gate backward from self.dgate (the combine's gate gradient),
        accumulated onto self.dx.  Renormalised gates only (the full-softmax
        form needs the logits, which the plan does not keep)."""
        if not renorm:
            raise NotImplementedError("the plan keeps no logits; call moe_route_bwd directly")
        if self.dw_router is None:
            self.dw_router = torch.empty(w_router.shape, dtype=torch.float32, device=self.device)
            self.dbias = torch.empty(self.E, dtype=torch.float32, device=self.device)
        api.moe_route_bwd(self.dgate, self.topk_idx, self.topk_gate, x, w_router, renorm=True,
                          offsets=self.offsets, row_src=self.row_src, dx=self.dx,
                          accumulate_dx=True, dw_router=self.dw_router,
                          dbias=self.dbias if want_dbias else None, ws=self.ws_route_bwd)
        return self.dx, self.dw_router

    def route_backward_weights_async(self, x, w_router, want_dbias=False):
        """dw_router (and dbias) from self.dgate on a side stream, started now:
        they need only the gate gradient, so they can run beside the expert
        backward.  route_backward_data waits for them."""
        if self.dw_router is None:
            self.dw_router = torch.empty(w_router.shape, dtype=torch.float32, device=self.device)
            self.dbias = torch.empty(self.E, dtype=torch.float32, device=self.device)
        if self._side is None:
            self._side = torch.cuda.Stream(device=self.device)   # default priority
            self._side_done = torch.cuda.Event()
        main = torch.cuda.current_stream(self.device)
        self._side.wait_stream(main)
        with torch.cuda.stream(self._side):
            api.moe_route_bwd(self.dgate, self.topk_idx, self.topk_gate, x, w_router,
                              renorm=True, offsets=self.offsets, row_src=self.row_src,
                              data=False, dw_router=self.dw_router,
                              want_dbias=want_dbias, dbias=self.dbias if want_dbias else None,
                              ws=self.ws_route_bwd_w)
            self._side_done.record(self._side)

    def route_backward_data(self, x, w_router):
        """The router's dx, accumulated onto self.dx; then the current stream
        waits for route_backward_weights_async."""
        api.moe_route_bwd(self.dgate, self.topk_idx, self.topk_gate, x, w_router, renorm=True,
                          offsets=self.offsets, row_src=self.row_src, dx=self.dx,
                          accumulate_dx=True, weights=False, ws=self.ws_route_bwd)
        torch.cuda.current_stream(self.device).wait_event(self._side_done)
        return self.dx, self.dw_router

    def backward(self, dout, w_gate_up, w_down, expert_map=None, accumulate=False,
                 router=None, want_dbias=False):
        """Expert backward; with router=(x, w_router) (renormalised gates) also
        the router's, its weight gradients beside the expert backward."""
        api.moe_combine_bwd(dout, self.y_perm, self.topk_gate, self.dest_row,
                            dy_perm=self.dy_perm, dgate=self.dgate,
                            want_dy=self.dy_perm is not None)
        if router is not None:
            self.route_backward_weights_async(router[0], router[1], want_dbias=want_dbias)
        if self.dw_gate_up is None:
            self.dw_gate_up = torch.empty(w_gate_up.shape, dtype=torch.float32,
                                          device=self.device)
            self.dw_down = torch.empty(w_down.shape, dtype=torch.float32, device=self.device)
        # dW_d from the H the forward computed (left in its workspace)
        h_fwd = api.ffn_fwd_h_view(self.ws_ffn, self.R, self.f, self.dtype)
        if self.fused:   # X gathered from the forward's token rows, dY formed on load
            api.moe_grouped_ffn_bwd_gather(None, self.x_in, self.row_src, self.k,
                                           self.act_save, w_gate_up, w_down, self.offsets,
                                           dout=dout, topk_gate=self.topk_gate,
                                           h_fwd=h_fwd, expert_map=expert_map,
                                           dw_gate_up=self.dw_gate_up, dw_down=self.dw_down,
                                           accumulate=accumulate, ws=self.ws_bwd,
                                           dx_perm=self.dx_perm)
        else:
            api.moe_grouped_ffn_bwd(self.dy_perm, self.x_perm, self.act_save, w_gate_up,
                                    w_down, self.offsets, h_fwd=h_fwd, expert_map=expert_map,
                                    dw_gate_up=self.dw_gate_up, dw_down=self.dw_down,
                                    accumulate=accumulate, ws=self.ws_bwd, dx_perm=self.dx_perm)
        api.moe_permute_bwd(self.dx_perm, self.dest_row, self.T, self.k, out=self.dx)
        if router is not None:
            self.route_backward_data(router[0], router[1])
        return self.dx, self.dgate, self.dw_gate_up, self.dw_down


def layer_forward(x, w_router, w_gate_up, w_down, k, bias=None, renorm=True,
                  prune_beta=None, prune_alpha=math.inf):
    """One forward pass with freshly allocated buffers; returns the plan."""
    T, d = x.shape
    E = w_router.shape[0]
    f = w_down.shape[2]
    plan = MoELayerPlan(T, d, E, k, f, dtype=x.dtype, device=x.device)
    plan.forward(x, w_router, w_gate_up, w_down, bias=bias, renorm=renorm,
                 prune_beta=prune_beta, prune_alpha=prune_alpha)
    return plan
