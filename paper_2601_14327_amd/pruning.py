"""LAEP expert pruning over a recorded window, and physical compaction.

Algorithm 1 (Appendix) records the tokens every expert of every layer
receives over ITER training iterations (Step 1), marks low-load experts per
iteration and layer with the Eq. (1)-(2) rule (Step 2), and prunes per layer
the most-marked experts (Step 3).  Pruned experts then leave the model
(Section 3.2): the survivors' router rows and FFN weights are repacked into
compact tensors and the layer runs with E' = n_alive experts.

Every step runs on the device: recording through moe_expert_counts'
``etn_accum``, the decision in ``laep_expert_pruning``, the slot map in
``laep_compact_experts`` and the copy in ``laep_repack_experts``.  Reading the
survivor counts back to size the compact tensors is the one synchronisation,
once per pruning event.
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Sequence

import torch

from . import api


def hybrid_alpha(n_layers: int, edge: float = 0.2, middle: float = 0.4):
    """Per-layer alpha: ``edge`` on the first and last sixth of the layers,
    ``middle`` on the rest (the schedule of the Section 3.4 ablation and of the
    Section 4 pre-training run).  A sixth of L layers is round(L / 6), halves
    rounded up."""
    if n_layers < 1:
        raise ValueError("n_layers must be >= 1")
    n_edge = int(math.floor(n_layers / 6 + 0.5))
    return [edge if (l < n_edge or l >= n_layers - n_edge) else middle for l in range(n_layers)]


class ExpertPruner:
    """ETN window [ITER, L, E] (int64, on the device) and the pruning decision.

    ``slot(it, layer)`` is the int64 [E] row that moe_expert_counts adds the
    layer's loads of iteration ``it`` into (its ``etn_accum`` argument).
    """

    def __init__(self, iters: int, n_layers: int, E: int, tokens: int, k: int,
                 alpha, beta: float, device="cuda"):
        if iters < 1:
            raise ValueError("iters must be >= 1")
        self.iters, self.n_layers, self.E = iters, n_layers, E
        self.total = int(tokens) * int(k)                      # S * topK
        self.alpha = ([float(alpha)] * n_layers if isinstance(alpha, (int, float))
                      else [float(a) for a in alpha])
        if len(self.alpha) != n_layers:
            raise ValueError(f"alpha has {len(self.alpha)} entries for {n_layers} layers")
        self.beta = float(beta)
        self.etn = torch.zeros((iters, n_layers, E), dtype=torch.int64, device=device)

    def slot(self, it: int, layer: int) -> torch.Tensor:
        return self.etn[it, layer]

    def reset(self):
        self.etn.zero_()

    def decide(self, want_marker: bool = False):
        """(alive [L, E] uint8, n_pruned [L] int32, marker or None), on the device."""
        return api.laep_expert_pruning(self.etn, self.total, self.alpha, self.beta,
                                       want_marker=want_marker)


def compact_layer(alive: torch.Tensor, *, w_router: torch.Tensor, w_gate_up: torch.Tensor,
                  w_down: torch.Tensor, bias: Optional[torch.Tensor] = None,
                  extra: Sequence[Dict[str, torch.Tensor]] = ()):
    """Remove one layer's pruned experts.

    alive [E] uint8 (device).  Returns a dict with ``expert_map`` [E] (logical
    id -> slot, -1 pruned), ``n_alive``, the compact ``w_router`` [E', d],
    ``w_gate_up`` [E', 2f, d], ``w_down`` [E', d, f], ``bias`` [E'] (if given),
    and ``extra``: the same repack applied to each further dict of per-expert
    tensors (optimizer states, fp32 master weights).
    """
    expert_map, n_alive_t = api.laep_compact_experts(alive)
    n_alive = int(n_alive_t[0].item())                       # sizes the compact tensors
    out = api.laep_repack_experts(expert_map, n_alive, w_router=w_router, bias=bias,
                                  w_gate_up=w_gate_up, w_down=w_down)
    res = dict(expert_map=expert_map, n_alive=n_alive, **out)
    res["extra"] = [api.laep_repack_experts(expert_map, n_alive, **x) for x in extra]
    return res
