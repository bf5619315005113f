"""LAEP MoE layer on MI355X: Python binding of the liblaep_moe C ABI.

Steps of one MoE layer (the data-parallel hot path that Layer-Adaptive
Expert Pruning acts on), each a call into hand-written gfx950 HIP kernels:

    moe_route            router scoring + top-k gating
    moe_expert_counts    per-expert token loads (ETN), offsets, dispatch rows
    moe_route_count      the two above in one call (the router writes the count masks)
    laep_prune_mask      LAEP prune decision (alpha / beta thresholds)
    laep_expert_pruning  Algorithm 1 over a recorded ETN window (per-layer alpha)
    laep_compact_experts, laep_repack_experts   physical removal of pruned experts
    moe_permute          dispatch of token rows to expert order
    moe_grouped_ffn_fwd  grouped SwiGLU expert FFN (bf16 MFMA)
    moe_grouped_ffn_fwd_gather   the same with the dispatch folded into the operand loads
    moe_grouped_ffn_fwd_gather_combine   and, for one slot per token, the combine folded
                         into the down projection's epilogue
    moe_combine          gate-weighted combine
    moe_combine_bwd, moe_grouped_ffn_bwd, moe_permute_bwd   backward
    moe_route_bwd        router / gate backward (softmax Jacobian, dW_r, dx)
    laep_rearrange       host utility: balanced expert placement
    laep_calib_copy, laep_calib_read,  measurement kernels (attained peaks,
    laep_calib_mfma                    the router's feed bound)
"""
from ._lib import (  # noqa: F401
    LAEP_BF16, LAEP_CALL_FFN_BWD, LAEP_CALL_FFN_FWD, LAEP_F32, LaepError, LIB_PATH, lib)
from .api import (  # noqa: F401
    ffn_bwd_ws_views,
    ffn_fwd_h_view,
    laep_calib_copy,
    laep_calib_mfma,
    laep_calib_read,
    laep_compact_experts,
    laep_expert_pruning,
    laep_prune_mask,
    laep_rearrange,
    laep_repack_experts,
    moe_combine,
    moe_combine_bwd,
    moe_expert_counts,
    moe_grouped_ffn_bwd,
    moe_grouped_ffn_bwd_gather,
    moe_grouped_ffn_fwd,
    moe_grouped_ffn_fwd_gather,
    moe_grouped_ffn_fwd_gather_combine,
    moe_permute,
    moe_permute_bwd,
    moe_route,
    moe_route_bwd,
    moe_route_count,
    moe_route_count_noalloc,
    workspace_bytes,
)
from .layer import MoELayerPlan, layer_forward  # noqa: F401
from .placement import placement_report  # noqa: F401
from .pruning import ExpertPruner, compact_layer, hybrid_alpha  # noqa: F401
