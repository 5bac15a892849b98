"""MI355X-native path-compositional MoE layer (PCoMoE, arXiv 2609.01024).

The layer runs in libpcomoe.so (hand-written HIP for gfx950) behind the C ABI in
include/pcomoe.h; this package is its thin Python binding. The library is loaded
on first use and there is no fallback path: if it is missing, calls raise.
"""
from .binding import (BETA_GLOBAL, BETA_PRODUCT, BETA_SRC_COND, PCM_BF16, PCM_BF16_F16DOWN, PCM_F32,
                      LayerPlan,
                      PathLayout, PathTable, ScoredLayerPlan, ScoredPathTable, Tuning,
                      layer_forward, lib, project_workspace_layout,
                      pcm_build_paths, pcm_dense_swiglu, pcm_expand, pcm_expand_scored,
                      pcm_layer_per_path, pcm_path_layout_build, pcm_project_combine, pcm_project_combine_noalloc,
                      pcm_project_combine_scored,
                      pcm_residual_add, pcm_route, pcm_route_logits, pcm_route_scored,
                      pcm_mask_pack, pcm_route_paths, pcm_widen_f16,
                      capture_graph, workspace_bytes)

__all__ = ["BETA_GLOBAL", "BETA_PRODUCT", "BETA_SRC_COND", "PCM_BF16", "PCM_BF16_F16DOWN", "PCM_F32",
           "LayerPlan",
           "PathLayout", "PathTable", "ScoredLayerPlan", "ScoredPathTable", "Tuning", "layer_forward",
           "lib", "project_workspace_layout",
           "pcm_build_paths", "pcm_dense_swiglu", "pcm_expand", "pcm_expand_scored",
           "pcm_layer_per_path", "pcm_path_layout_build", "pcm_project_combine", "pcm_project_combine_noalloc",
           "pcm_project_combine_scored",
           "pcm_residual_add", "pcm_route", "pcm_route_logits", "pcm_route_scored",
           "pcm_mask_pack", "pcm_route_paths", "pcm_widen_f16",
           "capture_graph", "workspace_bytes"]
