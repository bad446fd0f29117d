"""E2S-Pruner token-scoring path on AMD Instinct MI355X (gfx950).

The computation lives in libe2s.so (HIP kernels behind the C ABI of
include/e2s.h); this package only builds and binds it.  Importing it without a
built library raises ImportError: there is no CPU fallback.
"""
from ._lib import (VARIANTS, CompactShape, E2SError, Image, Params, Pruner, QKViews,
                   RaggedPruner, RaggedShape, Shape, StagePruner, compact_tokens,
                   ds_combine_layers, fuse_evidence, fuse_select, head_masses, head_reliability,
                   layer_reliability, lib, make_params, make_shape, packed_images, prune,
                   prune_noalloc, prune_ragged, prune_stage, prune_views, qk_views, score_heads, spatial_select,
                   workspace_size)

__all__ = ["VARIANTS", "CompactShape", "E2SError", "Image", "Params", "Pruner", "QKViews",
           "RaggedPruner", "RaggedShape", "Shape", "StagePruner", "compact_tokens",
           "ds_combine_layers", "fuse_evidence", "fuse_select", "head_masses",
           "head_reliability", "layer_reliability", "lib", "make_params", "make_shape",
           "packed_images", "prune", "prune_noalloc", "prune_ragged", "prune_stage", "prune_views", "qk_views",
           "score_heads", "spatial_select", "workspace_size"]
