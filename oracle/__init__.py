"""CPU oracle for the E2S-Pruner scoring path.

Test infrastructure only: the test suite, the smoke check and the benchmark's
CPU-baseline leg may import it; the product path never does.
"""
from .e2s_oracle import (SCORE_MODES, VARIANTS, ImageResult, avg_tokens, cell_of_token,
                         compact_tokens,
                         cell_representatives, dempster_step, ds_combine_layers, head_masses,
                         head_reliability, normalized_attention, prune, prune_image,
                         prune_progressive, prune_stage, score_heads, softmax_over_visual,
                         spatial_select, support_from_attention, text_visual_logits)

__all__ = ["SCORE_MODES", "VARIANTS", "ImageResult", "avg_tokens", "cell_of_token",
           "compact_tokens",
           "cell_representatives", "dempster_step", "ds_combine_layers", "head_masses",
           "head_reliability", "normalized_attention", "prune", "prune_image",
           "prune_progressive", "prune_stage", "score_heads", "softmax_over_visual",
           "spatial_select", "support_from_attention", "text_visual_logits"]
