"""CPU oracle for the Action Cache sparse-FFN hot path (float64, NumPy).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this
package.  It shares no code with the GPU library and never calls it.
"""
from . import context_cache, group_masks
from .ffn import (ACTIVATIONS, RMS_EPS, anchor_stack, ceil_budget, compact_mask, contribution_score, delta_stack,
                  dense_ffn, ffn_input, ffn_stack, gelu_tanh, hidden, local_update, mask_multiplicity, masked_ffn,
                  mean_abs_activation, multiplicity, nested_topk_masks, rel_err, rms_norm, silu,
                  stack_masks_from_dense, topk_mask)

__all__ = ["ACTIVATIONS", "RMS_EPS", "anchor_stack", "ceil_budget", "compact_mask", "contribution_score",
           "context_cache", "delta_stack", "dense_ffn", "ffn_input", "ffn_stack", "gelu_tanh", "group_masks", "hidden",
           "local_update", "mask_multiplicity", "masked_ffn", "mean_abs_activation", "multiplicity",
           "nested_topk_masks", "rel_err", "rms_norm", "silu", "stack_masks_from_dense", "topk_mask"]
