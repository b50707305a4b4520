"""Plain fp64 CPU oracle for protected block-sparse video self-attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls, links
or executes this package: only the tests, the smoke check and the CPU-baseline
leg of the benchmark do.  It shares no code with the HIP kernels or their
binding, and it imports nothing from them.

It computes, in float64 with numpy, what the method defines (Sec. 4 of the
paper, "Efficient Audio-Visual Generation via Synchrony-Aware Cross-Modal
Sparse Attention"):

* ``saliency``   -- Eq. (1)-(2): a->v cross-attention probabilities summed over
  audio queries and heads into a video-token saliency map, and the reverse
  v->a direction into an audio-token saliency map (Sec. 4.1);
* ``selection``  -- Eq. (3)/(8): protected set by top-k with a fixed
  tie-break (lower index wins), at block granularity;
* ``mask``       -- Eq. (6) and (9): the sparse pattern S_m as pooled-QK block
  top-k per query block, OR-ed with full rows for protected query blocks;
* ``attention``  -- Eq. (5), (7), (10)/(11): dense and masked softmax attention;
* ``tokens``     -- Eq. (4) lagged saliency update, Eq. (8) at token level and
  Eq. (11) with protected query tokens (dense rows over the block pattern);
* ``cache``      -- Eq. (12)-(15): the synchronization-aware cache-reuse
  indicator (relative L1 changes, protected-row change, saliency drift);
* ``layer``      -- the steps composed: the video layer with protected blocks,
  token-protected sparse self-attention of either modality (Eq. (8)-(11),
  m in {v, a}; the audio branch with the audio-token saliency), and the two
  cross-modal attention forwards with the saliency of their softmax.

Where the paper is silent or ambiguous the reading taken is stated in the
function that depends on it.  Parity status: every public function here is
pinned by a CPU test against a closed form, an invariant, a library special
case or brute force; none is "parity unpinned".
"""
from .saliency import cross_scores, token_to_block_saliency
from .selection import topk_order, select_protected
from .mask import block_pool, pooled_scores, block_mask, kv_lists_from_mask
from .attention import (dense_attention, masked_attention,
                        additive_mask_attention, key_tokens_of_row)
from .layer import (protected_sparse_layer, modality_protected_layer,
                    cross_attention_with_saliency, computed_flops, dense_flops)
from .tokens import (saliency_ema, select_protected_tokens,
                     token_protected_attention, token_protected_rows)
from .cache import relative_l1, saliency_drift, cache_indicator

__all__ = [
    "cross_scores", "token_to_block_saliency", "topk_order",
    "select_protected", "block_pool", "pooled_scores", "block_mask",
    "kv_lists_from_mask", "dense_attention", "masked_attention",
    "additive_mask_attention", "key_tokens_of_row", "protected_sparse_layer",
    "modality_protected_layer", "cross_attention_with_saliency",
    "computed_flops", "dense_flops", "saliency_ema", "select_protected_tokens",
    "token_protected_attention", "token_protected_rows", "relative_l1",
    "saliency_drift", "cache_indicator",
]
