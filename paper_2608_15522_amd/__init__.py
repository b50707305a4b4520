"""Protected block-sparse video attention for MI355X (gfx950).

The video hot path of "Efficient Audio-Visual Generation via Synchrony-Aware
Cross-Modal Sparse Attention" (Sec. 4.1-4.2): cross-modal saliency, protected
block selection, the protected pooled-QK block mask and block-sparse flash
attention; beside it the lagged saliency update and token-granular protection
(Eq. (4), (8)-(11)) for either modality, the cross-modal attention forwards
with the saliency taken from their row log-sum-exps, the mask's block means
pooled inside the saliency streams (``sa_cross_scores_pooled`` +
``sa_build_block_mask_pooled``), and the
synchronization-aware cache-reuse indicator (Sec. 4.3).  Everything runs in
hand-written HIP kernels behind a C ABI (``include/sa.h``, ``libsa.so``); this
package is a thin ctypes binding over it.
"""
from .binding import (  # noqa: F401
    SaError, lib, sa_build_block_mask, sa_cross_scores, sa_last_error,
    sa_select_protected, sa_sparse_attention, sa_sparse_attention_noalloc, sa_version, sa_build_id, sa_workspace_size,
    sa_saliency_ema, sa_select_protected_tokens, sa_protected_token_attention,
    sa_cache_indicator, SA_CALL_CACHE_INDICATOR, SA_CALL_TOKEN_ATTENTION,
    sa_cross_attention, sa_cross_scores_from_lse, SA_CALL_CROSS_ATTENTION,
    sa_pool_columns, sa_cross_scores_pooled, sa_build_block_mask_pooled,
    SA_BF16, SA_F32, SA_CALL_CROSS_SCORES, SA_CALL_BUILD_BLOCK_MASK,
    SA_CALL_SPARSE_ATTENTION, SA_CALL_SELECT_PROTECTED, SA_OK,
    SA_ERR_INVALID_ARG, SA_ERR_UNSUPPORTED, SA_ERR_WORKSPACE, SA_ERR_HIP,
)
from .layer import protected_sparse_layer  # noqa: F401
