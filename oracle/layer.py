"""One layer of the method's video hot path, composed from the oracle steps,
and its exact work count (Sec. 4.4, Eq. (16)).

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

import numpy as np

from .saliency import cross_scores, token_to_block_saliency
from .selection import select_protected
from .mask import block_mask
from .attention import dense_attention, masked_attention
from .tokens import select_protected_tokens, token_protected_attention


def protected_sparse_layer(q_v, k_v, v_v, q_a, k_a, scale, block, k_keep,
                           k_prot, with_audio=True):
    """Saliency (Eq. (1)-(2)), protected blocks (Eq. (8)), protected block
    mask (Eq. (9)) and protected sparse attention (Eq. (10)/(11))."""
    s_v, s_a = cross_scores(q_a, k_v, scale,
                            q_v if with_audio else None,
                            k_a if with_audio else None)
    s_blk = token_to_block_saliency(s_v, block)
    prot_idx, prot_flag = select_protected(s_blk, k_prot)
    m = block_mask(q_v, k_v, scale, block, k_keep, prot_flag)
    O, lse = masked_attention(q_v, k_v, v_v, scale, block, m["kv_idx"],
                              m["kv_cnt"])
    return {"sal_v_tok": s_v, "sal_v_blk": s_blk, "sal_a_tok": s_a,
            "prot_idx": prot_idx, "prot_flag": prot_flag, **m,
            "O": O, "lse": lse}


def modality_protected_layer(q, k, v, sal_bar, scale, block, k_keep, k_tok):
    """Protected sparse self-attention of one modality m in {v, a}
    (Sec. 4.2, Eq. (8)-(11)).

    The protected query tokens P^m are the top ``k_tok`` = ceil(rho_m N_m)
    tokens of the lagged saliency map ``sal_bar`` [B, N_m] (Eq. (8), ties to
    the lower index); the sparse pattern S_m is the pooled-QK block top-k of
    the modality's own Q and K (Eq. (6)) with no block protection; a
    protected query keeps every key (Eq. (9)), any other query the key blocks
    of its query block (Eq. (11)).  For the audio branch ``sal_bar`` is the
    audio-token saliency of the v->a direction (Sec. 4.1)."""
    tok_idx, tok_flag = select_protected_tokens(sal_bar, k_tok)
    m = block_mask(q, k, scale, block, k_keep, None)
    O, lse = token_protected_attention(q, k, v, scale, block, m["kv_idx"],
                                       m["kv_cnt"], tok_flag)
    return {"tok_idx": tok_idx, "tok_flag": tok_flag, **m, "O": O, "lse": lse}


def cross_attention_with_saliency(q_a, k_a, v_a, q_v, k_v, v_v, scale):
    """The two cross-modal attention forwards of a layer and the saliency of
    Eq. (1)-(2) taken from the same softmax: O^a = softmax(Q^a (K^v)^T s) V^v
    and O^v = softmax(Q^v (K^a)^T s) V^a with their row log-sum-exps, and
    (s_v, s_a) the column masses of those two softmax matrices, summed over
    queries and heads and divided by H*L_a and H*L_v.  Returns a dict."""
    O_a, lse_a = dense_attention(q_a, k_v, v_v, scale)
    O_v, lse_v = dense_attention(q_v, k_a, v_a, scale)
    s_v, s_a = cross_scores(q_a, k_v, scale, q_v, k_a)
    return {"O_a": O_a, "lse_a": lse_a, "O_v": O_v, "lse_v": lse_v,
            "sal_v_tok": s_v, "sal_a_tok": s_a}


def computed_flops(kv_idx, kv_cnt, N, block, d):
    """Attention flops actually computed over kept pairs:
    ``4 * d * sum_r rows(r) * sum_{c in keep(r)} cols(c)`` (QK^T and PV, two
    flops per multiply-add), the exact form of Eq. (16)."""
    kv_idx = np.asarray(kv_idx)
    kv_cnt = np.asarray(kv_cnt)
    B, H, n_b = kv_cnt.shape
    lens = np.array([min((c + 1) * block, N) - c * block for c in range(n_b)],
                    dtype=np.int64)
    total = 0
    for b in range(B):
        for h in range(H):
            for r in range(n_b):
                cols = kv_idx[b, h, r, :kv_cnt[b, h, r]]
                total += int(lens[r]) * int(lens[cols].sum())
    return 4 * d * total


def dense_flops(B, H, N, d):
    """Flops of dense attention, Eq. (5): ``4 * B * H * N^2 * d``."""
    return 4 * B * H * N * N * d
