"""Token-granular protection and the lagged saliency cache (Sec. 4.1 Eq. (4)
and Eq. (3)/(8) at token level; Sec. 4.2 Eq. (9)-(11) with protected query
tokens).

Test infrastructure only; see the package docstring.

Readings:
* Eq. (4) gives no value for alpha: it is a parameter here.  The refresh
  interval (every K denoising steps, K = 4 in Sec. 5) is the caller's
  schedule; ``saliency_ema`` is one update.
* The protected set of Eq. (8) is per batch item and shared by all heads,
  because the saliency map of Eq. (2) sums over heads.  Its size
  k_tok = ceil(rho * N) is passed in as an integer.  Ties: larger saliency
  first, then lower token index.
* Eq. (9)-(11): a protected query token keeps every key (its row of the mask
  is all zero, ``DenseAttn``); every other query token keeps the key blocks
  of its query block in the sparse pattern S_m (Eq. (6)), ``SparseAttn``.
"""
from __future__ import annotations

import numpy as np

from .attention import masked_attention
from .selection import topk_order


def saliency_ema(s_bar_prev, s, alpha):
    """Eq. (4): ``alpha * s_bar_prev + (1 - alpha) * s`` in float64."""
    s_bar_prev = np.asarray(s_bar_prev, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    return alpha * s_bar_prev + (1.0 - alpha) * s


def select_protected_tokens(sal_tok, k_tok):
    """Protected query tokens per batch item (Eq. (8) at token level).

    Args:
        sal_tok: [B, N] token saliency (the lagged map of Eq. (4)).
        k_tok: number of protected tokens, 0 <= k_tok <= N.
    Returns:
        tok_idx [B, k_tok] int64, ascending token order; tok_flag [B, N] uint8.
    """
    sal_tok = np.asarray(sal_tok, dtype=np.float64)
    B, N = sal_tok.shape
    tok_idx = np.zeros((B, k_tok), dtype=np.int64)
    tok_flag = np.zeros((B, N), dtype=np.uint8)
    for b in range(B):
        idx = np.sort(topk_order(sal_tok[b], k_tok))
        tok_idx[b] = idx
        tok_flag[b, idx] = 1
    return tok_idx, tok_flag


def token_protected_attention(q, k, v, scale, block, kv_idx, kv_cnt, tok_flag):
    """Eq. (11) with protected query tokens.

    Args:
        q, k, v: [B, H, N, d].
        kv_idx, kv_cnt: the sparse pattern S_m as key-block lists per query
            block (no block-level protection).
        tok_flag: [B, N], nonzero for protected query tokens (all heads).
    Returns:
        (O [B, H, N, d], lse [B, H, N]) in float64: a protected token's row is
        the dense softmax over all N keys, any other row the block-sparse one.
    """
    q = np.asarray(q)
    k = np.asarray(k)
    v = np.asarray(v)
    B, H, N, d = q.shape
    O, lse = masked_attention(q, k, v, scale, block, kv_idx, kv_cnt)
    for b in range(B):
        rows = np.nonzero(np.asarray(tok_flag[b]))[0]
        if rows.size == 0:
            continue
        for h in range(H):
            qr = np.asarray(q[b, h, rows], dtype=np.float64)
            kh = np.asarray(k[b, h], dtype=np.float64)
            vh = np.asarray(v[b, h], dtype=np.float64)
            S = scale * (qr @ kh.T)
            m = S.max(axis=1, keepdims=True)
            p = np.exp(S - m)
            den = p.sum(axis=1, keepdims=True)
            O[b, h, rows] = (p @ vh) / den
            lse[b, h, rows] = (m + np.log(den))[:, 0]
    return O, lse


def token_protected_rows(q, k, v, scale, tok_idx, rows):
    """Dense rows of selected protected tokens only: for each (b, h, j) in
    ``rows`` the output and log-sum-exp of token ``tok_idx[b, j]`` over all
    keys (Eq. (11), first case).  Returns dicts keyed by (b, h, j)."""
    O, lse = {}, {}
    for (b, h, j) in rows:
        t = int(tok_idx[b, j])
        qr = np.asarray(q[b, h, t], dtype=np.float64)
        kh = np.asarray(k[b, h], dtype=np.float64)
        vh = np.asarray(v[b, h], dtype=np.float64)
        S = scale * (kh @ qr)
        m = S.max()
        p = np.exp(S - m)
        den = p.sum()
        O[(b, h, j)] = (p @ vh) / den
        lse[(b, h, j)] = m + np.log(den)
    return O, lse
