"""Dense, sparse and protected sparse self-attention (Sec. 4.2, Eq. (5), (7),
(10) and the row form Eq. (11)).

Test infrastructure only; see the package docstring.

Readings:
* Self-attention is non-causal (the paper states no causal mask).
* A masked pair carries an additive -inf (Eq. (6), (9)), so its weight is
  exactly zero.  ``masked_attention`` therefore gathers, for each query row,
  only the key tokens of its kept blocks: the masked keys are never read,
  which is the row form of Eq. (11).  ``additive_mask_attention`` evaluates
  Eq. (10) literally with the full N x N additive mask, for small inputs.
* The last key block may be shorter than ``block``; it contributes only its
  true tokens.
* A row with no kept key (possible only in hand-built lists) is defined to
  output zeros and a log-sum-exp of -inf.
"""
from __future__ import annotations

import numpy as np


def dense_attention(q, k, v, scale):
    """Eq. (5): ``softmax(Q K^T * scale) V`` for [B, H, N, d] inputs.
    Returns (O [B, H, N, d], lse [B, H, N]) in float64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, N, d = q.shape
    O = np.zeros((B, H, N, v.shape[3]), dtype=np.float64)
    lse = np.zeros((B, H, N), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            S = scale * (q[b, h] @ k[b, h].T)
            m = S.max(axis=1, keepdims=True)
            p = np.exp(S - m)
            den = p.sum(axis=1, keepdims=True)
            O[b, h] = (p @ v[b, h]) / den
            lse[b, h] = (m + np.log(den))[:, 0]
    return O, lse


def key_tokens_of_row(kv_idx_row, kv_cnt_row, block, N):
    """Token indices of the kept key blocks of one query block, ascending
    within each block, blocks in list order."""
    toks = [np.arange(c * block, min((c + 1) * block, N))
            for c in np.asarray(kv_idx_row)[:int(kv_cnt_row)]]
    if not toks:
        return np.zeros(0, dtype=np.int64)
    return np.concatenate(toks)


def masked_attention(q, k, v, scale, block, kv_idx, kv_cnt, rows=None):
    """Protected sparse attention, Eq. (10) in its row form Eq. (11).

    Query block r of head (b, h) attends to the tokens of key blocks
    ``kv_idx[b, h, r, :kv_cnt[b, h, r]]``; protected query blocks carry the
    full list, so their rows are exactly dense rows (Eq. (11), first case).

    Args:
        q, k, v: [B, H, N, d].
        kv_idx: [B, H, n_b, >= max count] int, kv_cnt: [B, H, n_b] int.
        rows: optional iterable of (b, h, r) query blocks to evaluate; the
            default evaluates all of them.
    Returns:
        (O, lse): with ``rows`` None, O [B, H, N, d] and lse [B, H, N];
        otherwise dicts keyed by (b, h, r) holding that block's O rows
        [rows_in_block, d] and lse rows.
    """
    q = np.asarray(q)
    k = np.asarray(k)
    v = np.asarray(v)
    B, H, N, d = q.shape
    n_b = -(-N // block)
    full = rows is None
    if full:
        rows = [(b, h, r) for b in range(B) for h in range(H)
                for r in range(n_b)]
        O = np.zeros((B, H, N, v.shape[3]), dtype=np.float64)
        lse = np.full((B, H, N), -np.inf, dtype=np.float64)
    else:
        O, lse = {}, {}
    for (b, h, r) in rows:
        lo, hi = r * block, min((r + 1) * block, N)
        toks = key_tokens_of_row(kv_idx[b, h, r], kv_cnt[b, h, r], block, N)
        qb = np.asarray(q[b, h, lo:hi], dtype=np.float64)
        if toks.size == 0:
            o_blk = np.zeros((hi - lo, v.shape[3]), dtype=np.float64)
            l_blk = np.full(hi - lo, -np.inf, dtype=np.float64)
        else:
            kb = np.asarray(k[b, h, toks], dtype=np.float64)
            vb = np.asarray(v[b, h, toks], dtype=np.float64)
            S = scale * (qb @ kb.T)
            m = S.max(axis=1, keepdims=True)
            p = np.exp(S - m)
            den = p.sum(axis=1, keepdims=True)
            o_blk = (p @ vb) / den
            l_blk = (m + np.log(den))[:, 0]
        if full:
            O[b, h, lo:hi] = o_blk
            lse[b, h, lo:hi] = l_blk
        else:
            O[(b, h, r)] = o_blk
            lse[(b, h, r)] = l_blk
    return O, lse


def additive_mask_attention(q, k, v, scale, token_mask):
    """Eq. (7)/(10) evaluated literally: ``softmax(Q K^T * scale + M) V`` with
    ``M = 0`` where ``token_mask`` is true and ``-inf`` elsewhere.

    token_mask: [B, H, N, N] bool.  Small inputs only (N x N is formed)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, N, d = q.shape
    O = np.zeros((B, H, N, v.shape[3]), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            M = np.where(token_mask[b, h], 0.0, -np.inf)
            S = scale * (q[b, h] @ k[b, h].T) + M
            m = S.max(axis=1, keepdims=True)
            p = np.exp(S - m)
            O[b, h] = (p @ v[b, h]) / p.sum(axis=1, keepdims=True)
    return O
