"""Block mask of protected sparse attention (Sec. 4.2, Eq. (6) and (9)).

Test infrastructure only; see the package docstring.

The sparse pattern S_m of Eq. (6) is not specified by the paper beyond being
an intra-modal block pattern of a standard sparse-attention method with an
average keep ratio kappa (Sec. 4.4).  Reading taken: pooled-QK block top-k.

* Q and K are mean-pooled over each block of ``block`` consecutive tokens; the
  last block divides by its true (possibly shorter) length.
* Pooled score ``G[r, c] = scale * qbar_r . kbar_c``.
* Every non-protected query block r keeps the ``k_keep`` key blocks of largest
  G[r, :] (ties: lower block index first).  No diagonal is forced, no softmax
  or mass threshold is applied (a softmax is monotone and would not change
  the set).
* Eq. (9): a protected query block keeps every key block.  Protection restores
  rows only; protected blocks are not added to other rows' key sets.  The
  protected set is per batch item and shared by all heads.
"""
from __future__ import annotations

import numpy as np

from .selection import topk_order


def block_pool(x, block):
    """Mean over each block of consecutive tokens: [B, H, N, d] ->
    [B, H, n_b, d] (float64), the tail block averaged over its own length."""
    x = np.asarray(x, dtype=np.float64)
    B, H, N, d = x.shape
    n_b = -(-N // block)
    out = np.zeros((B, H, n_b, d), dtype=np.float64)
    for c in range(n_b):
        lo, hi = c * block, min((c + 1) * block, N)
        out[:, :, c, :] = x[:, :, lo:hi, :].sum(axis=2) / (hi - lo)
    return out


def pooled_scores(q, k, scale, block):
    """G[b, h, r, c] = scale * mean(Q block r) . mean(K block c)."""
    qb = block_pool(q, block)
    kb = block_pool(k, block)
    return scale * np.einsum("bhrd,bhcd->bhrc", qb, kb)


def block_mask(q, k, scale, block, k_keep, prot_flag=None):
    """Protected block mask M~ of Eq. (9) at block granularity.

    Args:
        q, k: [B, H, N, d].  scale: softmax scale.  block: tokens per block.
        k_keep: key blocks kept per non-protected query block, 1..n_b.
        prot_flag: [B, n_b] (nonzero = protected query block) or None.
    Returns:
        dict with ``mask`` [B, H, n_b, n_b] uint8 (1 = attend), ``kv_idx``
        [B, H, n_b, n_b] int64 (ascending kept key blocks, first kv_cnt valid,
        the rest -1), ``kv_cnt`` [B, H, n_b] int64 and ``G`` (float64).
    """
    G = pooled_scores(q, k, scale, block)
    B, H, n_b, _ = G.shape
    if not 1 <= k_keep <= n_b:
        raise ValueError(f"k_keep={k_keep} outside [1, {n_b}]")
    mask = np.zeros((B, H, n_b, n_b), dtype=np.uint8)
    for b in range(B):
        for h in range(H):
            for r in range(n_b):
                if prot_flag is not None and prot_flag[b, r]:
                    mask[b, h, r, :] = 1
                else:
                    mask[b, h, r, topk_order(G[b, h, r], k_keep)] = 1
    kv_idx, kv_cnt = kv_lists_from_mask(mask)
    return {"mask": mask, "kv_idx": kv_idx, "kv_cnt": kv_cnt, "G": G}


def kv_lists_from_mask(mask):
    """Compacted ascending key-block lists of a block mask."""
    mask = np.asarray(mask)
    B, H, n_b, _ = mask.shape
    kv_idx = np.full((B, H, n_b, n_b), -1, dtype=np.int64)
    kv_cnt = np.zeros((B, H, n_b), dtype=np.int64)
    for b in range(B):
        for h in range(H):
            for r in range(n_b):
                cols = np.nonzero(mask[b, h, r])[0]
                kv_cnt[b, h, r] = cols.size
                kv_idx[b, h, r, :cols.size] = cols
    return kv_idx, kv_cnt
