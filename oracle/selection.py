"""Top-k selection of the protected set (Sec. 4.1 Eq. (3), Sec. 4.2 Eq. (8)).

Test infrastructure only; see the package docstring.

Readings:
* Ties: the paper fixes no order.  The order used everywhere is "larger score
  first, then lower index first".
* Eq. (3) takes rho*N items from the current map, Eq. (8) takes ceil(rho*N)
  from the lagged map.  The budget is passed in as an integer (computed by the
  caller); which map (current or lagged) is ranked is the caller's choice.
* Granularity: blocks of video tokens (the block map is the token map summed
  per block).
"""
from __future__ import annotations

import numpy as np


def topk_order(scores, k):
    """Indices of the k largest entries of a 1-D array, in rank order
    (score descending, index ascending on equal scores)."""
    scores = np.asarray(scores, dtype=np.float64)
    n = scores.shape[0]
    if not 0 <= k <= n:
        raise ValueError(f"k={k} outside [0, {n}]")
    # A stable sort on the negated score keeps equal scores in index order.
    order = np.argsort(-scores, kind="stable")
    return order[:k].astype(np.int64)


def select_protected(sal_blk, k_prot):
    """Protected blocks per batch item (Eq. (8) at block level).

    Args:
        sal_blk: [B, n_b] block saliency.
        k_prot: number of protected blocks, 0 <= k_prot <= n_b.
    Returns:
        prot_idx [B, k_prot] int64 in rank order, prot_flag [B, n_b] uint8.
    """
    sal_blk = np.asarray(sal_blk, dtype=np.float64)
    B, n_b = sal_blk.shape
    prot_idx = np.zeros((B, k_prot), dtype=np.int64)
    prot_flag = np.zeros((B, n_b), dtype=np.uint8)
    for b in range(B):
        idx = topk_order(sal_blk[b], k_prot)
        prot_idx[b] = idx
        prot_flag[b, idx] = 1
    return prot_idx, prot_flag
