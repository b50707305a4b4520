"""Cross-modal saliency (Sec. 4.1, Eq. (1)-(2) and the reverse direction).

Test infrastructure only; see the package docstring.

Readings taken where the paper is silent:

* ``Norm`` in Eq. (2) is not defined.  It is read as L1 normalisation by the
  exact constant ``H * N_a`` (a->v) or ``H * N_v`` (v->a): every softmax row
  sums to one, so the normalised map sums to one per batch item.  Any positive
  rescaling would leave the top-k unchanged.
* The layer set L_c is not given.  One layer is scored per call; summing over
  layers is the caller's job (``accumulate``).
* Keys are the video tokens only (a->v) or the audio tokens only (v->a), with
  no mask, no bias and no causality; Q and K are taken as given.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor

import numpy as np


def _softmax_rows(logits: np.ndarray) -> np.ndarray:
    """Row softmax of a 2-D float64 array (max-shifted for range only)."""
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    return e / e.sum(axis=1, keepdims=True)


def _column_mass(q, k, scale):
    """Column sums of the row softmax of ``scale * q k^T`` (one head)."""
    return _softmax_rows(scale * (q @ k.T)).sum(axis=0)


def _direction(q, k, scale, workers):
    """sum_h of the column mass, per batch item, heads added in order."""
    B, H = q.shape[:2]
    jobs = [(b, h) for b in range(B) for h in range(H)]
    run = lambda bh: _column_mass(np.asarray(q[bh], dtype=np.float64),
                                  np.asarray(k[bh], dtype=np.float64), scale)
    if workers > 1:
        with ThreadPoolExecutor(max_workers=workers) as ex:
            cols = list(ex.map(run, jobs))
    else:
        cols = [run(bh) for bh in jobs]
    out = np.zeros((B, k.shape[2]), dtype=np.float64)
    for (b, h), c in zip(jobs, cols):
        out[b] += c
    return out


def cross_scores(q_a, k_v, scale, q_v=None, k_a=None, workers=1):
    """Token saliency of both modalities for one layer.

    Eq. (1): ``A^{a->v} = softmax(Q^a (K^v)^T * scale)`` per batch item and
    head, rows indexed by audio queries j, columns by video keys i.
    Eq. (2): ``s^v_i = Norm(sum_h sum_j A^{a->v}[j, i])``.
    Reverse direction (the sentence after Eq. (2)): ``A^{v->a}`` with video
    queries and audio keys, ``s^a_j = Norm(sum_h sum_i A^{v->a}[i, j])``.

    Args:
        q_a: [B, H, N_a, d] audio queries.  k_v: [B, H, N_v, d] video keys.
        q_v: [B, H, N_v, d] video queries, k_a: [B, H, N_a, d] audio keys;
            both None to skip the reverse direction.
        scale: the softmax scale (1/sqrt(d_h)).
        workers: heads evaluated concurrently (threads); the per-head terms
            are still added in head order, so the result does not depend on it.
    Returns:
        (s_v [B, N_v], s_a [B, N_a] or None), float64, each row summing to 1.
    """
    H, N_a = q_a.shape[1], q_a.shape[2]
    s_v = _direction(q_a, k_v, scale, workers) / (H * N_a)
    s_a = None
    if q_v is not None:
        N_v = q_v.shape[2]
        s_a = _direction(q_v, k_a, scale, workers) / (H * N_v)
    return s_v, s_a


def token_to_block_saliency(s_tok, block):
    """Block saliency: the sum of token saliency over each block of ``block``
    consecutive video tokens (the last block may be shorter and counts only
    its own tokens).

    Reading: the protected set is chosen at block granularity, and a block's
    score is the total saliency mass of its tokens, so that choosing the top
    blocks maximises the protected saliency mass (Eq. (3) ranks tokens).
    """
    s_tok = np.asarray(s_tok, dtype=np.float64)
    B, N = s_tok.shape
    n_b = -(-N // block)
    out = np.zeros((B, n_b), dtype=np.float64)
    for c in range(n_b):
        out[:, c] = s_tok[:, c * block:min((c + 1) * block, N)].sum(axis=1)
    return out
