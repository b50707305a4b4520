"""Synchronization-aware cache-reuse indicator (Sec. 4.3, Eq. (12)-(15)).

Test infrastructure only; see the package docstring.

Readings:
* One decision per (denoising step, block): every norm runs over the whole
  block output, all batch items and channels together.  Block outputs are
  [B, L, C] (token rows of C channels).
* Eq. (13) restricts both norms to the rows of the protected video tokens
  P_v (the token set of Eq. (8), one set per batch item).
* Eq. (14) takes the inner product and the 2-norms over the whole saliency
  map [B, L_v].
* epsilon is not given by the paper: it is a parameter.  A missing audio
  stream or saliency pair contributes 0 to the max of Eq. (15).
* The block is reused iff Delta_sync < tau (strict, Eq. (15) text).
"""
from __future__ import annotations

import numpy as np


def relative_l1(y, y_hat, eps, rows=None):
    """Eq. (12)/(13): ||Y - Y_hat||_1 / (||Y||_1 + eps); ``rows`` is an
    optional [B, L] boolean row selection."""
    y = np.asarray(y, dtype=np.float64)
    y_hat = np.asarray(y_hat, dtype=np.float64)
    diff = np.abs(y - y_hat)
    mag = np.abs(y)
    if rows is not None:
        sel = np.asarray(rows, dtype=bool)
        diff = diff[sel]
        mag = mag[sel]
    return float(diff.sum() / (mag.sum() + eps))


def saliency_drift(s_bar, s_hat, eps):
    """Eq. (14): 1 - <s_bar, s_hat> / (||s_bar||_2 ||s_hat||_2 + eps)."""
    a = np.asarray(s_bar, dtype=np.float64).ravel()
    b = np.asarray(s_hat, dtype=np.float64).ravel()
    return float(1.0 - (a @ b) / (np.sqrt(a @ a) * np.sqrt(b @ b) + eps))


def cache_indicator(y_v, y_v_hat, prot_flag, y_a, y_a_hat, s_bar, s_hat,
                    lambda_p, lambda_s, tau, eps):
    """Eq. (15).  Returns dict(dv, da, dp, ds, sync, reuse)."""
    dv = relative_l1(y_v, y_v_hat, eps)
    da = relative_l1(y_a, y_a_hat, eps) if y_a is not None else 0.0
    dp = relative_l1(y_v, y_v_hat, eps, rows=prot_flag) if prot_flag is not None else 0.0
    ds = saliency_drift(s_bar, s_hat, eps) if s_bar is not None else 0.0
    sync = max(dv, da, lambda_p * dp, lambda_s * ds)
    return dict(dv=dv, da=da, dp=dp, ds=ds, sync=sync, reuse=bool(sync < tau))
