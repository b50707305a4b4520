"""One layer of the video hot path, as four C-ABI calls on one stream.

``LayerPlan`` allocates every output and workspace once (with torch), so a
``run()`` enqueues only the library's kernels: saliency (Eq. (1)-(2)),
protected selection (Eq. (8)), protected block mask (Eq. (9)) and protected
block-sparse attention (Eq. (10)/(11)).  ``run_pooled()`` is the same layer
with the mask's block means (Eq. (6)) taken from the saliency streams
(``sa_cross_scores_pooled`` + ``sa_build_block_mask_pooled``).
"""
from __future__ import annotations

import torch

from . import binding as sa


class LayerPlan:
    def __init__(self, B, H, L_v, L_a, d, block, k_keep, k_prot, scale,
                 dtype=torch.bfloat16, device="cuda", with_audio=True,
                 want_lse=False):
        self.B, self.H, self.L_v, self.L_a, self.d = B, H, L_v, L_a, d
        self.block, self.k_keep, self.k_prot = block, k_keep, k_prot
        self.scale, self.with_audio = float(scale), with_audio
        n_b = -(-L_v // block)
        self.n_b = n_b
        f32, i32, u8 = torch.float32, torch.int32, torch.uint8
        e = lambda *s, dt=f32: torch.empty(*s, dtype=dt, device=device)
        self.sal_v_tok = e(B, L_v)
        self.sal_v_blk = e(B, n_b)
        self.sal_a_tok = e(B, L_a) if with_audio else None
        self.prot_idx = e(B, max(k_prot, 1), dt=i32)
        self.prot_flag = e(B, n_b, dt=u8)
        self.kv_idx = e(B, H, n_b, n_b, dt=i32)
        self.kv_cnt = e(B, H, n_b, dt=i32)
        self.o = e(B, H, L_v, d, dt=dtype)
        self.lse = e(B, H, L_v) if want_lse else None
        ws = max(sa.sa_workspace_size(c, B, H, L_v, L_a, d, block)
                 for c in (sa.SA_CALL_CROSS_SCORES, sa.SA_CALL_BUILD_BLOCK_MASK,
                           sa.SA_CALL_SPARSE_ATTENTION))
        self.ws = e(max(ws, 1), dt=u8)
        n_pad = sa.sa_pool_columns(n_b)
        self.qbar = e(B, H, d, n_pad, dt=torch.float64) if with_audio else None
        self.kbar = e(B, H, d, n_pad, dt=torch.float64) if with_audio else None

    def cross_scores(self, q_a, k_v, q_v, k_a):
        sa.sa_cross_scores(q_a, k_v, q_v if self.with_audio else None,
                           k_a if self.with_audio else None, self.scale,
                           self.block, sal_v_tok=self.sal_v_tok,
                           sal_v_blk=self.sal_v_blk, sal_a_tok=self.sal_a_tok,
                           ws=self.ws)

    def cross_scores_pooled(self, q_a, k_v, q_v, k_a, lse_a=None, lse_v=None):
        """The saliency (standalone, or from the forwards' row LSEs) and the
        block means of Q^v and K^v into qbar, kbar."""
        sa.sa_cross_scores_pooled(q_a, k_v, q_v, k_a, self.scale, self.block,
                                  lse_a=lse_a, lse_v=lse_v, sal_v_tok=self.sal_v_tok,
                                  sal_v_blk=self.sal_v_blk, sal_a_tok=self.sal_a_tok,
                                  qbar=self.qbar, kbar=self.kbar, ws=self.ws)

    def select_protected(self):
        sa.sa_select_protected(self.sal_v_blk, self.k_prot,
                               prot_idx=self.prot_idx if self.k_prot > 0 else None,
                               prot_flag=self.prot_flag, want_idx=False)

    def build_block_mask(self, q_v, k_v):
        sa.sa_build_block_mask(q_v, k_v, self.scale, self.block, self.k_keep,
                               self.prot_flag, kv_idx=self.kv_idx,
                               kv_cnt=self.kv_cnt, ws=self.ws)

    def build_block_mask_pooled(self):
        sa.sa_build_block_mask_pooled(self.qbar, self.kbar, self.L_v, self.scale, self.block,
                                      self.k_keep, self.prot_flag, kv_idx=self.kv_idx,
                                      kv_cnt=self.kv_cnt)

    def sparse_attention(self, q_v, k_v, v_v):
        sa.sa_sparse_attention(q_v, k_v, v_v, self.scale, self.block,
                               self.kv_idx, self.kv_cnt, o=self.o, lse=self.lse,
                               ws=self.ws)

    def run(self, q_v, k_v, v_v, q_a, k_a):
        self.cross_scores(q_a, k_v, q_v, k_a)
        self.select_protected()
        self.build_block_mask(q_v, k_v)
        self.sparse_attention(q_v, k_v, v_v)
        return self.o

    def run_pooled(self, q_v, k_v, v_v, q_a, k_a):
        self.cross_scores_pooled(q_a, k_v, q_v, k_a)
        self.select_protected()
        self.build_block_mask_pooled()
        self.sparse_attention(q_v, k_v, v_v)
        return self.o


def protected_sparse_layer(q_v, k_v, v_v, q_a, k_a, scale, block, k_keep,
                           k_prot, with_audio=True, want_lse=False):
    """One-shot layer: returns the LayerPlan holding every output."""
    B, H, L_v, d = q_v.shape
    plan = LayerPlan(B, H, L_v, q_a.shape[2], d, block, k_keep, k_prot, scale,
                     dtype=q_v.dtype, device=q_v.device, with_audio=with_audio,
                     want_lse=want_lse)
    plan.run(q_v, k_v, v_v, q_a, k_a)
    return plan
