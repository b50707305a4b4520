"""GPU parity over the density sweep at the full Ovi-like size: every cell
of density {10, 25, 50, 100} % x protection {0, 5, 10} % for seeds 0-2.

Per seed the saliency (both directions) and the pooled scores G are
compared once, since neither depends on the budgets.  Per cell: the
protected blocks against the oracle's block saliency, every list of every
row against the oracle's G (tie rule), and the attention on sampled query
blocks against the oracle run on the GPU's lists (every protected block of
head 0, the first and the ragged last block, random blocks)."""
import functools

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import (TOL_LSE, TOL_O, check_kv_lists, check_protected, check_saliency,
                       sample_rows, to_dev, workers)

pytestmark = pytest.mark.gpu

CELLS = [w for w in synth.sweep_workloads()]
CELLS.sort(key=lambda w: (w.seed, w.density, w.rho))


@functools.lru_cache(maxsize=1)
def seed_context(seed):
    """Inputs of one seed on the device, the GPU saliency, and the oracle's
    saliency and G (checked here once)."""
    w = synth.WORKLOADS["ovi_bf16"].with_(seed=seed)
    print(f"seed {seed}: inputs", flush=True)
    x = synth.make_inputs(w)
    t = {k: to_dev(x[k], w.dtype) for k in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    sal_v_tok, sal_v_blk, sal_a_tok = sa.sa_cross_scores(t["q_a"], t["k_v"], t["q_v"],
                                                         t["k_a"], w.scale, w.block)
    _, _, _, scores = sa.sa_build_block_mask(t["q_v"], t["k_v"], w.scale, w.block, 1,
                                             None, want_scores=True)
    torch.cuda.synchronize()
    s_v, s_a = oracle.cross_scores(x["q_a"], x["k_v"], w.scale, x["q_v"], x["k_a"],
                                   workers=workers())
    s_blk = oracle.token_to_block_saliency(s_v, w.block)
    check_saliency(sal_v_tok.cpu().numpy(), s_v, "sal_v_tok")
    check_saliency(sal_v_blk.cpu().numpy(), s_blk, "sal_v_blk")
    check_saliency(sal_a_tok.cpu().numpy(), s_a, "sal_a_tok")
    G = oracle.pooled_scores(x["q_v"], x["k_v"], w.scale, w.block)
    sc = scores.cpu().numpy()
    assert np.all(np.abs(sc - G) <= 2.0 ** -24 * np.abs(G) + 1e-12)
    print(f"seed {seed}: saliency and G checked", flush=True)
    return dict(x=x, t=t, sal_v_blk=sal_v_blk, s_blk=s_blk, G=G)


@pytest.mark.parametrize("w", CELLS, ids=[w.name for w in CELLS])
def test_sweep_cell_parity(w):
    print(f"case {w.name}: k_keep={w.k_keep} k_prot={w.k_prot}", flush=True)
    ctx = seed_context(w.seed)
    t, x = ctx["t"], ctx["x"]
    prot_idx, prot_flag = sa.sa_select_protected(ctx["sal_v_blk"], w.k_prot)
    kv_idx, kv_cnt, mask, _ = sa.sa_build_block_mask(t["q_v"], t["k_v"], w.scale, w.block,
                                                     w.k_keep, prot_flag, want_mask=True)
    o, lse = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, w.block, kv_idx,
                                    kv_cnt, want_lse=True)
    torch.cuda.synchronize()
    g = dict(prot_idx=prot_idx.cpu().numpy(), prot_flag=prot_flag.cpu().numpy(),
             kv_idx=kv_idx.cpu().numpy(), kv_cnt=kv_cnt.cpu().numpy(),
             mask=mask.cpu().numpy())
    ties = check_protected(g["prot_idx"], g["prot_flag"], ctx["s_blk"], w.k_prot)
    ties += check_kv_lists(g["kv_idx"], g["kv_cnt"], g["prot_flag"], ctx["G"], w.k_keep,
                           g["mask"])
    rows = sample_rows(g, w, n_random=12 if w.seed == 0 else 4, seed=w.seed)
    O_ref, lse_ref = oracle.masked_attention(x["q_v"], x["k_v"], x["v_v"], w.scale, w.block,
                                             g["kv_idx"], g["kv_cnt"], rows=rows)
    o_err = l_err = 0.0
    for (b, h, r) in rows:
        lo, hi = r * w.block, min((r + 1) * w.block, w.L_v)
        o_blk = o[b, h, lo:hi].float().cpu().numpy()
        l_blk = lse[b, h, lo:hi].cpu().numpy()
        o_err = max(o_err, float(np.abs(o_blk - O_ref[(b, h, r)]).max()))
        l_err = max(l_err, float(np.abs(l_blk - lse_ref[(b, h, r)]).max()))
    assert bool(torch.isfinite(o).all())
    print(w.name, dict(ties=ties, rows=len(rows), o_err=o_err, lse_err=l_err), flush=True)
    assert o_err <= TOL_O["bf16"] and l_err <= TOL_LSE["bf16"]
