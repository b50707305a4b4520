"""GPU parity of the block means pooled inside the saliency streams
(sa_cross_scores_pooled) and of the mask built from them
(sa_build_block_mask_pooled), through the C ABI.

The means of Eq. (6) are exact fp64 sums of the bf16 (or fp32) inputs divided
once, so they must equal the oracle's block means to the last bit but one
rounding, and the mask built from them must equal, bit for bit, the mask that
sa_build_block_mask pools itself (lists, flags and G).  The saliency of the
pooled call is that of the plain calls, bit for bit, and both are checked
against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import check_kv_lists, check_saliency, to_dev, workers

pytestmark = pytest.mark.gpu

BASE = synth.WORKLOADS["ovi_bf16"]
CASES = [
    # ragged tail (L_v = 520), one K2 chunk, one slab of audio queries
    ("small", BASE.with_(name="p1", H=2, frames=4, rows=10, cols=13, L_a=200, n_plant=2)),
    # d = 64, block = 64, two audio slabs (pooling runs in the first only)
    ("d64_b64", BASE.with_(name="p2", H=3, d=64, block=64, frames=3, rows=10, cols=11,
                           L_a=1000, n_plant=1)),
    # block 64 at d = 128 over three K2 chunks and five v->a chunks, B = 2
    ("d128_b64", BASE.with_(name="p3", B=2, H=2, block=64, frames=4, rows=10, cols=55,
                            L_a=700, n_plant=2)),
    # three audio slabs, L_v a multiple of 1024 (no tail)
    ("slabs3", BASE.with_(name="p4", H=2, frames=4, rows=16, cols=32, L_a=1100, n_plant=2)),
    # shorter than one 64-key tile: one block, one partial unit, 7 audio tokens
    ("tiny", BASE.with_(name="p5", H=1, d=64, block=64, frames=1, rows=5, cols=10, L_a=7,
                        n_plant=0)),
    ("ovi", BASE),
    ("ltx", synth.WORKLOADS["ltx_bf16"]),
]


def _np(t):
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy()


def _means(m, n_b):
    """[B,H,d,n_pad] device means -> [B,H,n_b,d] numpy."""
    return m[..., :n_b].transpose(2, 3).cpu().numpy()


def _check_means(got, ref, name):
    # exact sums, one rounding of the division: at most 1 ulp from the oracle
    err = np.abs(got - ref)
    bad = err > np.spacing(np.abs(ref))
    assert not bad.any(), (name, float(err.max()), int(bad.sum()))


@pytest.mark.parametrize("name,w", CASES, ids=[c[0] for c in CASES])
def test_pooled_saliency_and_mask(name, w):
    k_keep, k_prot = w.k_keep, w.k_prot
    print(f"case pooled {name}: B={w.B} H={w.H} L_v={w.L_v} L_a={w.L_a} d={w.d} "
          f"block={w.block} n_b={w.n_b} n_pad={sa.sa_pool_columns(w.n_b)}", flush=True)
    x = synth.make_inputs(w)
    v_a = synth.make_audio_values(w)
    t = {kk: to_dev(x[kk], w.dtype) for kk in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    args = (t["q_a"], t["k_v"], t["q_v"], t["k_a"], w.scale, w.block)
    # standalone saliency, plain and pooled
    r_v, r_blk, r_a = sa.sa_cross_scores(*args)
    p_v, p_blk, p_a, qbar, kbar = sa.sa_cross_scores_pooled(*args)
    # from the forwards' row LSEs, plain and pooled
    _, lse_a = sa.sa_cross_attention(t["q_a"], t["k_v"], t["v_v"], w.scale, want_lse=True)
    _, lse_v = sa.sa_cross_attention(t["q_v"], t["k_a"], to_dev(v_a, w.dtype), w.scale,
                                     want_lse=True)
    f_v, f_blk, f_a = sa.sa_cross_scores_from_lse(t["q_a"], t["k_v"], t["q_v"], t["k_a"],
                                                  lse_a, lse_v, w.scale, w.block)
    g_v, g_blk, g_a, qbar2, kbar2 = sa.sa_cross_scores_pooled(*args, lse_a=lse_a, lse_v=lse_v)
    prot_idx, prot_flag = sa.sa_select_protected(p_blk, k_prot)
    # the mask from the pooled means and the mask that pools Q^v, K^v itself
    m_idx, m_cnt, m_mask, m_G = sa.sa_build_block_mask_pooled(
        qbar, kbar, w.L_v, w.scale, w.block, k_keep, prot_flag, want_mask=True,
        want_scores=True)
    s_idx, s_cnt, s_mask, s_G = sa.sa_build_block_mask(
        t["q_v"], t["k_v"], w.scale, w.block, k_keep, prot_flag, want_mask=True,
        want_scores=True)
    torch.cuda.synchronize()
    print(f"{name}: gpu done", flush=True)
    # the saliency is the plain calls', bit for bit
    for a, b, nm in ((p_v, r_v, "sal_v_tok"), (p_blk, r_blk, "sal_v_blk"),
                     (p_a, r_a, "sal_a_tok"), (g_v, f_v, "lse sal_v_tok"),
                     (g_blk, f_blk, "lse sal_v_blk"), (g_a, f_a, "lse sal_a_tok")):
        assert torch.equal(a, b), nm
    # both forms pool the same means
    assert torch.equal(qbar[..., :w.n_b], qbar2[..., :w.n_b])
    assert torch.equal(kbar[..., :w.n_b], kbar2[..., :w.n_b])
    # the means against the oracle's block means (Eq. (6))
    _check_means(_means(qbar, w.n_b), oracle.block_pool(x["q_v"], w.block), "qbar")
    _check_means(_means(kbar, w.n_b), oracle.block_pool(x["k_v"], w.block), "kbar")
    # the mask is the standalone mask's, bit for bit
    for a, b, nm in ((m_idx, s_idx, "kv_idx"), (m_cnt, s_cnt, "kv_cnt"),
                     (m_mask, s_mask, "mask"), (m_G, s_G, "G")):
        assert torch.equal(a, b), nm
    # and a valid top-k of the oracle's G, with the protected rows full
    G = oracle.pooled_scores(x["q_v"], x["k_v"], w.scale, w.block)
    g_np = m_G.cpu().numpy()
    assert np.all(np.abs(g_np - G) <= 2.0 ** -24 * np.abs(G) + 1e-12)
    ties = check_kv_lists(m_idx.cpu().numpy(), m_cnt.cpu().numpy(), prot_flag.cpu().numpy(),
                          G, k_keep, m_mask.cpu().numpy())
    # the saliency against the oracle (both directions)
    s_v_ref, s_a_ref = oracle.cross_scores(x["q_a"], x["k_v"], w.scale, x["q_v"], x["k_a"],
                                           workers=workers())
    check_saliency(_np(p_v), s_v_ref, "sal_v_tok")
    check_saliency(_np(p_a), s_a_ref, "sal_a_tok")
    check_saliency(_np(p_blk), oracle.token_to_block_saliency(s_v_ref, w.block), "sal_v_blk")
    print(name, dict(mask_ties=ties), flush=True)


def test_pooled_fp32_path():
    """fp32 inputs (the tiny workload): the standalone form pools in a pass of
    its own; means against the oracle, mask equal to the standalone mask."""
    w = synth.WORKLOADS["tiny_f32"]
    print(f"case pooled fp32: L_v={w.L_v} L_a={w.L_a}", flush=True)
    x = synth.make_inputs(w)
    t = {kk: to_dev(x[kk], w.dtype) for kk in ("q_v", "k_v", "q_a", "k_a")}
    args = (t["q_a"], t["k_v"], t["q_v"], t["k_a"], w.scale, w.block)
    r_v, r_blk, r_a = sa.sa_cross_scores(*args)
    p_v, p_blk, p_a, qbar, kbar = sa.sa_cross_scores_pooled(*args)
    _, prot_flag = sa.sa_select_protected(p_blk, w.k_prot)
    m = sa.sa_build_block_mask_pooled(qbar, kbar, w.L_v, w.scale, w.block, w.k_keep,
                                      prot_flag, want_mask=True, want_scores=True)
    s = sa.sa_build_block_mask(t["q_v"], t["k_v"], w.scale, w.block, w.k_keep, prot_flag,
                               want_mask=True, want_scores=True)
    torch.cuda.synchronize()
    assert torch.equal(p_v, r_v) and torch.equal(p_blk, r_blk) and torch.equal(p_a, r_a)
    _check_means(_means(qbar, w.n_b), oracle.block_pool(x["q_v"], w.block), "qbar")
    _check_means(_means(kbar, w.n_b), oracle.block_pool(x["k_v"], w.block), "kbar")
    for a, b in zip(m, s):
        assert torch.equal(a, b)


def test_pooled_accumulate():
    """accumulate = 1 adds the layer's saliency to what the outputs hold; the
    means are written as usual."""
    w = CASES[0][1]
    print("case pooled accumulate", flush=True)
    x = synth.make_inputs(w)
    t = {kk: to_dev(x[kk], w.dtype) for kk in ("q_v", "k_v", "q_a", "k_a")}
    args = (t["q_a"], t["k_v"], t["q_v"], t["k_a"], w.scale, w.block)
    p_v, p_blk, p_a, qbar, kbar = sa.sa_cross_scores_pooled(*args)
    base = [torch.full_like(a, 0.25) for a in (p_v, p_blk, p_a)]
    acc = [b.clone() for b in base]
    _, _, _, qbar2, kbar2 = sa.sa_cross_scores_pooled(*args, sal_v_tok=acc[0], sal_v_blk=acc[1],
                                                      sal_a_tok=acc[2], accumulate=True)
    torch.cuda.synchronize()
    for a, b, p in zip(acc, base, (p_v, p_blk, p_a)):
        assert torch.equal(a, b + p)
    assert torch.equal(qbar[..., :w.n_b], qbar2[..., :w.n_b])
    assert torch.equal(kbar[..., :w.n_b], kbar2[..., :w.n_b])
