"""Helpers of the GPU parity tests: device upload, the tie-aware set check of
the comparison rule, and a full-layer run through the C ABI compared against
the oracle."""
from __future__ import annotations

import os

import numpy as np
import torch

import oracle
import synth
import paper_2608_15522_amd as sa

TIE = 1e-6          # scores within this of the k-th value may go either way
TOL_O = {"f32": 1e-5, "bf16": 1.5e-2}
TOL_LSE = {"f32": 1e-5, "bf16": 2.5e-3}   # bf16: the row sum adds the bf16-rounded
                                             # probabilities (<= 2^-9 relative each)
TOL_SAL = 1e-6      # absolute, on L1-normalised saliency (the survey's diagnostic bound)
# Saliency is also bounded relative to each value: a token's saliency is about
# 1/L (3e-5 at L = 32760), so the absolute bound alone would allow a few
# percent.  fp32 exponentials and sums give ~1e-6 relative.
SAL_REL, SAL_ABS = 1e-4, 1e-9


def workers():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def to_dev(x, dtype):
    t = torch.from_numpy(np.ascontiguousarray(x))
    t = t.to(torch.bfloat16 if dtype == "bf16" else torch.float32)
    return t.to("cuda")


def logit_ramp_inputs(Lq, Lk, d, H, profile, dtype, seed=7):
    """Q [1,H,Lq,d] and K, V [1,H,Lk,d] whose logits follow a profile along
    the keys: q_i = 0.5 z + 2 sqrt(d) u, k_j = 0.5 z' + b_j sqrt(d) u with u a
    unit vector, so that scale * q_i . k_j is about 2 sqrt(d) b_j.  "grow":
    b_j rises from 0 to 3 (logits up to ~70, ~100 log2 units), "fall": the
    reverse, "jump": b_j = 4.5 on the last 50 keys and 0 before (a jump of
    ~150 log2 units, past fp32's exp2 range)."""
    rng = np.random.default_rng(seed)
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    j = np.arange(Lk) / Lk
    b = {"grow": 3.0 * j, "fall": 3.0 * (1.0 - j),
         "jump": np.where(np.arange(Lk) >= Lk - 50, 4.5, 0.0)}[profile]
    q = 0.5 * rng.standard_normal((1, H, Lq, d)) + 2.0 * np.sqrt(d) * u
    k = 0.5 * rng.standard_normal((1, H, Lk, d)) + (b * np.sqrt(d))[None, None, :, None] * u
    v = rng.standard_normal((1, H, Lk, d))
    out = [a.astype(np.float32) for a in (q, k, v)]
    if dtype == "bf16":
        out = [synth.round_to_bf16(a).reshape(a.shape) for a in out]
    return out


def check_topk_set(chosen, scores, k, tie=TIE):
    """The comparison rule for a top-k selection: exactly k distinct members,
    every index scoring above v_k + tie is in, none scoring below v_k - tie
    is.  Returns the number of members decided inside the tie window."""
    chosen = np.asarray(chosen, dtype=np.int64)
    assert chosen.size == k, (chosen.size, k)
    assert np.unique(chosen).size == k
    if k == 0:
        return 0
    order = oracle.topk_order(scores, k)
    vk = scores[order[-1]]
    must = np.nonzero(scores > vk + tie)[0]
    never = np.nonzero(scores < vk - tie)[0]
    cs = set(chosen.tolist())
    assert set(must.tolist()) <= cs, "a clear top-k member is missing"
    assert not (set(never.tolist()) & cs), "a clear non-member was chosen"
    # candidates other than the k-th itself inside the tie window
    return int(np.sum(np.abs(scores - vk) <= tie)) - 1


def check_saliency(got, ref, name="saliency"):
    """|got - ref| <= SAL_REL |ref| + SAL_ABS elementwise, and <= TOL_SAL.
    Returns the largest relative error."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    err = np.abs(got - ref)
    bad = err > SAL_REL * np.abs(ref) + SAL_ABS
    assert not bad.any(), (name, int(bad.sum()), float(err[bad].max()),
                           float(np.abs(ref[bad]).min()))
    assert float(err.max()) <= TOL_SAL, (name, float(err.max()))
    return float((err / np.maximum(np.abs(ref), 1e-30)).max())


def check_token_selection(tok_idx, sal_ref, k):
    """Protected tokens against the oracle's fp64 saliency: per batch item an
    ascending list of k tokens forming a top-k, where tokens whose reference
    saliency lies within the relative saliency bound (twice, for both sides)
    of the k-th value may go either way.  Returns the number of such
    tokens."""
    tok_idx = np.asarray(tok_idx)
    ties = 0
    for b in range(sal_ref.shape[0]):
        lst = tok_idx[b]
        assert np.all(np.diff(lst) > 0)
        if k == 0:
            continue
        vk = float(sal_ref[b][oracle.topk_order(sal_ref[b], k)[-1]])
        ties += check_topk_set(lst, sal_ref[b], k, tie=2 * (SAL_REL * abs(vk) + SAL_ABS))
    return ties


def check_rank_order(prot_idx, scores, tie=TIE):
    """Rank order of a top-k list: scores descending; among scores equal
    within the tie window any order is accepted."""
    s = scores[np.asarray(prot_idx)]
    assert np.all(s[:-1] >= s[1:] - tie)


def check_protected(prot_idx, prot_flag, sal_blk_ref, k_prot):
    B, n_b = sal_blk_ref.shape
    ties = 0
    for b in range(B):
        ties += check_topk_set(prot_idx[b], sal_blk_ref[b], k_prot)
        check_rank_order(prot_idx[b], sal_blk_ref[b])
        flag = np.zeros(n_b, dtype=np.uint8)
        flag[prot_idx[b]] = 1
        assert np.array_equal(prot_flag[b], flag)
    return ties


def check_kv_lists(kv_idx, kv_cnt, prot_flag, G_ref, k_keep, mask=None):
    """Every row: protected rows hold 0..n_b-1; other rows hold k_keep
    ascending block indices forming a valid top-k of the oracle's G row;
    unused entries are -1; the optional u8 mask agrees with the lists."""
    B, H, n_b, _ = kv_idx.shape
    ties = 0
    full = np.arange(n_b)
    for b in range(B):
        for h in range(H):
            for r in range(n_b):
                cnt = int(kv_cnt[b, h, r])
                lst = kv_idx[b, h, r, :cnt]
                if prot_flag[b, r]:
                    assert cnt == n_b and np.array_equal(lst, full)
                else:
                    assert cnt == k_keep, (b, h, r, cnt)
                    assert np.all(np.diff(lst) > 0)
                    ties += check_topk_set(lst, G_ref[b, h, r], k_keep)
                assert np.all(kv_idx[b, h, r, cnt:] == -1)
                if mask is not None:
                    m = np.zeros(n_b, dtype=np.uint8)
                    m[lst] = 1
                    assert np.array_equal(mask[b, h, r], m)
    return ties


def full_masked_attention(q, k, v, scale, block, kv_idx, kv_cnt):
    """oracle.masked_attention over every query block, its (b, h) slabs run
    concurrently in threads (the oracle is called unchanged, once per slab)."""
    from concurrent.futures import ThreadPoolExecutor
    B, H, N, d = q.shape
    n_b = -(-N // block)
    O = np.zeros((B, H, N, v.shape[3]), dtype=np.float64)
    lse = np.full((B, H, N), -np.inf, dtype=np.float64)

    def run(bh):
        b, h = bh
        rows = [(b, h, r) for r in range(n_b)]
        o_d, l_d = oracle.masked_attention(q, k, v, scale, block, kv_idx, kv_cnt, rows=rows)
        for (_, _, r) in rows:
            lo, hi = r * block, min((r + 1) * block, N)
            O[b, h, lo:hi] = o_d[(b, h, r)]
            lse[b, h, lo:hi] = l_d[(b, h, r)]

    from threadpoolctl import threadpool_limits
    with threadpool_limits(1), ThreadPoolExecutor(max_workers=workers()) as ex:
        list(ex.map(run, [(b, h) for b in range(B) for h in range(H)]))
    return O, lse


def sample_rows(g, w, n_random=16, seed=0):
    """Query blocks whose attention is compared at full size: every protected
    block of head 0, the first block and the ragged last block of each batch
    item, and random ones."""
    rng = np.random.default_rng(seed)
    rows = {(0, 0, int(r)) for r in np.nonzero(g["prot_flag"][0])[0]}
    for b in range(w.B):
        rows.add((b, w.H - 1, w.n_b - 1))
        rows.add((b, 0, 0))
    for _ in range(n_random):
        rows.add((int(rng.integers(w.B)), int(rng.integers(w.H)),
                  int(rng.integers(w.n_b))))
    return sorted(rows)


def gpu_layer(x, w, k_keep, k_prot, with_audio=True):
    """All four C-ABI calls on the workload's inputs, with every optional
    output requested.  Returns numpy copies."""
    t = {k: to_dev(x[k], w.dtype) for k in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    sal_v_tok, sal_v_blk, sal_a_tok = sa.sa_cross_scores(
        t["q_a"], t["k_v"], t["q_v"] if with_audio else None,
        t["k_a"] if with_audio else None, w.scale, w.block)
    prot_idx, prot_flag = sa.sa_select_protected(sal_v_blk, k_prot)
    kv_idx, kv_cnt, mask, scores = sa.sa_build_block_mask(
        t["q_v"], t["k_v"], w.scale, w.block, k_keep, prot_flag,
        want_mask=True, want_scores=True)
    o, lse = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale,
                                    w.block, kv_idx, kv_cnt, want_lse=True)
    torch.cuda.synchronize()
    out = dict(sal_v_tok=sal_v_tok, sal_v_blk=sal_v_blk, sal_a_tok=sal_a_tok,
               prot_idx=prot_idx, prot_flag=prot_flag, kv_idx=kv_idx,
               kv_cnt=kv_cnt, mask=mask, scores=scores, o=o, lse=lse)
    res = {k: (v.float().cpu().numpy() if v is not None and v.dtype == torch.bfloat16
               else (v.cpu().numpy() if v is not None else None))
           for k, v in out.items()}
    del t, out
    torch.cuda.empty_cache()
    return res


def compare_layer(x, w, g, k_keep, k_prot, rows=None, with_audio=True,
                  report=None):
    """Compare a gpu_layer() result with the oracle.  ``rows`` (list of
    (b, h, r)) restricts the attention comparison to those query blocks."""
    rep = {} if report is None else report
    s_v, s_a = oracle.cross_scores(x["q_a"], x["k_v"], w.scale,
                                   x["q_v"] if with_audio else None,
                                   x["k_a"] if with_audio else None,
                                   workers=workers())
    s_blk = oracle.token_to_block_saliency(s_v, w.block)
    rep["sal_v_tok_err"] = float(np.abs(g["sal_v_tok"] - s_v).max())
    rep["sal_v_blk_err"] = float(np.abs(g["sal_v_blk"] - s_blk).max())
    rep["sal_v_tok_rel"] = check_saliency(g["sal_v_tok"], s_v, "sal_v_tok")
    rep["sal_v_blk_rel"] = check_saliency(g["sal_v_blk"], s_blk, "sal_v_blk")
    if with_audio:
        rep["sal_a_tok_err"] = float(np.abs(g["sal_a_tok"] - s_a).max())
        rep["sal_a_tok_rel"] = check_saliency(g["sal_a_tok"], s_a, "sal_a_tok")
    rep["prot_ties"] = check_protected(g["prot_idx"], g["prot_flag"], s_blk, k_prot)
    G = oracle.pooled_scores(x["q_v"], x["k_v"], w.scale, w.block)
    # the scores output is the fp64 score rounded once to fp32
    rep["G_err"] = float(np.abs(g["scores"] - G).max())
    assert np.all(np.abs(g["scores"] - G) <= 2.0 ** -24 * np.abs(G) + 1e-12), rep
    rep["mask_ties"] = check_kv_lists(g["kv_idx"], g["kv_cnt"], g["prot_flag"],
                                      G, k_keep, g["mask"])
    if rows is None:
        O_ref, lse_ref = full_masked_attention(x["q_v"], x["k_v"], x["v_v"], w.scale,
                                               w.block, g["kv_idx"], g["kv_cnt"])
    else:
        O_ref, lse_ref = oracle.masked_attention(x["q_v"], x["k_v"], x["v_v"],
                                                 w.scale, w.block, g["kv_idx"],
                                                 g["kv_cnt"], rows=rows)
    if rows is None:
        o_err = np.abs(g["o"] - O_ref).max()
        l_err = np.abs(g["lse"] - lse_ref).max()
    else:
        o_err = l_err = 0.0
        for (b, h, r) in rows:
            lo = r * w.block
            hi = min(lo + w.block, w.L_v)
            o_err = max(o_err, np.abs(g["o"][b, h, lo:hi] - O_ref[(b, h, r)]).max())
            l_err = max(l_err, np.abs(g["lse"][b, h, lo:hi] - lse_ref[(b, h, r)]).max())
    rep["o_err"], rep["lse_err"] = float(o_err), float(l_err)
    assert rep["o_err"] <= TOL_O[w.dtype], rep
    assert rep["lse_err"] <= TOL_LSE[w.dtype], rep
    assert np.all(np.isfinite(g["o"]))
    return rep
