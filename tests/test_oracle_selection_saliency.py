"""Pins of the oracle's saliency (Eq. (1)-(2) and the reverse direction),
protected selection (Eq. (3)/(8)) and block mask (Eq. (6), (9)).  CPU only."""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- selection
def _brute_force_topk(s, k):
    """Among all k-subsets with the largest sum, the lexicographically
    smallest sorted index tuple."""
    best, best_sum = None, -math.inf
    for sub in itertools.combinations(range(len(s)), k):
        tot = sum(s[i] for i in sub)
        if tot > best_sum + 1e-12:
            best, best_sum = sub, tot
        elif abs(tot - best_sum) <= 1e-12 and sub < best:
            best = sub
    return best


def test_topk_brute_force_with_ties():
    rng = np.random.default_rng(0)
    for trial in range(60):
        n = int(rng.integers(1, 8))
        s = rng.integers(-3, 4, size=n).astype(float)   # many exact ties
        for k in range(n + 1):
            got = oracle.topk_order(s, k)
            assert tuple(sorted(got.tolist())) == _brute_force_topk(s.tolist(), k)
            # rank order: score descending, index ascending
            ref = sorted(range(n), key=lambda c: (-s[c], c))[:k]
            assert got.tolist() == ref


def test_topk_rejects_bad_k():
    with pytest.raises(ValueError):
        oracle.topk_order(np.zeros(3), 4)
    with pytest.raises(ValueError):
        oracle.topk_order(np.zeros(3), -1)


def test_select_protected_flags_and_rank_order():
    sal = np.array([[0.1, 0.4, 0.4, 0.05, 0.05],
                    [0.2, 0.2, 0.2, 0.2, 0.2]])
    idx, flag = oracle.select_protected(sal, 3)
    assert idx.tolist() == [[1, 2, 0], [0, 1, 2]]
    assert flag.tolist() == [[1, 1, 1, 0, 0], [1, 1, 1, 0, 0]]
    idx0, flag0 = oracle.select_protected(sal, 0)
    assert idx0.shape == (2, 0) and flag0.sum() == 0


# ---------------------------------------------------------------- saliency
def test_golden_saliency_closed_form():
    g = json.load(open(os.path.join(GOLDEN, "closed_form_saliency.json")))
    w = np.array(g["video_key_weights"])
    N_v = w.size
    q_a = np.ones((1, 1, 1, 1))
    k_v = np.log(w).reshape(1, 1, N_v, 1)
    s_v, _ = oracle.cross_scores(q_a, k_v, g["scale"])
    np.testing.assert_allclose(s_v[0], g["s_v"], rtol=1e-14)
    s_blk = oracle.token_to_block_saliency(s_v, g["block"])
    np.testing.assert_allclose(s_blk[0], g["s_blk"], rtol=1e-14)
    idx, _ = oracle.select_protected(s_blk, 1)
    assert idx[0].tolist() == g["protected_top1"]
    idx, _ = oracle.select_protected(s_blk, 2)
    assert idx[0].tolist() == g["protected_top2"]


def test_saliency_two_queries_two_heads_closed_form():
    """Head 0: audio queries +1 and -1 against keys ln w_i give rows w/sum(w)
    and (1/w)/sum(1/w).  Head 1: zero queries give uniform rows.  Norm
    divides by H * N_a = 4."""
    w = np.array([1.0, 2.0, 5.0, 0.5, 3.0, 3.0])
    N_v = w.size
    q_a = np.zeros((1, 2, 2, 1))
    q_a[0, 0, :, 0] = [1.0, -1.0]
    k_v = np.zeros((1, 2, N_v, 1))
    k_v[0, 0, :, 0] = np.log(w) / 0.5               # scale 0.5 undoes it
    k_v[0, 1, :, 0] = np.log(w) * 7.0
    s_v, _ = oracle.cross_scores(q_a, k_v, 0.5)
    expect = (w / w.sum() + (1 / w) / (1 / w).sum() + 2.0 / N_v) / 4
    np.testing.assert_allclose(s_v[0], expect, rtol=1e-13)


def test_reverse_direction_closed_form():
    """v->a: video queries against audio keys ln w_j; s^a sums over video
    queries and divides by H * N_v."""
    w = np.array([4.0, 1.0, 3.0])
    q_v = np.zeros((1, 1, 3, 1))
    q_v[0, 0, :, 0] = [1.0, 0.0, 2.0]
    k_a = (np.log(w) / 0.25).reshape(1, 1, 3, 1)     # scale 0.25 undoes it
    q_a = np.zeros((1, 1, 3, 1))
    k_v = np.zeros((1, 1, 3, 1))
    _, s_a = oracle.cross_scores(q_a, k_v, 0.25, q_v=q_v, k_a=k_a)
    expect = (w / w.sum() + 1 / 3 + w ** 2 / (w ** 2).sum()) / 3
    np.testing.assert_allclose(s_a[0], expect, rtol=1e-13)


def test_saliency_invariants_and_equivariance():
    rng = np.random.default_rng(1)
    B, H, N_a, N_v, d = 2, 3, 7, 19, 4
    q_a, k_a = rng.standard_normal((2, B, H, N_a, d))
    q_v, k_v = rng.standard_normal((2, B, H, N_v, d))
    s_v, s_a = oracle.cross_scores(q_a, k_v, 0.5, q_v=q_v, k_a=k_a)
    np.testing.assert_allclose(s_v.sum(1), 1.0, atol=1e-14)
    np.testing.assert_allclose(s_a.sum(1), 1.0, atol=1e-14)
    assert np.all(s_v > 0) and np.all(s_a > 0)
    perm = rng.permutation(N_v)
    s_v2, s_a2 = oracle.cross_scores(q_a, k_v[:, :, perm], 0.5,
                                     q_v=q_v[:, :, perm], k_a=k_a)
    np.testing.assert_allclose(s_v2, s_v[:, perm], atol=1e-15)
    np.testing.assert_allclose(s_a2, s_a, atol=1e-15)
    # permuting audio queries leaves s^v unchanged
    perm_a = rng.permutation(N_a)
    s_v3, _ = oracle.cross_scores(q_a[:, :, perm_a], k_v, 0.5)
    np.testing.assert_allclose(s_v3, s_v, atol=1e-15)


def test_zero_audio_queries_give_exact_uniform_saliency_and_ties():
    """Q^a = 0: every row is uniform, s^v = 1/N_v, block sums are
    |block|/N_v; all blocks of equal length tie, so the lower indices win and
    the shorter tail block ranks last."""
    B, H, N_a, N_v, d, block = 1, 2, 3, 10, 2, 4
    q_a = np.zeros((B, H, N_a, d))
    k_v = np.random.default_rng(2).standard_normal((B, H, N_v, d))
    s_v, _ = oracle.cross_scores(q_a, k_v, 1.0)
    np.testing.assert_allclose(s_v, 1.0 / N_v, rtol=1e-15)
    s_blk = oracle.token_to_block_saliency(s_v, block)
    np.testing.assert_allclose(s_blk[0], [0.4, 0.4, 0.2], rtol=1e-14)
    idx, _ = oracle.select_protected(s_blk, 3)
    assert idx[0].tolist() == [0, 1, 2]


# ---------------------------------------------------------------- mask
def test_block_pool_tail_divides_by_true_length():
    N, d, block = 10, 3, 4                      # blocks of 4, 4, 2
    x = np.zeros((1, 1, N, d))
    x[0, 0, 0:4] = 1.5
    x[0, 0, 4:8] = -2.0
    x[0, 0, 8:10] = 7.0
    p = oracle.block_pool(x, block)
    np.testing.assert_array_equal(p[0, 0, :, 0], [1.5, -2.0, 7.0])
    y = np.arange(N, dtype=float).reshape(1, 1, N, 1)
    np.testing.assert_array_equal(oracle.block_pool(y, block)[0, 0, :, 0],
                                  [1.5, 5.5, 8.5])


def test_pooled_scores_closed_form():
    """Block-constant Q and K: pooled means are the constants, so
    G[r, c] = scale * a_r . b_c."""
    rng = np.random.default_rng(3)
    n_b, block, d = 3, 4, 5
    a, bv = rng.standard_normal((2, n_b, d))
    q = np.repeat(a, block, 0)[:10].reshape(1, 1, 10, d)
    k = np.repeat(bv, block, 0)[:10].reshape(1, 1, 10, d)
    G = oracle.pooled_scores(q, k, 0.3, block)
    np.testing.assert_allclose(G[0, 0], 0.3 * a @ bv.T, atol=1e-14)


def test_block_mask_brute_force_rows_and_protection():
    rng = np.random.default_rng(4)
    B, H, N, d, block, k_keep = 2, 2, 22, 3, 4, 2    # n_b = 6, tail 2
    q, k = rng.standard_normal((2, B, H, N, d))
    prot = np.zeros((B, 6), dtype=np.uint8)
    prot[0, [1, 4]] = 1
    prot[1, [0]] = 1
    m = oracle.block_mask(q, k, 0.5, block, k_keep, prot)
    G = m["G"]
    for b in range(B):
        for h in range(H):
            for r in range(6):
                kept = tuple(np.nonzero(m["mask"][b, h, r])[0].tolist())
                if prot[b, r]:
                    assert kept == tuple(range(6))
                else:
                    assert kept == _brute_force_topk(G[b, h, r].tolist(), k_keep)
                cnt = m["kv_cnt"][b, h, r]
                assert cnt == len(kept)
                assert tuple(m["kv_idx"][b, h, r, :cnt].tolist()) == kept
                assert np.all(m["kv_idx"][b, h, r, cnt:] == -1)
    # protection restores rows only: protected block 1 of batch 0 is not
    # forced into the key sets of other rows
    unprot = m["mask"][0][:, prot[0] == 0]
    assert unprot.sum() == H * 4 * k_keep


def test_constant_keys_tie_to_first_blocks():
    """Constant K^v makes every pooled key equal, so each row's scores tie
    exactly and the first k_keep blocks are kept."""
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 2, 24, 4))
    k = np.ones((1, 2, 24, 4)) * 0.75
    m = oracle.block_mask(q, k, 0.5, 4, 3, None)
    assert np.all(m["kv_idx"][..., :3] == np.arange(3))
    assert np.all(m["kv_cnt"] == 3)


def test_dense_keep_gives_all_ones():
    rng = np.random.default_rng(6)
    q, k = rng.standard_normal((2, 1, 1, 20, 2))
    m = oracle.block_mask(q, k, 1.0, 4, 5, None)
    assert m["mask"].all() and np.all(m["kv_cnt"] == 5)
    with pytest.raises(ValueError):
        oracle.block_mask(q, k, 1.0, 4, 6, None)
    with pytest.raises(ValueError):
        oracle.block_mask(q, k, 1.0, 4, 0, None)


# ---------------------------------------------------------------- layer
def test_flop_count_closed_forms():
    golden = json.load(open(os.path.join(GOLDEN, "budgets.json")))
    B, H, N, d, block = 1, 2, 36, 8, 4
    kv_idx = np.tile(np.arange(9), (B, H, 9, 1))
    kv_cnt = np.full((B, H, 9), 9)
    assert oracle.computed_flops(kv_idx, kv_cnt, N, block, d) == \
        oracle.dense_flops(B, H, N, d)
    # ragged: N = 10, block 4 -> lengths 4, 4, 2; row 2 keeps block 0 only
    kv_idx = np.array([[[[0, 1, 2], [2, -1, -1], [0, -1, -1]]]])
    kv_cnt = np.array([[[3, 1, 1]]])
    assert oracle.computed_flops(kv_idx, kv_cnt, 10, 4, 1) == \
        4 * (4 * 10 + 4 * 2 + 2 * 4)
    w = synth.WORKLOADS["tiny_f32"]
    g = golden["workloads"]["tiny_f32"]
    pairs = (w.n_b - w.k_prot) * w.k_keep + w.k_prot * w.n_b
    assert pairs == g["computed_pairs_blocks"]


def test_tiny_layer_protects_planted_blocks():
    """Statistical sanity of the synthetic workload, not parity: the
    protected blocks of the tiny workload lie inside its planted blocks."""
    w = synth.WORKLOADS["tiny_f32"]
    x = synth.make_inputs(w)
    out = oracle.protected_sparse_layer(x["q_v"], x["k_v"], x["v_v"],
                                        x["q_a"], x["k_a"], w.scale, w.block,
                                        w.k_keep, w.k_prot)
    planted_blocks = set(np.nonzero(x["planted"][0, ::w.block])[0].tolist())
    assert set(out["prot_idx"][0].tolist()) <= planted_blocks
    np.testing.assert_allclose(out["sal_v_tok"].sum(1), 1.0, atol=1e-13)
    np.testing.assert_allclose(out["sal_a_tok"].sum(1), 1.0, atol=1e-13)
    assert np.all(out["kv_cnt"][0][:, out["prot_idx"][0]] == w.n_b)
