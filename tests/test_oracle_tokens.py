"""Pins of the oracle's token-granular protection: the lagged saliency update
(Eq. (4)), token top-k (Eq. (8) at token level) and attention with protected
query tokens (Eq. (9)-(11)).  CPU only."""
import itertools
import math

import numpy as np
import pytest

import oracle


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _random_lists(B, H, n_b, seed):
    rng = np.random.default_rng(seed)
    mask = (rng.random((B, H, n_b, n_b)) < 0.4).astype(np.uint8)
    mask[mask.sum(-1) == 0, 0] = 1           # no empty row
    return oracle.kv_lists_from_mask(mask), mask


# ------------------------------------------------------------------ Eq. (4)
def test_ema_limits_and_exact_binary_values():
    prev = np.array([0.5, 0.25, 1.0, 0.0])
    cur = np.array([0.0, 0.75, 1.0, 0.125])
    np.testing.assert_array_equal(oracle.saliency_ema(prev, cur, 0.0), cur)
    np.testing.assert_array_equal(oracle.saliency_ema(prev, cur, 1.0), prev)
    # alpha = 1/4: every value below is exact in binary floating point
    np.testing.assert_array_equal(oracle.saliency_ema(prev, cur, 0.25),
                                  [0.125, 0.625, 1.0, 0.09375])


def test_ema_fixed_point_and_normalisation():
    """A constant map is a fixed point; L1-normalised maps stay normalised."""
    s = np.random.default_rng(0).random(50)
    s /= s.sum()
    sb = oracle.saliency_ema(s, s, 0.7)
    np.testing.assert_allclose(sb, s, rtol=0, atol=1e-16)
    t = np.random.default_rng(1).random(50)
    t /= t.sum()
    for _ in range(5):
        sb = oracle.saliency_ema(sb, t, 0.6)
        assert abs(sb.sum() - 1.0) < 1e-14
    # repeated updates with a fixed map converge to it geometrically
    np.testing.assert_allclose(sb - t, 0.6 ** 5 * (s - t), rtol=0, atol=1e-15)


# ------------------------------------------------------- Eq. (8), token level
def _brute_force_topk(s, k):
    best, best_sum = None, -math.inf
    for sub in itertools.combinations(range(len(s)), k):
        tot = sum(s[i] for i in sub)
        if tot > best_sum + 1e-12:
            best, best_sum = sub, tot
        elif abs(tot - best_sum) <= 1e-12 and sub < best:
            best = sub
    return best


def test_token_selection_brute_force_and_ties():
    rng = np.random.default_rng(2)
    for trial in range(20):
        n = int(rng.integers(3, 10))
        s = np.round(rng.random(n), 1)       # coarse values: many exact ties
        for k in range(0, n + 1):
            idx, flag = oracle.select_protected_tokens(s[None], k)
            assert tuple(idx[0]) == _brute_force_topk(list(s), k)
            assert flag[0].sum() == k and all(flag[0, i] for i in idx[0])
            assert np.all(np.diff(idx[0]) > 0)   # ascending token order


def test_uniform_saliency_protects_first_tokens():
    idx, flag = oracle.select_protected_tokens(np.full((2, 37), 1.0 / 37), 5)
    np.testing.assert_array_equal(idx, [[0, 1, 2, 3, 4]] * 2)


# -------------------------------------------------------- Eq. (9)-(11), tokens
def test_all_tokens_protected_is_dense_attention():
    B, H, N, d, block = 2, 2, 22, 5, 4
    q, k, v = (_rand((B, H, N, d), s) for s in (3, 4, 5))
    (kv_idx, kv_cnt), _ = _random_lists(B, H, -(-N // block), 6)
    O, lse = oracle.token_protected_attention(q, k, v, 0.3, block, kv_idx, kv_cnt,
                                              np.ones((B, N), np.uint8))
    Od, lsed = oracle.dense_attention(q, k, v, 0.3)
    np.testing.assert_allclose(O, Od, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, lsed, rtol=0, atol=1e-13)


def test_no_tokens_protected_is_block_sparse_attention():
    B, H, N, d, block = 1, 3, 26, 4, 4
    q, k, v = (_rand((B, H, N, d), s) for s in (7, 8, 9))
    (kv_idx, kv_cnt), _ = _random_lists(B, H, -(-N // block), 10)
    O, lse = oracle.token_protected_attention(q, k, v, 0.5, block, kv_idx, kv_cnt,
                                              np.zeros((B, N), np.uint8))
    Om, lsem = oracle.masked_attention(q, k, v, 0.5, block, kv_idx, kv_cnt)
    np.testing.assert_array_equal(O, Om)
    np.testing.assert_array_equal(lse, lsem)


def test_literal_eq9_mask_with_protected_tokens():
    """Eq. (9)-(10) evaluated with the explicit N x N additive mask: a
    protected query row is all zero, any other row keeps its block pattern."""
    B, H, N, d, block = 2, 2, 30, 5, 4        # ragged tail block of 2
    q, k, v = (_rand((B, H, N, d), s) for s in (11, 12, 13))
    n_b = -(-N // block)
    (kv_idx, kv_cnt), mask = _random_lists(B, H, n_b, 14)
    tok_flag = (np.random.default_rng(15).random((B, N)) < 0.2).astype(np.uint8)
    O, _ = oracle.token_protected_attention(q, k, v, 0.3, block, kv_idx, kv_cnt, tok_flag)
    tok = np.repeat(np.repeat(mask, block, 2), block, 3)[:, :, :N, :N].astype(bool)
    tok = tok | tok_flag[:, None, :, None].astype(bool)
    O2 = oracle.additive_mask_attention(q, k, v, 0.3, tok)
    np.testing.assert_allclose(O, O2, rtol=0, atol=1e-13)


def test_zero_queries_closed_form():
    """Q = 0: a protected row is the mean of V over all tokens, any other row
    the mean over the tokens of its kept key blocks."""
    N, d, block = 8, 3, 2
    k, v = _rand((1, 1, N, d), 16), _rand((1, 1, N, d), 17)
    q = np.zeros((1, 1, N, d))
    kv_idx = np.array([[[[0, -1, -1, -1], [1, 3, -1, -1],
                         [2, -1, -1, -1], [3, 0, -1, -1]]]])
    kv_cnt = np.array([[[1, 2, 1, 2]]])
    tok_flag = np.array([[0, 1, 0, 0, 1, 0, 0, 0]], np.uint8)
    O, lse = oracle.token_protected_attention(q, k, v, 1.0, block, kv_idx, kv_cnt, tok_flag)
    kept = {0: [0, 1], 1: [2, 3, 6, 7], 2: [4, 5], 3: [6, 7, 0, 1]}
    for i in range(N):
        toks = list(range(N)) if tok_flag[0, i] else kept[i // block]
        np.testing.assert_allclose(O[0, 0, i], v[0, 0, toks].mean(0), rtol=0, atol=1e-15)
        assert abs(lse[0, 0, i] - math.log(len(toks))) < 1e-14


def test_protected_rows_helper_matches_full_evaluation():
    B, H, N, d, block = 2, 2, 21, 4, 4
    q, k, v = (_rand((B, H, N, d), s) for s in (18, 19, 20))
    (kv_idx, kv_cnt), _ = _random_lists(B, H, -(-N // block), 21)
    s = np.random.default_rng(22).random((B, N))
    tok_idx, tok_flag = oracle.select_protected_tokens(s, 6)
    O, lse = oracle.token_protected_attention(q, k, v, 0.4, block, kv_idx, kv_cnt, tok_flag)
    rows = [(b, h, j) for b in range(B) for h in range(H) for j in range(6)]
    Or, lr = oracle.token_protected_rows(q, k, v, 0.4, tok_idx, rows)
    for (b, h, j) in rows:
        t = tok_idx[b, j]
        np.testing.assert_allclose(Or[(b, h, j)], O[b, h, t], rtol=0, atol=1e-14)
        assert abs(lr[(b, h, j)] - lse[b, h, t]) < 1e-14
