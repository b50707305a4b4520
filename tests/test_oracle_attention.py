"""Pins of the oracle's attention (Eq. (5), (7), (10), (11)) against closed
forms, a library routine, invariants and brute force.  CPU only."""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _dense_lists(B, H, n_b):
    kv_idx = np.tile(np.arange(n_b), (B, H, n_b, 1))
    kv_cnt = np.full((B, H, n_b), n_b)
    return kv_idx, kv_cnt


def _random_lists(B, H, n_b, seed):
    rng = np.random.default_rng(seed)
    mask = (rng.random((B, H, n_b, n_b)) < 0.4).astype(np.uint8)
    mask[..., 0, :] = 1                      # one dense row per head
    mask[mask.sum(-1) == 0, 0] = 1           # no empty row
    return oracle.kv_lists_from_mask(mask), mask


def test_golden_closed_form():
    g = json.load(open(os.path.join(GOLDEN, "closed_form_attention.json")))
    N, d = g["N"], g["d"]
    q = np.array(g["q"]).reshape(1, 1, N, d)
    k = np.log(np.array(g["key_weights"])).reshape(1, 1, N, d)
    v = np.array(g["v"]).reshape(1, 1, N, d)
    for case in g["cases"]:
        kv_idx = np.array(case["kv_idx"]).reshape(1, 1, 2, 2)
        kv_cnt = np.array(case["kv_cnt"]).reshape(1, 1, 2)
        O, lse = oracle.masked_attention(q, k, v, g["scale"], g["block"],
                                         kv_idx, kv_cnt)
        np.testing.assert_allclose(O.reshape(-1), case["O"], rtol=1e-14)
        if case["name"] == "dense":
            np.testing.assert_allclose(lse.reshape(-1), g["lse_dense"],
                                       rtol=1e-14)
        if case["name"] == "empty_row1":
            assert np.all(np.isneginf(lse[0, 0, 2:]))


def test_dense_case_matches_torch_sdpa_fp64():
    B, H, N, d, block = 1, 2, 40, 8, 8
    q, k, v = (_rand((B, H, N, d), s) for s in (1, 2, 3))
    scale = 1 / math.sqrt(d)
    kv_idx, kv_cnt = _dense_lists(B, H, N // block)
    O, lse = oracle.masked_attention(q, k, v, scale, block, kv_idx, kv_cnt)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        scale=scale).numpy()
    np.testing.assert_allclose(O, ref, atol=1e-12, rtol=0)
    Od, lsed = oracle.dense_attention(q, k, v, scale)
    np.testing.assert_allclose(Od, ref, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, lsed, atol=1e-12, rtol=0)
    # lse against torch.logsumexp of the logits
    S = scale * torch.from_numpy(q) @ torch.from_numpy(k).transpose(-1, -2)
    np.testing.assert_allclose(lse, torch.logsumexp(S, -1).numpy(),
                               atol=1e-12, rtol=0)


def test_brute_force_pure_python_tiny():
    """Element-by-element softmax in plain Python on a 5-token input with a
    ragged last block (block 2: blocks {0,1}, {2,3}, {4})."""
    N, d, block = 5, 3, 2
    q, k, v = (_rand((1, 1, N, d), s) for s in (4, 5, 6))
    kv_idx = np.array([[[[0, 2, -1], [1, -1, -1], [0, 1, 2]]]])
    kv_cnt = np.array([[[2, 1, 3]]])
    O, lse = oracle.masked_attention(q, k, v, 0.7, block, kv_idx, kv_cnt)
    keep = {0: [0, 1, 4], 1: [0, 1, 4], 2: [2, 3], 3: [2, 3], 4: [0, 1, 2, 3, 4]}
    for i in range(N):
        logits = {j: 0.7 * sum(q[0, 0, i, t] * k[0, 0, j, t] for t in range(d))
                  for j in keep[i]}
        z = sum(math.exp(x) for x in logits.values())
        for t in range(d):
            o = sum(math.exp(logits[j]) * v[0, 0, j, t] for j in keep[i]) / z
            assert abs(O[0, 0, i, t] - o) < 1e-13
        assert abs(lse[0, 0, i] - math.log(z)) < 1e-13


def test_identity_values_expose_probabilities():
    """With V = I (one value column per key), O[i] is row i of P: each row
    sums to 1, masked entries are exactly 0, and kept ratios follow
    exp(scale * q_i . (k_j - k_j'))."""
    B, H, N, d, block = 1, 1, 12, 4, 3
    q, k = _rand((B, H, N, d), 7), _rand((B, H, N, d), 8)
    v = np.eye(N).reshape(1, 1, N, N)
    (kv_idx, kv_cnt), mask = _random_lists(B, H, N // block, 9)
    scale = 0.9
    P, _ = oracle.masked_attention(q, k, v, scale, block, kv_idx, kv_cnt)
    P = P[0, 0]
    np.testing.assert_allclose(P.sum(1), 1.0, atol=1e-14)
    tok_mask = np.repeat(np.repeat(mask[0, 0], block, 0), block, 1).astype(bool)
    assert np.all(P[~tok_mask] == 0.0)
    assert np.all(P[tok_mask] > 0.0)
    for i in range(N):
        js = np.nonzero(tok_mask[i])[0]
        a, b = js[0], js[-1]
        expect = math.exp(scale * float(q[0, 0, i] @ (k[0, 0, a] - k[0, 0, b])))
        assert abs(P[i, a] / P[i, b] - expect) < 1e-12 * max(1.0, expect)


def test_masked_positions_contribute_exactly_zero():
    B, H, N, d, block = 1, 2, 32, 8, 4
    q, k, v = (_rand((B, H, N, d), s) for s in (10, 11, 12))
    n_b = N // block
    (kv_idx, kv_cnt), mask = _random_lists(B, H, n_b, 13)
    O, lse = oracle.masked_attention(q, k, v, 0.5, block, kv_idx, kv_cnt)
    for b in range(B):
        for h in range(H):
            for c in range(n_b):
                users = mask[b, h, :, c].astype(bool)
                k2, v2 = k.copy(), v.copy()
                k2[b, h, c * block:(c + 1) * block] = np.nan
                v2[b, h, c * block:(c + 1) * block] = 1e300
                O2, lse2 = oracle.masked_attention(q, k2, v2, 0.5, block,
                                                   kv_idx, kv_cnt)
                for r in np.nonzero(~users)[0]:
                    sl = slice(r * block, (r + 1) * block)
                    assert np.array_equal(O2[b, h, sl], O[b, h, sl])
                    assert np.array_equal(lse2[b, h, sl], lse[b, h, sl])


def test_literal_additive_mask_equals_gather_form():
    """Eq. (10) with the explicit N x N additive mask equals the row form."""
    B, H, N, d, block = 2, 2, 30, 5, 4        # ragged: last block has 2
    q, k, v = (_rand((B, H, N, d), s) for s in (14, 15, 16))
    n_b = -(-N // block)
    (kv_idx, kv_cnt), mask = _random_lists(B, H, n_b, 17)
    O, _ = oracle.masked_attention(q, k, v, 0.3, block, kv_idx, kv_cnt)
    tok = np.repeat(np.repeat(mask, block, 2), block, 3)[:, :, :N, :N]
    O2 = oracle.additive_mask_attention(q, k, v, 0.3, tok.astype(bool))
    np.testing.assert_allclose(O, O2, atol=1e-13, rtol=0)


def test_hand_enumerated_masks_closed_forms():
    """n_b = 4, block = 2, d = 2.  Q = 0 makes attention uniform over kept
    keys: O_r is the mean of V over the kept tokens.  Constant V gives that
    constant.  A single kept one-token key block returns its V row."""
    N, d, block = 8, 2, 2
    k, v = _rand((1, 1, N, d), 18), _rand((1, 1, N, d), 19)
    q = np.zeros((1, 1, N, d))
    kv_idx = np.array([[[[0, -1, -1, -1], [1, 3, -1, -1],
                         [0, 1, 2, 3], [2, 0, -1, -1]]]])
    kv_cnt = np.array([[[1, 2, 4, 2]]])
    O, lse = oracle.masked_attention(q, k, v, 1.0, block, kv_idx, kv_cnt)
    kept = {0: [0, 1], 1: [2, 3, 6, 7], 2: list(range(8)), 3: [4, 5, 0, 1]}
    for r, toks in kept.items():
        expect = v[0, 0, toks].mean(0)
        for i in (2 * r, 2 * r + 1):
            np.testing.assert_allclose(O[0, 0, i], expect, atol=1e-15)
            assert abs(lse[0, 0, i] - math.log(len(toks))) < 1e-15
    vc = np.full((1, 1, N, d), 3.25)
    Oc, _ = oracle.masked_attention(_rand((1, 1, N, d), 20), k, vc, 1.0,
                                    block, kv_idx, kv_cnt)
    np.testing.assert_allclose(Oc, 3.25, atol=1e-14)
    # one-token tail block: N = 7, block 2 -> block 3 holds token 6 only
    N = 7
    q7, k7, v7 = (_rand((1, 1, N, d), s) for s in (21, 22, 23))
    kv_idx = np.array([[[[3, -1, -1, -1]] * 4]])
    kv_cnt = np.array([[[1, 1, 1, 1]]])
    O7, _ = oracle.masked_attention(q7, k7, v7, 1.0, block, kv_idx, kv_cnt)
    np.testing.assert_allclose(O7[0, 0], np.repeat(v7[0, 0, 6:7], N, 0),
                               atol=1e-15)


def test_protected_rows_are_dense_rows():
    """Eq. (11): a query block with the full key list equals dense attention."""
    B, H, N, d, block = 1, 2, 36, 6, 4
    q, k, v = (_rand((B, H, N, d), s) for s in (24, 25, 26))
    n_b = N // block
    (kv_idx, kv_cnt), _ = _random_lists(B, H, n_b, 27)
    kv_idx[:, :, 5] = np.arange(n_b)
    kv_cnt[:, :, 5] = n_b
    O, lse = oracle.masked_attention(q, k, v, 0.4, block, kv_idx, kv_cnt)
    Od, lsed = oracle.dense_attention(q, k, v, 0.4)
    sl = slice(5 * block, 6 * block)
    np.testing.assert_allclose(O[:, :, sl], Od[:, :, sl], atol=1e-13)
    np.testing.assert_allclose(lse[:, :, sl], lsed[:, :, sl], atol=1e-13)


def test_row_subset_matches_full_evaluation():
    B, H, N, d, block = 2, 2, 26, 4, 4
    q, k, v = (_rand((B, H, N, d), s) for s in (28, 29, 30))
    n_b = -(-N // block)
    (kv_idx, kv_cnt), _ = _random_lists(B, H, n_b, 31)
    O, lse = oracle.masked_attention(q, k, v, 0.5, block, kv_idx, kv_cnt)
    rows = [(1, 0, 6), (0, 1, 2)]
    Os, ls = oracle.masked_attention(q, k, v, 0.5, block, kv_idx, kv_cnt,
                                     rows=rows)
    for (b, h, r) in rows:
        sl = slice(r * block, min((r + 1) * block, N))
        assert np.array_equal(Os[(b, h, r)], O[b, h, sl])
        assert np.array_equal(ls[(b, h, r)], lse[b, h, sl])


def test_scale_enters_as_logit_multiplier():
    B, H, N, d, block = 1, 1, 16, 4, 4
    q, k, v = (_rand((B, H, N, d), s) for s in (32, 33, 34))
    (kv_idx, kv_cnt), _ = _random_lists(B, H, 4, 35)
    O1, _ = oracle.masked_attention(q, k, v, 0.25, block, kv_idx, kv_cnt)
    O2, _ = oracle.masked_attention(2 * q, k, v, 0.125, block, kv_idx, kv_cnt)
    np.testing.assert_allclose(O1, O2, atol=1e-14)
    O3, _ = oracle.masked_attention(q, k, v, 0.5, block, kv_idx, kv_cnt)
    assert np.abs(O3 - O1).max() > 1e-3
