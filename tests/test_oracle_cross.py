"""Pins of the oracle's cross-modal attention forwards and of the saliency
taken from their softmax (Eq. (1)-(2)).  CPU only."""
import numpy as np
import torch

import oracle


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_dense_attention_with_other_key_length_is_sdpa():
    """Queries and keys of different lengths: torch's fp64 SDPA."""
    q, k, v = _rand((2, 3, 7, 16), 0), _rand((2, 3, 29, 16), 1), _rand((2, 3, 29, 16), 2)
    O, lse = oracle.dense_attention(q, k, v, 0.3)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), scale=0.3)
    np.testing.assert_allclose(O, ref.numpy(), rtol=0, atol=1e-13)
    S = 0.3 * np.einsum("bhqd,bhkd->bhqk", q, k)
    np.testing.assert_allclose(lse, np.log(np.exp(S).sum(-1)), rtol=0, atol=1e-12)


def test_saliency_is_the_column_mass_of_the_forward_softmax():
    """With V^v = I (one value channel per video key) row j of O^a is row j of
    A^{a->v}; its sum over audio queries and heads is H*L_a*s^v (Eq. (2)).
    Likewise V^a = I gives H*L_v*s^a from O^v."""
    B, H, La, Lv = 2, 3, 5, 11
    d = 8
    q_a, k_a = _rand((B, H, La, d), 3), _rand((B, H, La, d), 4)
    q_v, k_v = _rand((B, H, Lv, d), 5), _rand((B, H, Lv, d), 6)
    v_v = np.broadcast_to(np.eye(Lv), (B, H, Lv, Lv)).copy()
    v_a = np.broadcast_to(np.eye(La), (B, H, La, La)).copy()
    r = oracle.cross_attention_with_saliency(q_a, k_a, v_a, q_v, k_v, v_v, 0.4)
    np.testing.assert_allclose(r["O_a"].sum(axis=(1, 2)), H * La * r["sal_v_tok"],
                               rtol=1e-13, atol=0)
    np.testing.assert_allclose(r["O_v"].sum(axis=(1, 2)), H * Lv * r["sal_a_tok"],
                               rtol=1e-13, atol=0)
    # and exp(scale q.k - lse) is that softmax
    S = 0.4 * np.einsum("bhjd,bhid->bhji", q_a, k_v)
    np.testing.assert_allclose(np.exp(S - r["lse_a"][..., None]), r["O_a"], rtol=1e-12,
                               atol=1e-15)
