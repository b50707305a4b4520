"""Pins of the oracle's token-protected sparse self-attention of one modality
(Eq. (8)-(11), m in {v, a}; the audio branch uses the audio-token saliency):
a pure-Python evaluation of every step on tiny inputs, and the dense limit.
CPU only."""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle
import synth


def _first_k(vals, k):
    """The k-subset whose every member beats every non-member (larger value,
    then lower index), found by trying all subsets."""
    n = len(vals)
    for sub in itertools.combinations(range(n), k):
        rest = [j for j in range(n) if j not in sub]
        if all(vals[i] > vals[j] or (vals[i] == vals[j] and i < j)
               for i in sub for j in rest):
            return set(sub)
    raise AssertionError("no dominating subset")


def _loops(q, k, v, sal, scale, block, k_keep, k_tok):
    B, H, N, d = q.shape
    n_b = -(-N // block)
    O = np.zeros((B, H, N, d))
    lse = np.zeros((B, H, N))
    for b in range(B):
        prot = _first_k(list(sal[b]), k_tok)
        for h in range(H):
            def mean_rows(x, c):
                rows = range(c * block, min((c + 1) * block, N))
                return [sum(x[b, h, i, e] for i in rows) / len(rows) for e in range(d)]
            qb = [mean_rows(q, c) for c in range(n_b)]
            kb = [mean_rows(k, c) for c in range(n_b)]
            G = [[scale * sum(qb[r][e] * kb[c][e] for e in range(d)) for c in range(n_b)]
                 for r in range(n_b)]
            for i in range(N):
                if i in prot:
                    keys = list(range(N))
                else:
                    kept = _first_k(G[i // block], k_keep)
                    keys = [j for j in range(N) if j // block in kept]
                s = [scale * sum(q[b, h, i, e] * k[b, h, j, e] for e in range(d)) for j in keys]
                mx = max(s)
                p = [math.exp(x - mx) for x in s]
                den = sum(p)
                for e in range(d):
                    O[b, h, i, e] = sum(pi * v[b, h, j, e] for pi, j in zip(p, keys)) / den
                lse[b, h, i] = mx + math.log(den)
    return O, lse, prot


@pytest.mark.parametrize("N,block,k_keep,k_tok", [(10, 4, 2, 3), (9, 3, 1, 0), (8, 4, 1, 8),
                                                  (11, 4, 3, 2)])
def test_layer_against_loops(N, block, k_keep, k_tok):
    rng = np.random.default_rng(N * 10 + k_tok)
    B, H, d = 1, 2, 3
    q, k, v = (rng.standard_normal((B, H, N, d)) for _ in range(3))
    sal = np.round(rng.random((B, N)), 1)     # ties among the saliencies
    scale = 0.7
    r = oracle.modality_protected_layer(q, k, v, sal, scale, block, k_keep, k_tok)
    O, lse, prot = _loops(q, k, v, sal, scale, block, k_keep, k_tok)
    assert set(r["tok_idx"][0].tolist()) == prot
    np.testing.assert_allclose(r["O"], O, rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["lse"], lse, rtol=0, atol=1e-12)


def test_every_token_protected_is_dense_attention():
    """k_tok = N: Eq. (11) is dense attention for every row (torch's fp64
    scaled_dot_product_attention)."""
    w = synth.WORKLOADS["tiny_f32"]
    x = synth.make_inputs(w)
    v_a = synth.make_audio_values(w)
    q, k = x["q_a"].astype(np.float64), x["k_a"].astype(np.float64)
    v = v_a.astype(np.float64)
    sal = np.random.default_rng(0).random((w.B, w.L_a))
    r = oracle.modality_protected_layer(q, k, v, sal, w.scale, w.block_a, 1, w.L_a)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), scale=w.scale)
    np.testing.assert_allclose(r["O"], ref.numpy(), rtol=0, atol=1e-12)


def test_audio_budgets_and_values():
    w = synth.WORKLOADS["ovi_bf16"]
    assert (w.n_b_a, w.k_keep_a, w.k_tok_a) == (8, 2, 26)
    w = synth.WORKLOADS["ltx_bf16"]
    assert (w.n_b_a, w.k_keep_a, w.k_tok_a) == (16, 4, 52)
    w = synth.WORKLOADS["tiny_f32"]
    a = synth.make_audio_values(w)
    assert a.shape == (w.B, w.H, w.L_a, w.d)
    np.testing.assert_array_equal(a, synth.make_audio_values(w))
    # the other inputs' draws do not depend on the audio values
    x0 = synth.make_inputs(w)
    synth.make_audio_values(w)
    np.testing.assert_array_equal(x0["q_v"], synth.make_inputs(w)["q_v"])
    b = synth.make_audio_values(synth.WORKLOADS["ovi_bf16"].with_(H=1))
    assert np.array_equal(b, synth.round_to_bf16(b).reshape(b.shape))
