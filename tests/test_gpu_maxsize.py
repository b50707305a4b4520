"""GPU parity at the largest supported sizes (n_b = 2048 key blocks,
L = 262144 tokens) through the C ABI against the oracle: the four-call layer
with saliency, selection and lists in full and attention on sampled rows, and
token selection over the longest sequence."""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import (TOL_LSE, TOL_O, check_saliency, check_kv_lists, check_protected, gpu_layer,
                       workers)

pytestmark = pytest.mark.gpu

BASE = synth.WORKLOADS["ovi_bf16"]
MAX = [
    # 2047 full blocks of 128 and an 84-token tail
    ("b128_d128_nb2048_tail84", BASE.with_(name="m1", H=1, frames=1, rows=1, cols=262100,
                                           L_a=64, n_plant=8), 16, 8),
    # 2048 blocks of 64, head dimension 64
    ("b64_d64_nb2048", BASE.with_(name="m2", H=1, d=64, block=64, frames=32, rows=64,
                                  cols=64, L_a=40, n_plant=4), 8, 3),
]


@pytest.mark.parametrize("name,w,k_keep,k_prot", MAX, ids=[c[0] for c in MAX])
def test_layer_at_maximum_block_count(name, w, k_keep, k_prot):
    assert w.n_b == 2048
    print(f"case max {name}: L_v={w.L_v} n_b={w.n_b} k_keep={k_keep} k_prot={k_prot}",
          flush=True)
    x = synth.make_inputs(w)
    g = gpu_layer(x, w, k_keep, k_prot)
    print(f"{name}: gpu done", flush=True)
    s_v, s_a = oracle.cross_scores(x["q_a"], x["k_v"], w.scale, x["q_v"], x["k_a"],
                                   workers=workers())
    s_blk = oracle.token_to_block_saliency(s_v, w.block)
    check_saliency(g["sal_v_tok"], s_v, "sal_v_tok")
    check_saliency(g["sal_v_blk"], s_blk, "sal_v_blk")
    check_saliency(g["sal_a_tok"], s_a, "sal_a_tok")
    check_protected(g["prot_idx"], g["prot_flag"], s_blk, k_prot)
    G = oracle.pooled_scores(x["q_v"], x["k_v"], w.scale, w.block)
    assert np.all(np.abs(g["scores"] - G) <= 2.0 ** -24 * np.abs(G) + 1e-12)
    check_kv_lists(g["kv_idx"], g["kv_cnt"], g["prot_flag"], G, k_keep, g["mask"])
    prot = int(g["prot_idx"][0, 0])
    rows = sorted({(0, 0, 0), (0, 0, 1000), (0, 0, w.n_b - 1), (0, 0, prot)})
    O_ref, lse_ref = oracle.masked_attention(x["q_v"], x["k_v"], x["v_v"], w.scale, w.block,
                                             g["kv_idx"], g["kv_cnt"], rows=rows)
    for (b, h, r) in rows:
        lo, hi = r * w.block, min((r + 1) * w.block, w.L_v)
        assert float(np.abs(g["o"][b, h, lo:hi] - O_ref[(b, h, r)]).max()) <= TOL_O["bf16"]
        assert float(np.abs(g["lse"][b, h, lo:hi] - lse_ref[(b, h, r)]).max()) <= TOL_LSE["bf16"]


@pytest.mark.parametrize("values", ["random", "coarse"])
def test_token_selection_at_maximum_length(values):
    L, k = 262144, 13108
    rng = np.random.default_rng(7)
    s = rng.random((1, L)).astype(np.float32)
    if values == "coarse":
        s = np.round(s * 50).astype(np.float32) / 50
    idx, flag = sa.sa_select_protected_tokens(torch.from_numpy(s).cuda(), k)
    torch.cuda.synchronize()
    ref_idx, ref_flag = oracle.select_protected_tokens(s, k)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    assert np.array_equal(flag.cpu().numpy(), ref_flag)
