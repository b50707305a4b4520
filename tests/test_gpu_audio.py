"""GPU parity of the audio branch's protected sparse self-attention
(Sec. 4.2, Eq. (8)-(11) with m = a) through the C ABI against the oracle:
audio-token saliency of the v->a direction (Sec. 4.1), protected audio tokens,
the pooled-QK block pattern of the audio Q/K, block-sparse attention, then
the dense rows of the protected tokens."""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import (TOL_LSE, TOL_O, check_kv_lists, check_saliency,
                       check_token_selection, to_dev, workers)

pytestmark = pytest.mark.gpu

BASE = synth.WORKLOADS["ovi_bf16"]
# (name, workload, saliency from the cross scores (True) or a seeded map)
CASES = [
    ("bf16_La200_tail8", BASE.with_(name="a1", H=2, frames=4, rows=10, cols=13, L_a=200,
                                    n_plant=2), True),
    ("bf16_d64_La1000", BASE.with_(name="a2", H=3, d=64, block=64, frames=3, rows=10,
                                   cols=11, L_a=1000, n_plant=1), True),
    ("bf16_block128_La700", BASE.with_(name="a3", H=2, frames=2, rows=10, cols=13, L_a=700,
                                       n_plant=1, block_a=128, rho_a=0.1), True),
    ("f32_tiny", synth.WORKLOADS["tiny_f32"], True),
    ("bf16_B2_La300", BASE.with_(name="a6", B=2, H=2, frames=2, rows=10, cols=13, L_a=300,
                                 n_plant=1), True),
    # the audio shapes of the Ovi-like and LTX-like workloads; a short video
    # side, and a seeded L1-normalised map as the lagged audio saliency
    ("ovi_audio_full", BASE.with_(name="a4", frames=1, rows=1, cols=128, n_plant=0), False),
    ("ltx_audio_full", synth.WORKLOADS["ltx_bf16"].with_(name="a5", frames=1, rows=1,
                                                         cols=128, plant="blocks",
                                                         n_plant=0), False),
]


def gpu_audio_branch(x, v_a, w, sal):
    t = {kk: to_dev(x[kk], w.dtype) for kk in ("q_a", "k_a", "q_v", "k_v")}
    va = to_dev(v_a, w.dtype)
    if sal is None:
        _, _, sal_a = sa.sa_cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"], w.scale,
                                         w.block)
    else:
        sal_a = torch.from_numpy(sal).cuda()
    tok_idx, tok_flag = sa.sa_select_protected_tokens(sal_a, w.k_tok_a)
    kv_idx, kv_cnt, mask, scores = sa.sa_build_block_mask(
        t["q_a"], t["k_a"], w.scale, w.block_a, w.k_keep_a, None, want_mask=True,
        want_scores=True)
    o, lse = sa.sa_sparse_attention(t["q_a"], t["k_a"], va, w.scale, w.block_a, kv_idx,
                                    kv_cnt, want_lse=True)
    o_sparse, lse_sparse = o.clone(), lse.clone()
    sa.sa_protected_token_attention(t["q_a"], t["k_a"], va, w.scale, tok_idx, o, lse)
    torch.cuda.synchronize()
    g = dict(sal_a=sal_a, tok_idx=tok_idx, tok_flag=tok_flag, kv_idx=kv_idx, kv_cnt=kv_cnt,
             mask=mask, scores=scores, o=o, lse=lse, o_sparse=o_sparse,
             lse_sparse=lse_sparse)
    return {kk: (v.float() if v.dtype == torch.bfloat16 else v).cpu().numpy()
            for kk, v in g.items()}


@pytest.mark.parametrize("name,w,from_cross", CASES, ids=[c[0] for c in CASES])
def test_audio_branch_matches_oracle(name, w, from_cross):
    print(f"case audio {name}: B={w.B} H={w.H} d={w.d} L_a={w.L_a} block_a={w.block_a} "
          f"k_keep_a={w.k_keep_a} k_tok_a={w.k_tok_a}", flush=True)
    x = synth.make_inputs(w)
    v_a = synth.make_audio_values(w)
    sal = None
    if not from_cross:
        sal = np.random.default_rng(w.L_a).random((w.B, w.L_a)).astype(np.float32)
        sal /= sal.sum(axis=1, keepdims=True)
    g = gpu_audio_branch(x, v_a, w, sal)
    if from_cross:
        _, s_a = oracle.cross_scores(x["q_a"], x["k_v"], w.scale, x["q_v"], x["k_a"],
                                     workers=workers())
        check_saliency(g["sal_a"], s_a, "sal_a_tok")
        # the protected audio tokens against the oracle's fp64 saliency
        check_token_selection(g["tok_idx"], s_a, w.k_tok_a)
    # and bit-exact against the oracle's selection on the same fp32 values
    ref_idx, ref_flag = oracle.select_protected_tokens(g["sal_a"], w.k_tok_a)
    assert np.array_equal(g["tok_idx"], ref_idx)
    assert np.array_equal(g["tok_flag"], ref_flag)
    G = oracle.pooled_scores(x["q_a"], x["k_a"], w.scale, w.block_a)
    assert np.all(np.abs(g["scores"] - G) <= 2.0 ** -24 * np.abs(G) + 1e-12)
    no_prot = np.zeros((w.B, w.n_b_a), dtype=np.uint8)
    check_kv_lists(g["kv_idx"], g["kv_cnt"], no_prot, G, w.k_keep_a, g["mask"])
    # rows of unprotected tokens keep the sparse result bitwise
    keep = np.broadcast_to(g["tok_flag"][:, None, :] == 0, g["lse"].shape)
    assert np.array_equal(g["o"][keep], g["o_sparse"][keep])
    assert np.array_equal(g["lse"][keep], g["lse_sparse"][keep])
    O_ref, lse_ref = oracle.token_protected_attention(
        x["q_a"], x["k_a"], v_a, w.scale, w.block_a, g["kv_idx"], g["kv_cnt"], g["tok_flag"])
    o_err = float(np.abs(g["o"] - O_ref).max())
    l_err = float(np.abs(g["lse"] - lse_ref).max())
    print(name, dict(o_err=o_err, lse_err=l_err), flush=True)
    assert o_err <= TOL_O[w.dtype] and l_err <= TOL_LSE[w.dtype]
