"""GPU parity of the token-granular protection path through the C ABI: the
lagged saliency update (Eq. (4)), protected token selection (Eq. (8) at token
level) and the dense rows of the protected tokens over the block-sparse
output (Eq. (9)-(11)), against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import (TOL_LSE, TOL_O, check_saliency, check_token_selection, to_dev,
                       workers)

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ Eq. (4)
@pytest.mark.parametrize("n,alpha", [(1, 0.5), (1000, 0.3), (300001, 0.75),
                                     (17, 0.0), (17, 1.0)])
def test_saliency_ema_matches_oracle(n, alpha):
    print(f"case ema n={n} alpha={alpha}", flush=True)
    rng = np.random.default_rng(n)
    prev = rng.random(n).astype(np.float32)
    cur = rng.random(n).astype(np.float32)
    sb = torch.from_numpy(prev.copy()).cuda()
    sa.sa_saliency_ema(sb, torch.from_numpy(cur).cuda(), alpha)
    torch.cuda.synchronize()
    ref = oracle.saliency_ema(prev, cur, alpha)
    # fp32: (1 - alpha), its product with sal and the fused add round once each
    np.testing.assert_allclose(sb.cpu().numpy(), ref, rtol=2.0 ** -22, atol=0)
    if alpha in (0.0, 1.0):
        np.testing.assert_array_equal(sb.cpu().numpy(), cur if alpha == 0.0 else prev)


def test_saliency_ema_in_place_is_a_fixed_point():
    x = torch.rand(4097, device="cuda")
    y = x.clone()
    sa.sa_saliency_ema(x, x, 0.3)
    torch.cuda.synchronize()
    np.testing.assert_allclose(x.cpu().numpy(), y.cpu().numpy(), rtol=2.0 ** -22, atol=0)


# ------------------------------------------------------- Eq. (8), token level
# one wave up to L = 512 and up to 2048; 16 waves with 4, 16 or 32 register
# keys per lane, or keys read from memory beyond L = 32768
SELECT = [(1, 1, 0), (1, 1, 1), (2, 5, 3), (1, 512, 26), (1, 513, 26), (1, 1000, 50),
          (2, 1000, 1000), (1, 1000, 0), (1, 2048, 103), (1, 2049, 103), (1, 4096, 205),
          (3, 16384, 820), (1, 16385, 5000), (1, 32760, 1638), (1, 32768, 4000),
          (1, 32769, 1639), (2, 75600, 3780)]


@pytest.mark.parametrize("B,L,k", SELECT)
@pytest.mark.parametrize("values", ["random", "coarse"])
def test_select_protected_tokens_matches_oracle(B, L, k, values):
    """Bit-exact against the oracle on the same fp32 values: random values,
    and coarse values with many exact ties (lower index first)."""
    print(f"case select B={B} L={L} k={k} {values}", flush=True)
    rng = np.random.default_rng(L + k)
    s = rng.random((B, L)).astype(np.float32)
    if values == "coarse":
        s = np.round(s * 20).astype(np.float32) / 20
    idx, flag = sa.sa_select_protected_tokens(torch.from_numpy(s).cuda(), k)
    torch.cuda.synchronize()
    ref_idx, ref_flag = oracle.select_protected_tokens(s, k)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    assert np.array_equal(flag.cpu().numpy(), ref_flag)


def test_uniform_saliency_protects_the_first_tokens():
    s = torch.full((2, 5000), 1.0 / 5000, device="cuda")
    idx, flag = sa.sa_select_protected_tokens(s, 250)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), np.tile(np.arange(250), (2, 1)))
    assert int(flag.sum()) == 500 and int(flag[:, :250].sum()) == 500


# -------------------------------------------------------- Eq. (9)-(11), tokens
BASE = synth.WORKLOADS["ovi_bf16"]
LAYERS = [
    ("bf16_d128", BASE.with_(name="t1", H=2, frames=4, rows=10, cols=13, L_a=64,
                             n_plant=2), 3, 0.05),
    ("bf16_d64_b64", BASE.with_(name="t2", H=3, d=64, block=64, frames=3, rows=10,
                                cols=11, L_a=40, n_plant=1), 2, 0.1),
    ("bf16_d128_many_tokens", BASE.with_(name="t3", H=1, frames=3, rows=10, cols=15,
                                         L_a=32, n_plant=1), 2, 0.6),
    ("f32_tiny", synth.WORKLOADS["tiny_f32"], 4, 0.1),
    # 16 key blocks of 128 with an 80-key tail: the keys of a row go to 4 runs
    ("bf16_d128_split4", BASE.with_(name="t4", H=2, frames=4, rows=10, cols=50, L_a=64,
                                    n_plant=2), 3, 0.05),
    # 11 key blocks of 128: two runs of 5 and 6 blocks
    ("bf16_d64_split2", BASE.with_(name="t5", H=3, d=64, block=64, frames=2, rows=10,
                                   cols=65, L_a=40, n_plant=1), 4, 0.1),
    # two batch items: each has its own protected tokens, shared by its heads
    ("bf16_B2_split4", BASE.with_(name="t7", B=2, H=2, frames=4, rows=10, cols=50, L_a=64,
                                  n_plant=2), 3, 0.05),
]


def gpu_token_layer(x, w, k_keep, k_tok):
    """Saliency, token selection, unprotected block mask, sparse attention,
    then the protected tokens' dense rows over it."""
    t = {kk: to_dev(x[kk], w.dtype) for kk in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    sal_v_tok, _, _ = sa.sa_cross_scores(t["q_a"], t["k_v"], None, None, w.scale, w.block)
    tok_idx, tok_flag = sa.sa_select_protected_tokens(sal_v_tok, k_tok)
    kv_idx, kv_cnt, _, _ = sa.sa_build_block_mask(t["q_v"], t["k_v"], w.scale, w.block,
                                                  k_keep, None)
    o, lse = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, w.block,
                                    kv_idx, kv_cnt, want_lse=True)
    o_sparse, lse_sparse = o.clone(), lse.clone()
    sa.sa_protected_token_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, tok_idx, o, lse)
    torch.cuda.synchronize()
    g = dict(sal_v_tok=sal_v_tok, tok_idx=tok_idx, tok_flag=tok_flag, kv_idx=kv_idx,
             kv_cnt=kv_cnt, o=o, lse=lse, o_sparse=o_sparse, lse_sparse=lse_sparse)
    return {kk: (v.float() if v.dtype == torch.bfloat16 else v).cpu().numpy()
            for kk, v in g.items()}


def check_untouched(g):
    """Rows of tokens outside the protected set keep the sparse result bitwise."""
    keep = g["tok_flag"][:, None, :] == 0
    keep = np.broadcast_to(keep, g["lse"].shape)
    assert np.array_equal(g["o"][keep], g["o_sparse"][keep])
    assert np.array_equal(g["lse"][keep], g["lse_sparse"][keep])


@pytest.mark.parametrize("name,w,k_keep,rho", LAYERS, ids=[c[0] for c in LAYERS])
def test_token_protected_layer_matches_oracle(name, w, k_keep, rho):
    k_tok = synth.budget(rho, w.L_v)
    print(f"case {name}: B={w.B} H={w.H} d={w.d} L_v={w.L_v} block={w.block} "
          f"k_keep={k_keep} k_tok={k_tok}", flush=True)
    x = synth.make_inputs(w)
    g = gpu_token_layer(x, w, k_keep, k_tok)
    # the saliency and the protected tokens against the oracle's fp64 saliency
    s_v, _ = oracle.cross_scores(x["q_a"], x["k_v"], w.scale, workers=workers())
    check_saliency(g["sal_v_tok"], s_v, "sal_v_tok")
    check_token_selection(g["tok_idx"], s_v, k_tok)
    # and bit-exact against the oracle's selection on the same fp32 values
    ref_idx, ref_flag = oracle.select_protected_tokens(g["sal_v_tok"], k_tok)
    assert np.array_equal(g["tok_idx"], ref_idx)
    assert np.array_equal(g["tok_flag"], ref_flag)
    check_untouched(g)
    O_ref, lse_ref = oracle.token_protected_attention(
        x["q_v"], x["k_v"], x["v_v"], w.scale, w.block, g["kv_idx"], g["kv_cnt"],
        g["tok_flag"])
    o_err = float(np.abs(g["o"] - O_ref).max())
    l_err = float(np.abs(g["lse"] - lse_ref).max())
    print(name, dict(o_err=o_err, lse_err=l_err), flush=True)
    assert o_err <= TOL_O[w.dtype] and l_err <= TOL_LSE[w.dtype]


def test_token_protected_layer_fullsize_ovi():
    """The Ovi-like layer with 5 % protected tokens: selection in full, every
    unprotected row untouched, sampled protected rows against dense fp64 rows."""
    w = BASE
    k_tok = synth.budget(0.05, w.L_v)
    print(f"case ovi tokens: L_v={w.L_v} k_keep={w.k_keep} k_tok={k_tok}", flush=True)
    x = synth.make_inputs(w)
    g = gpu_token_layer(x, w, w.k_keep, k_tok)
    print("ovi tokens: gpu done", flush=True)
    s_v, _ = oracle.cross_scores(x["q_a"], x["k_v"], w.scale, workers=workers())
    rel = check_saliency(g["sal_v_tok"], s_v, "sal_v_tok")
    ties = check_token_selection(g["tok_idx"], s_v, k_tok)
    print(f"ovi tokens: saliency rel err {rel:.2e}, {ties} tokens in the tie window",
          flush=True)
    ref_idx, _ = oracle.select_protected_tokens(g["sal_v_tok"], k_tok)
    assert np.array_equal(g["tok_idx"], ref_idx)
    check_untouched(g)
    rng = np.random.default_rng(0)
    rows = sorted({(0, int(rng.integers(w.H)), int(rng.integers(k_tok))) for _ in range(24)}
                  | {(0, 0, 0), (0, w.H - 1, k_tok - 1)})
    O_ref, lse_ref = oracle.token_protected_rows(x["q_v"], x["k_v"], x["v_v"], w.scale,
                                                 g["tok_idx"], rows)
    o_err = max(float(np.abs(g["o"][b, h, g["tok_idx"][b, j]] - O_ref[(b, h, j)]).max())
                for (b, h, j) in rows)
    l_err = max(abs(float(g["lse"][b, h, g["tok_idx"][b, j]]) - lse_ref[(b, h, j)])
                for (b, h, j) in rows)
    print("ovi tokens", dict(o_err=o_err, lse_err=l_err), flush=True)
    assert o_err <= TOL_O["bf16"] and l_err <= TOL_LSE["bf16"]
    assert np.all(np.isfinite(g["o"]))


def test_split_rows_skip_out_of_range_entries():
    """With the keys of each row split into runs, entries of tok_idx outside
    [0, L) leave O and lse alone and the other rows are the dense rows."""
    w = BASE.with_(name="t6", H=2, frames=4, rows=10, cols=50, L_a=64, n_plant=1)
    L = w.L_v
    assert sa.sa_workspace_size(sa.SA_CALL_TOKEN_ATTENTION, w.B, w.H, L, 6, w.d, 0) > 0
    x = synth.make_inputs(w)
    t = {kk: to_dev(x[kk], w.dtype) for kk in ("q_v", "k_v", "v_v")}
    idx = torch.tensor([[3, -1, 17, L, 400, L - 1]], dtype=torch.int32, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(1)
    o = torch.randn(t["q_v"].shape, device="cuda", generator=g).to(torch.bfloat16)
    lse = torch.randn(w.B, w.H, L, device="cuda", generator=g)
    o0, lse0 = o.clone(), lse.clone()
    sa.sa_protected_token_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, idx, o, lse)
    torch.cuda.synchronize()
    o, lse, o0, lse0 = (a.float().cpu().numpy() for a in (o, lse, o0, lse0))
    valid = [0, 2, 4, 5]
    tok = idx.cpu().numpy()
    rows = [(0, h, j) for h in range(w.H) for j in valid]
    O_ref, lse_ref = oracle.token_protected_rows(x["q_v"], x["k_v"], x["v_v"], w.scale,
                                                 tok, rows)
    for (b, h, j) in rows:
        r = tok[b, j]
        assert float(np.abs(o[b, h, r] - O_ref[(b, h, j)]).max()) <= TOL_O["bf16"]
        assert abs(float(lse[b, h, r]) - lse_ref[(b, h, j)]) <= TOL_LSE["bf16"]
    other = np.ones(L, dtype=bool)
    other[tok[0, valid]] = False
    assert np.array_equal(o[:, :, other], o0[:, :, other])
    assert np.array_equal(lse[:, :, other], lse0[:, :, other])
