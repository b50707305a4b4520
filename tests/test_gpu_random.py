"""Seeded random configurations through the C ABI against the oracle: the
four-call layer, the token-protected path and the cache indicator, drawn
over batch size, heads, head dimension, block size, ragged video and audio
lengths, budgets and dtype.  Every configuration is small enough for the
oracle to evaluate in full."""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import TOL_LSE, TOL_O, compare_layer, gpu_layer, to_dev

pytestmark = pytest.mark.gpu

BASE = synth.WORKLOADS["ovi_bf16"]


def draw(seed):
    """A workload with a ragged video length and its budgets."""
    rng = np.random.default_rng(1000 + seed)
    dtype = "f32" if seed % 5 == 0 else "bf16"
    d = int(rng.choice([64, 128]))
    block = int(rng.choice([64, 128]))
    frames, rows, cols = int(rng.integers(1, 5)), int(rng.integers(2, 12)), int(rng.integers(3, 40))
    L_v = frames * rows * cols
    n_b = -(-L_v // block)
    n_full = L_v // block
    w = BASE.with_(name=f"rand{seed}", B=int(rng.integers(1, 3)), H=int(rng.integers(1, 4)),
                   d=d, block=block, frames=frames, rows=rows, cols=cols,
                   L_a=int(rng.integers(1, 700)), dtype=dtype, prescale=dtype == "f32",
                   n_plant=int(rng.integers(0, min(n_full, 3) + 1)))
    return w, int(rng.integers(1, n_b + 1)), int(rng.integers(0, n_b + 1)), rng


def _desc(w, **kw):
    return (f"{w.name}: {w.dtype} B={w.B} H={w.H} d={w.d} block={w.block} L_v={w.L_v} "
            f"L_a={w.L_a} " + " ".join(f"{k}={v}" for k, v in kw.items()))


@pytest.mark.parametrize("seed", range(12))
def test_random_layer_matches_oracle(seed):
    w, k_keep, k_prot, _ = draw(seed)
    print("case layer " + _desc(w, k_keep=k_keep, k_prot=k_prot), flush=True)
    x = synth.make_inputs(w)
    g = gpu_layer(x, w, k_keep, k_prot)
    rep = compare_layer(x, w, g, k_keep, k_prot)
    print(rep, flush=True)


@pytest.mark.parametrize("seed", range(12, 20))
def test_random_token_path_matches_oracle(seed):
    w, k_keep, _, rng = draw(seed)
    k_tok = int(rng.integers(0, w.L_v + 1))
    print("case tokens " + _desc(w, k_keep=k_keep, k_tok=k_tok), flush=True)
    x = synth.make_inputs(w)
    t = {kk: to_dev(x[kk], w.dtype) for kk in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    sal, _, _ = sa.sa_cross_scores(t["q_a"], t["k_v"], None, None, w.scale, w.block)
    tok_idx, tok_flag = sa.sa_select_protected_tokens(sal, k_tok)
    kv_idx, kv_cnt, _, _ = sa.sa_build_block_mask(t["q_v"], t["k_v"], w.scale, w.block,
                                                  k_keep, None)
    o, lse = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, w.block, kv_idx,
                                    kv_cnt, want_lse=True)
    o0, lse0 = o.clone(), lse.clone()
    sa.sa_protected_token_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, tok_idx, o, lse)
    torch.cuda.synchronize()
    f = lambda v: (v.float() if v.dtype == torch.bfloat16 else v).cpu().numpy()
    sal, tok_idx, tok_flag, kv_idx, kv_cnt, o, lse, o0, lse0 = map(
        f, (sal, tok_idx, tok_flag, kv_idx, kv_cnt, o, lse, o0, lse0))
    ref_idx, ref_flag = oracle.select_protected_tokens(sal, k_tok)
    assert np.array_equal(tok_idx, ref_idx) and np.array_equal(tok_flag, ref_flag)
    keep = np.broadcast_to(tok_flag[:, None, :] == 0, lse.shape)
    assert np.array_equal(o[keep], o0[keep]) and np.array_equal(lse[keep], lse0[keep])
    O_ref, lse_ref = oracle.token_protected_attention(x["q_v"], x["k_v"], x["v_v"], w.scale,
                                                      w.block, kv_idx, kv_cnt, tok_flag)
    o_err, l_err = float(np.abs(o - O_ref).max()), float(np.abs(lse - lse_ref).max())
    print(dict(o_err=o_err, lse_err=l_err), flush=True)
    assert o_err <= TOL_O[w.dtype] and l_err <= TOL_LSE[w.dtype]


@pytest.mark.parametrize("seed", range(20, 28))
def test_random_cache_indicator_matches_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    B, L_v, L_a = int(rng.integers(1, 3)), int(rng.integers(1, 3000)), int(rng.integers(1, 300))
    C = 8 * int(rng.integers(1, 400))
    dtype = "f32" if seed % 3 == 0 else "bf16"
    audio, sal, prot = (bool(rng.integers(0, 2)) for _ in range(3))
    print(f"case cache seed={seed} {dtype} B={B} L_v={L_v} L_a={L_a} C={C} audio={audio} "
          f"sal={sal} prot={prot}", flush=True)
    dev = lambda a: to_dev(a.astype(np.float32), dtype)
    yv = rng.standard_normal((B, L_v, C))
    yvh = yv + float(rng.random()) * rng.standard_normal((B, L_v, C))
    ya = rng.standard_normal((B, L_a, C)) if audio else None
    yah = ya + 0.2 * rng.standard_normal((B, L_a, C)) if audio else None
    flag = (rng.random((B, L_v)) < 0.1).astype(np.uint8) if prot else None
    sb = rng.random((B, L_v)).astype(np.float32) if sal else None
    sh = rng.random((B, L_v)).astype(np.float32) if sal else None
    t = lambda a: None if a is None else torch.from_numpy(a).cuda()
    out = sa.sa_cache_indicator(dev(yv), dev(yvh), prot_flag=t(flag),
                                y_a=None if ya is None else dev(ya),
                                y_a_hat=None if yah is None else dev(yah), s_bar=t(sb),
                                s_hat=t(sh), lambda_p=0.5, lambda_s=0.1, tau=0.2, eps=1e-6)
    torch.cuda.synchronize()
    g = out.cpu().numpy()
    h = lambda a: None if a is None else to_dev(a.astype(np.float32), dtype).float().cpu().numpy()
    ref = oracle.cache_indicator(h(yv), h(yvh), flag, h(ya), h(yah), sb, sh, 0.5, 0.1, 0.2, 1e-6)
    for i, k in enumerate(("dv", "da", "dp", "ds", "sync")):
        assert abs(g[i] - ref[k]) <= 1e-5 * max(1.0, abs(ref[k])), (k, g[i], ref[k])
    assert g[5] == (1.0 if np.float32(g[4]) < np.float32(0.2) else 0.0)
