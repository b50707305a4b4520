"""GPU parity of the cross-modal attention forwards and of the saliency taken
from their row log-sum-exps (Eq. (1)-(2)) through the C ABI, against the
oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import (TOL_LSE, TOL_O, check_saliency, logit_ramp_inputs, to_dev,
                       workers)

pytestmark = pytest.mark.gpu


def _np(t):
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy()


# (B, H, Lq, Lk, d): a->v shapes (few queries, many keys: the keys of a row
# block are split into runs), v->a shapes (many queries, few keys), ragged
# tails, a single query
FORWARD = [(1, 2, 64, 520, 128), (2, 3, 200, 1000, 64), (1, 2, 300, 4000, 128),
           (1, 1, 1, 700, 128), (1, 2, 2000, 130, 128), (2, 2, 777, 64, 64),
           (1, 24, 512, 4096, 128)]


@pytest.mark.parametrize("B,H,Lq,Lk,d", FORWARD)
def test_cross_attention_matches_oracle(B, H, Lq, Lk, d):
    print(f"case cross fwd B={B} H={H} Lq={Lq} Lk={Lk} d={d} ws="
          f"{sa.sa_workspace_size(sa.SA_CALL_CROSS_ATTENTION, B, H, Lq, Lk, d, 0)}", flush=True)
    rng = np.random.default_rng(Lq * 7 + Lk)
    q, k, v = (synth.round_to_bf16(rng.standard_normal((B, H, L, d), dtype=np.float32))
               .reshape(B, H, L, d) for L in (Lq, Lk, Lk))
    scale = float(np.float32(1.0 / np.sqrt(d)))
    o, lse = sa.sa_cross_attention(to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16"),
                                   scale, want_lse=True)
    torch.cuda.synchronize()
    O_ref, lse_ref = oracle.dense_attention(q, k, v, scale)
    o_err = float(np.abs(_np(o) - O_ref).max())
    l_err = float(np.abs(_np(lse) - lse_ref).max())
    print(dict(o_err=o_err, lse_err=l_err), flush=True)
    assert o_err <= TOL_O["bf16"] and l_err <= TOL_LSE["bf16"]


@pytest.mark.parametrize("profile", ["grow", "jump"])
@pytest.mark.parametrize("Lq,Lk", [(64, 4000), (300, 1000)])
def test_cross_attention_under_large_logit_changes(profile, Lq, Lk):
    """Logits rising by ~100 log2 units along the keys, or jumping by ~150 in
    the last 50: the running max of each key run, and the merge of runs whose
    maxima differ by that much (Lq = 64: the keys of a row block are cut into
    runs), against dense fp64 attention."""
    d, H = 128, 2
    ws = sa.sa_workspace_size(sa.SA_CALL_CROSS_ATTENTION, 1, H, Lq, Lk, d, 0)
    print(f"case cross ramp {profile} Lq={Lq} Lk={Lk} ws={ws}", flush=True)
    q, k, v = logit_ramp_inputs(Lq, Lk, d, H, profile, "bf16")
    scale = float(np.float32(1.0 / np.sqrt(d)))
    o, lse = sa.sa_cross_attention(to_dev(q, "bf16"), to_dev(k, "bf16"), to_dev(v, "bf16"),
                                   scale, want_lse=True)
    torch.cuda.synchronize()
    O_ref, lse_ref = oracle.dense_attention(q, k, v, scale)
    o_err = float(np.abs(_np(o) - O_ref).max())
    l_err = float(np.abs(_np(lse) - lse_ref).max())
    print(profile, dict(o_err=o_err, lse_err=l_err), flush=True)
    assert np.all(np.isfinite(_np(o)))
    assert o_err <= TOL_O["bf16"] and l_err <= TOL_LSE["bf16"]


SAL = [("small", synth.WORKLOADS["ovi_bf16"].with_(name="c1", H=2, frames=4, rows=10,
                                                   cols=13, L_a=200, n_plant=2)),
       ("d64", synth.WORKLOADS["ovi_bf16"].with_(name="c2", H=3, d=64, block=64, frames=3,
                                                 rows=10, cols=11, L_a=1000, n_plant=1)),
       ("B2", synth.WORKLOADS["ovi_bf16"].with_(name="c3", B=2, H=2, frames=3, rows=10,
                                                cols=13, L_a=150, n_plant=1)),
       ("ovi", synth.WORKLOADS["ovi_bf16"])]


@pytest.mark.parametrize("name,w", SAL, ids=[c[0] for c in SAL])
def test_saliency_from_forward_lse_matches_oracle(name, w):
    """Both forwards, then the saliency from their row LSEs: the forwards on
    sampled rows (all rows below the Ovi size), the saliency of both
    directions in full, and agreement with the standalone saliency call."""
    print(f"case cross sal {name}: H={w.H} L_v={w.L_v} L_a={w.L_a}", flush=True)
    x = synth.make_inputs(w)
    v_a = synth.make_audio_values(w)
    t = {kk: to_dev(x[kk], w.dtype) for kk in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    va = to_dev(v_a, w.dtype)
    o_a, lse_a = sa.sa_cross_attention(t["q_a"], t["k_v"], t["v_v"], w.scale, want_lse=True)
    o_v, lse_v = sa.sa_cross_attention(t["q_v"], t["k_a"], va, w.scale, want_lse=True)
    s_v, s_blk, s_a = sa.sa_cross_scores_from_lse(t["q_a"], t["k_v"], t["q_v"], t["k_a"],
                                                  lse_a, lse_v, w.scale, w.block)
    r_v, r_blk, r_a = sa.sa_cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"], w.scale,
                                         w.block)
    torch.cuda.synchronize()
    print(f"{name}: gpu done", flush=True)
    s_v_ref, s_a_ref = oracle.cross_scores(x["q_a"], x["k_v"], w.scale, x["q_v"], x["k_a"],
                                           workers=workers())
    errs = dict(sal_v=float(np.abs(_np(s_v) - s_v_ref).max()),
                sal_a=float(np.abs(_np(s_a) - s_a_ref).max()),
                blk=float(np.abs(_np(s_blk) - oracle.token_to_block_saliency(s_v_ref, w.block)).max()),
                vs_standalone=float(np.abs(_np(s_v) - _np(r_v)).max()))
    print(name, errs, flush=True)
    check_saliency(_np(s_v), s_v_ref, "sal_v_tok")
    check_saliency(_np(s_a), s_a_ref, "sal_a_tok")
    check_saliency(_np(s_blk), oracle.token_to_block_saliency(s_v_ref, w.block), "sal_v_blk")
    # forwards: every row below the Ovi size, else 16 sampled rows per direction
    rng = np.random.default_rng(0)
    for (q, k, v, o, lse, Lq) in ((x["q_a"], x["k_v"], x["v_v"], o_a, lse_a, w.L_a),
                                  (x["q_v"], x["k_a"], v_a, o_v, lse_v, w.L_v)):
        rows = np.arange(Lq) if Lq * w.H <= 20000 else np.unique(rng.integers(0, Lq, 16))
        O_ref, lse_ref = oracle.dense_attention(q[:, :, rows], k, v, w.scale)
        assert float(np.abs(_np(o)[:, :, rows] - O_ref).max()) <= TOL_O["bf16"]
        assert float(np.abs(_np(lse)[:, :, rows] - lse_ref).max()) <= TOL_LSE["bf16"]
