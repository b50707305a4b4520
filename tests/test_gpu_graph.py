"""The layer's calls under HIP graph capture: the four-call video layer
(Sec. 4.1-4.2, Eq. (1)-(2), (8)-(11)) and the audio branch's token path
(Eq. (4), (8)-(11) with m = a) are captured once into a graph and replayed
three times, with eager work and synchronisations between the replays.  The
library allocates nothing and records no memory set, so every replay must
reproduce the eager run bit for bit (every kernel sums in a fixed order, and
the attention output does not depend on which workgroup takes a row)."""
import pytest
import torch

import synth
import paper_2608_15522_amd as sa
from paper_2608_15522_amd.layer import LayerPlan
from sa_parity import to_dev

pytestmark = pytest.mark.gpu

BASE = synth.WORKLOADS["ovi_bf16"]
# B*H = 8: the attention runs its persistent, per-XCD scheduled form, whose
# row counters a kernel of the call resets on every replay
W = BASE.with_(name="g1", H=8, frames=4, rows=10, cols=26, L_a=300, n_plant=2)


def _capture(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()  # warm-up on the capture's side of the allocator
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fn()
    torch.cuda.synchronize()
    return graph


def _replays_match(graph, outputs, reference, reset=lambda: None):
    noise = torch.randn(512, 512, device="cuda")
    for rep in range(3):
        for t in outputs:  # poison every output before the replay
            if t.dtype.is_floating_point:
                t.fill_(float("nan"))
            else:
                t.fill_(-7)
        reset()
        _ = noise @ noise  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, t, ref in zip(range(len(outputs)), outputs, reference):
            assert torch.equal(t.view(torch.uint8), ref.view(torch.uint8)), (rep, name)


def test_layer_graph_replays_reproduce_the_eager_layer():
    w = W
    k_keep, k_prot = max(1, w.n_b // 4), 2
    print(f"case graph layer B={w.B} H={w.H} L_v={w.L_v} L_a={w.L_a} n_b={w.n_b}", flush=True)
    x = synth.make_inputs(w)
    t = {k: to_dev(x[k], w.dtype) for k in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    plan = LayerPlan(w.B, w.H, w.L_v, w.L_a, w.d, w.block, k_keep, k_prot, w.scale,
                     want_lse=True)

    def layer():
        plan.run(t["q_v"], t["k_v"], t["v_v"], t["q_a"], t["k_a"])

    layer()
    torch.cuda.synchronize()
    outputs = [plan.sal_v_tok, plan.sal_v_blk, plan.sal_a_tok, plan.prot_flag, plan.kv_idx,
               plan.kv_cnt, plan.o, plan.lse]
    reference = [o.clone() for o in outputs]
    graph = _capture(layer)
    _replays_match(graph, outputs, reference)


def test_pooled_layer_graph_replays_reproduce_the_eager_layer():
    """The same layer with the block means pooled inside the saliency streams
    (sa_cross_scores_pooled + sa_build_block_mask_pooled)."""
    w = W
    k_keep, k_prot = max(1, w.n_b // 4), 2
    print(f"case graph pooled layer B={w.B} H={w.H} L_v={w.L_v} n_b={w.n_b}", flush=True)
    x = synth.make_inputs(w)
    t = {k: to_dev(x[k], w.dtype) for k in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    plan = LayerPlan(w.B, w.H, w.L_v, w.L_a, w.d, w.block, k_keep, k_prot, w.scale,
                     want_lse=True)

    def layer():
        plan.run_pooled(t["q_v"], t["k_v"], t["v_v"], t["q_a"], t["k_a"])

    layer()
    torch.cuda.synchronize()
    n_b = w.n_b
    outputs = [plan.sal_v_tok, plan.sal_v_blk, plan.sal_a_tok, plan.prot_flag, plan.kv_idx,
               plan.kv_cnt, plan.o, plan.lse, plan.qbar[..., :n_b], plan.kbar[..., :n_b]]
    reference = [o.clone() for o in outputs]
    # the eager pooled layer equals the plain one
    plan.run(t["q_v"], t["k_v"], t["v_v"], t["q_a"], t["k_a"])
    torch.cuda.synchronize()
    for o, r in zip(outputs[:8], reference[:8]):
        assert torch.equal(o.view(torch.uint8), r.view(torch.uint8))
    graph = _capture(layer)
    _replays_match(graph, outputs, reference)


def test_audio_branch_graph_replays_reproduce_the_eager_branch():
    w = W
    print(f"case graph audio branch L_a={w.L_a} block_a={w.block_a} k_tok_a={w.k_tok_a}",
          flush=True)
    x = synth.make_inputs(w)
    t = {k: to_dev(x[k], w.dtype) for k in ("q_v", "k_v", "q_a", "k_a")}
    gen = torch.Generator(device="cuda").manual_seed(3)
    v_a = torch.randn(t["q_a"].shape, device="cuda", generator=gen).to(t["q_a"].dtype)
    _, _, sal_a = sa.sa_cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"], w.scale, w.block)
    sal0 = torch.rand(sal_a.shape, device="cuda", generator=gen) * 1e-3
    sal_bar = sal0.clone()
    n_b = -(-w.L_a // w.block_a)
    tok_idx = torch.empty(w.B, w.k_tok_a, dtype=torch.int32, device="cuda")
    kv_idx = torch.empty(w.B, w.H, n_b, n_b, dtype=torch.int32, device="cuda")
    kv_cnt = torch.empty(w.B, w.H, n_b, dtype=torch.int32, device="cuda")
    o = torch.empty_like(t["q_a"])
    lse = torch.empty(w.B, w.H, w.L_a, dtype=torch.float32, device="cuda")

    def ws(call, la):
        n = sa.sa_workspace_size(call, w.B, w.H, w.L_a, la, w.d, w.block_a)
        return torch.empty(max(1, n), dtype=torch.uint8, device="cuda")
    ws_mask = ws(sa.SA_CALL_BUILD_BLOCK_MASK, 1)
    ws_attn = ws(sa.SA_CALL_SPARSE_ATTENTION, 1)
    ws_tok = ws(sa.SA_CALL_TOKEN_ATTENTION, w.k_tok_a)

    def branch():
        sa.sa_saliency_ema(sal_bar, sal_a, 0.5)
        sa.sa_select_protected_tokens(sal_bar, w.k_tok_a, tok_idx=tok_idx, want_flag=False)
        sa.sa_build_block_mask(t["q_a"], t["k_a"], w.scale, w.block_a, w.k_keep_a, None,
                               kv_idx=kv_idx, kv_cnt=kv_cnt, ws=ws_mask)
        sa.sa_sparse_attention(t["q_a"], t["k_a"], v_a, w.scale, w.block_a, kv_idx, kv_cnt,
                               o=o, lse=lse, ws=ws_attn)
        sa.sa_protected_token_attention(t["q_a"], t["k_a"], v_a, w.scale, tok_idx, o, lse,
                                        ws=ws_tok)

    branch()
    torch.cuda.synchronize()
    outputs = [sal_bar, tok_idx, kv_idx, kv_cnt, o, lse]
    reference = [v.clone() for v in outputs]
    graph = _capture(branch)
    # the lagged update is in place: every replay starts from the same state
    _replays_match(graph, outputs, reference, reset=lambda: sal_bar.copy_(sal0))
