"""sa_sparse_attention_noalloc through the C ABI: the same outputs as
sa_sparse_attention (bitwise: the same kernels run), on two calls in a row
that share the library's scratch, the second with a smaller input, and
within the attention tolerance of the oracle on the small one."""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import TOL_LSE, TOL_O, to_dev

pytestmark = pytest.mark.gpu


def lists_and_inputs(B, H, L, block, k_keep, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    q, k, v = (torch.randn(B, H, L, 128, device="cuda", generator=g).to(torch.bfloat16)
               for _ in range(3))
    n_b = -(-L // block)
    prot = (torch.rand(B, n_b, device="cuda", generator=g) < 0.1).to(torch.uint8)
    kv_idx, kv_cnt, _, _ = sa.sa_build_block_mask(q, k, 128 ** -0.5, block, k_keep, prot)
    return q, k, v, kv_idx, kv_cnt


def test_noalloc_matches_the_workspace_call_on_two_calls():
    scale = float(np.float32(128 ** -0.5))
    # first the Ovi-like shape (24 heads, 256 key blocks, 120-key tail), then a
    # smaller one on the same scratch
    for (B, H, L, block, k_keep) in ((1, 24, 32760, 128, 64), (2, 3, 1000, 64, 3)):
        print(f"case noalloc B={B} H={H} L={L} block={block} k_keep={k_keep}", flush=True)
        q, k, v, kv_idx, kv_cnt = lists_and_inputs(B, H, L, block, k_keep, seed=L)
        o_ref, lse_ref = sa.sa_sparse_attention(q, k, v, scale, block, kv_idx, kv_cnt,
                                                want_lse=True)
        o = torch.full_like(q, float("nan"))
        lse = torch.full((B, H, L), float("nan"), device="cuda")
        sa.sa_sparse_attention_noalloc(q, k, v, scale, block, kv_idx, kv_cnt, o, lse)
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
        assert torch.equal(lse, lse_ref)
        if L <= 1000:
            O_or, lse_or = oracle.masked_attention(
                q.float().cpu().numpy(), k.float().cpu().numpy(), v.float().cpu().numpy(),
                scale, block, kv_idx.cpu().numpy(), kv_cnt.cpu().numpy())
            assert float(np.abs(o.float().cpu().numpy() - O_or).max()) <= TOL_O["bf16"]
            assert float(np.abs(lse.cpu().numpy() - lse_or).max()) <= TOL_LSE["bf16"]
        del q, k, v, o, o_ref


def test_noalloc_fp32_path():
    w = synth.WORKLOADS["tiny_f32"]
    x = synth.make_inputs(w)
    t = {kk: to_dev(x[kk], "f32") for kk in ("q_v", "k_v", "v_v")}
    kv_idx, kv_cnt, _, _ = sa.sa_build_block_mask(t["q_v"], t["k_v"], w.scale, w.block,
                                                  w.k_keep, None)
    o_ref, lse_ref = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, w.block,
                                            kv_idx, kv_cnt, want_lse=True)
    o = torch.empty_like(o_ref)
    lse = torch.empty_like(lse_ref)
    sa.sa_sparse_attention_noalloc(t["q_v"], t["k_v"], t["v_v"], w.scale, w.block, kv_idx,
                                   kv_cnt, o, lse)
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref)
