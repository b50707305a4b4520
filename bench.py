#!/usr/bin/env python3
"""Benchmark of one protected sparse video-attention layer on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input,
with every input already resident in HBM: cross-modal saliency (both
directions), protected block selection, the protected pooled-QK block mask
and block-sparse flash attention -- the four C-ABI calls, on one stream.

Printed (one JSON line): ``value`` = effective dense-equivalent TFLOP/s of
the layer (4*B*H*L_v^2*d / layer time), ``ms_per_step`` = ms per layer, a
per-call breakdown from HIP events, the roofline of the dominant kernel
(block-sparse attention, bf16 MFMA; against the published peak and against the
sustained MFMA rate measured on the device), the speedup over the same kernel
run with every list full, and the whole fp64 oracle layer timed on the
host.  ``token_protection`` reports the token-granular form of the
protection on the same inputs (protected tokens instead of protected query
blocks), ``cache_indicator`` the cache-reuse indicator on block outputs of
the same size (HBM-bound), and ``graph`` the layer and the audio branch
replayed from HIP graphs (the same kernels without host launch gaps).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
ATTN_KERNEL = "sparse_attn_bf16_kernel<128,128,false>"
ATTN_SOURCES = ("paper_2608_15522_amd/csrc/sa_attn.hip",
                "paper_2608_15522_amd/csrc/sa_device.h")
# Counter summaries per workload: profiles/<prefix>_layer_hbm_bytes.md.
TRAFFIC_FILES = {"ovi_bf16": "ovi", "ltx_bf16": "ltx", "long_cfg_bf16": "long_cfg"}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="ovi_bf16")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--dense-steps", type=int, default=5)
    p.add_argument("--calibrate-copy-mib", type=int, default=0,
                   help="run one device-to-device copy of this many MiB before "
                        "timing (a known-size reference for HBM byte counters)")
    p.add_argument("--no-mfma-probe", action="store_true",
                   help="skip the sustained-MFMA throughput probe")
    p.add_argument("--token-rho", type=float, default=0.05,
                   help="also time the token-granular protection (this fraction "
                        "of the video tokens protected; 0 = skip)")
    p.add_argument("--token-alpha", type=float, default=0.5,
                   help="lagged-saliency weight alpha of Eq. (4) in that run")
    p.add_argument("--no-cache-indicator", action="store_true",
                   help="skip timing the cache-reuse indicator")
    p.add_argument("--error-by-rank", action="store_true",
                   help="also report the attention error of vanilla, block-protected and "
                        "token-protected sparse attention against the dense run, by the "
                        "tokens' saliency rank")
    p.add_argument("--no-cross-attention", action="store_true",
                   help="skip timing the cross-modal attention forwards and the saliency "
                        "from their LSEs")
    p.add_argument("--layer", choices=("plain", "pooled"), default="plain",
                   help="the timed layer: the four calls of the boundary (plain), or the "
                        "same steps with the mask's block means pooled inside the saliency "
                        "streams (pooled)")
    p.add_argument("--no-pooled", action="store_true",
                   help="skip the layer with the block means pooled inside the saliency "
                        "streams")
    p.add_argument("--no-graph", action="store_true",
                   help="skip the graph-replay leg (the layer and the audio branch "
                        "captured into HIP graphs)")
    p.add_argument("--no-audio-branch", action="store_true",
                   help="skip timing the audio branch's protected sparse attention")
    p.add_argument("--sweep", default=None,
                   help="also run the density x protection sweep, one JSON "
                        "line per cell appended to this file")
    return p.parse_args()


def attention_traffic(workload):
    """Bytes past L2 per attention launch (FETCH_SIZE + WRITE_SIZE, each scaled
    by a same-run copy of known size) from the committed counter summary, or
    None when that summary was taken on another workload or on kernel sources
    other than the ones in this tree."""
    import hashlib
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    src = h.hexdigest()[:16]
    if workload not in TRAFFIC_FILES:
        return None, None
    path = "profiles/%s_layer_hbm_bytes.md" % TRAFFIC_FILES[workload]
    try:
        text = open(os.path.join(ROOT, path)).read()
    except OSError:
        return None, None
    for line in text.splitlines():
        if not line.startswith("traffic "):
            continue
        kv = dict(f.split("=", 1) for f in line.split()[1:])
        if (kv.get("kernel") == ATTN_KERNEL and kv.get("workload") == workload
                and kv.get("src") == src):
            return int(kv["fetch_bytes"]) + int(kv["write_bytes"]), path
    return None, None


def computed_flops(kv_idx, kv_cnt, L, block, d):
    """Exact attention flops over the kept (query block, key block) pairs,
    tails counted at their true length (4 * d per query-key pair)."""
    import numpy as np
    B, H, n_b = kv_cnt.shape
    lens = np.minimum((np.arange(n_b) + 1) * block, L) - np.arange(n_b) * block
    total = 0
    for b in range(B):
        for h in range(H):
            cnt = kv_cnt[b, h]
            for r in range(n_b):
                total += int(lens[r]) * int(lens[kv_idx[b, h, r, :cnt[r]]].sum())
    return 4 * d * total


def time_layer(plan, t, steps, warmup, torch, pooled=False):
    """The four calls of one layer, HIP events between them.  pooled: the
    layer with the mask's block means pooled inside the saliency streams."""
    run = plan.run_pooled if pooled else plan.run
    for _ in range(warmup):
        run(t["q_v"], t["k_v"], t["v_v"], t["q_a"], t["k_a"])
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        e = ev[i]
        e[0].record()
        if pooled:
            plan.cross_scores_pooled(t["q_a"], t["k_v"], t["q_v"], t["k_a"])
        else:
            plan.cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"])
        e[1].record()
        plan.select_protected()
        e[2].record()
        if pooled:
            plan.build_block_mask_pooled()
        else:
            plan.build_block_mask(t["q_v"], t["k_v"])
        e[3].record()
        plan.sparse_attention(t["q_v"], t["k_v"], t["v_v"])
        e[4].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    names = (["sa_cross_scores_pooled", "sa_select_protected", "sa_build_block_mask_pooled",
              "sa_sparse_attention"] if pooled else
             ["sa_cross_scores", "sa_select_protected", "sa_build_block_mask",
              "sa_sparse_attention"])
    per_call = {n: sum(ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(steps)) / steps
                for j, n in enumerate(names)}
    med = {n: sorted(ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(steps))[steps // 2]
           for j, n in enumerate(names)}
    return wall * 1e3 / steps, per_call, med


def time_pooled_layer(plan, t, steps, warmup, torch):
    """The layer with the mask's block means pooled inside the saliency
    streams (sa_cross_scores_pooled, select, sa_build_block_mask_pooled,
    attention) against the plain layer, the two alternating step by step so
    that clock drift under the power limit falls on both alike.  Returns
    (per-call median ms of the pooled layer, of the plain layer)."""
    args = (t["q_v"], t["k_v"], t["v_v"], t["q_a"], t["k_a"])
    for _ in range(warmup):
        plan.run_pooled(*args)
        plan.run(*args)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(10)] for _ in range(steps)]
    for i in range(steps):
        e = ev[i]
        e[0].record()
        plan.cross_scores_pooled(t["q_a"], t["k_v"], t["q_v"], t["k_a"])
        e[1].record()
        plan.select_protected()
        e[2].record()
        plan.build_block_mask_pooled()
        e[3].record()
        plan.sparse_attention(t["q_v"], t["k_v"], t["v_v"])
        e[4].record()
        plan.cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"])
        e[5].record()
        plan.select_protected()
        e[6].record()
        plan.build_block_mask(t["q_v"], t["k_v"])
        e[7].record()
        plan.sparse_attention(t["q_v"], t["k_v"], t["v_v"])
        e[8].record()
    torch.cuda.synchronize()

    def med(j0, names):
        return {n: sorted(ev[i][j0 + j].elapsed_time(ev[i][j0 + j + 1])
                          for i in range(steps))[steps // 2] for j, n in enumerate(names)}
    pooled = med(0, ["sa_cross_scores_pooled", "sa_select_protected",
                     "sa_build_block_mask_pooled", "sa_sparse_attention"])
    plain = med(4, ["sa_cross_scores", "sa_select_protected", "sa_build_block_mask",
                    "sa_sparse_attention"])
    return pooled, plain


def time_token_layer(plan, t, w, k_tok, alpha, steps, warmup, torch, sa):
    """The token-granular form of the protection on the same inputs, one
    saliency-refresh step: cross-modal saliency, the lagged-cache update
    (Eq. (4)), the protected tokens (Eq. (8) at token level), the block mask
    without block protection, block-sparse attention, and the dense rows of
    the protected tokens written over it (Eq. (11)).  Returns (ms per layer,
    per-call ms, kv_cnt, kv_idx) of the last step."""
    dev = t["q_v"].device
    sal_bar = torch.zeros(w.B, w.L_v, dtype=torch.float32, device=dev)
    tok_idx = torch.empty(w.B, k_tok, dtype=torch.int32, device=dev)
    kv_idx = torch.empty_like(plan.kv_idx)
    kv_cnt = torch.empty_like(plan.kv_cnt)
    o = torch.empty_like(t["q_v"])
    tok_ws = torch.empty(max(1, sa.sa_workspace_size(sa.SA_CALL_TOKEN_ATTENTION, w.B, w.H, w.L_v,
                                                     k_tok, w.d, 0)),
                         dtype=torch.uint8, device=dev)
    names = ["sa_cross_scores", "sa_saliency_ema", "sa_select_protected_tokens",
             "sa_build_block_mask", "sa_sparse_attention", "sa_protected_token_attention"]

    def step(e=None):
        rec = (lambda j: e[j].record()) if e else (lambda j: None)
        rec(0)
        plan.cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"])
        rec(1)
        sa.sa_saliency_ema(sal_bar, plan.sal_v_tok, alpha)
        rec(2)
        sa.sa_select_protected_tokens(sal_bar, k_tok, tok_idx=tok_idx, want_flag=False)
        rec(3)
        sa.sa_build_block_mask(t["q_v"], t["k_v"], plan.scale, plan.block, plan.k_keep,
                               None, kv_idx=kv_idx, kv_cnt=kv_cnt, ws=plan.ws)
        rec(4)
        sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], plan.scale, plan.block,
                               kv_idx, kv_cnt, o=o, ws=plan.ws)
        rec(5)
        sa.sa_protected_token_attention(t["q_v"], t["k_v"], t["v_v"], plan.scale,
                                        tok_idx, o, ws=tok_ws)
        rec(6)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(7)] for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        step(ev[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_call = {n: sum(ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(steps)) / steps
                for j, n in enumerate(names)}
    return wall * 1e3 / steps, per_call, kv_idx.cpu().numpy(), kv_cnt.cpu().numpy()


def make_audio_branch(plan, t, w, torch, sa):
    """The audio branch's protected sparse self-attention (Eq. (8)-(11),
    m = a) at the workload's audio shape, on the audio-token saliency of the
    layer's cross scores: lagged update, protected audio tokens, the audio
    block pattern, block-sparse attention and the dense rows.  V^a is drawn
    on the device.  Returns (step, call names, kv_idx, kv_cnt, k_tok), with
    step(e) recording event e[j] before call j when given."""
    dev = t["q_a"].device
    g = torch.Generator(device="cuda").manual_seed(1)
    v_a = torch.randn(t["q_a"].shape, device=dev, generator=g).to(t["q_a"].dtype)
    plan.cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"])
    sal_bar = plan.sal_a_tok.clone()
    n_b, k_tok = w.n_b_a, w.k_tok_a
    tok_idx = torch.empty(w.B, k_tok, dtype=torch.int32, device=dev)
    kv_idx = torch.empty(w.B, w.H, n_b, n_b, dtype=torch.int32, device=dev)
    kv_cnt = torch.empty(w.B, w.H, n_b, dtype=torch.int32, device=dev)
    o = torch.empty_like(t["q_a"])

    def ws(call, la):
        return torch.empty(max(1, sa.sa_workspace_size(call, w.B, w.H, w.L_a, la, w.d,
                                                       w.block_a)),
                           dtype=torch.uint8, device=dev)
    ws_mask = ws(sa.SA_CALL_BUILD_BLOCK_MASK, 1)
    ws_attn = ws(sa.SA_CALL_SPARSE_ATTENTION, 1)
    ws_tok = ws(sa.SA_CALL_TOKEN_ATTENTION, k_tok)
    names = ["sa_saliency_ema", "sa_select_protected_tokens", "sa_build_block_mask",
             "sa_sparse_attention", "sa_protected_token_attention"]

    def step(e=None):
        rec = (lambda j: e[j].record()) if e else (lambda j: None)
        rec(0)
        sa.sa_saliency_ema(sal_bar, plan.sal_a_tok, 0.5)
        rec(1)
        sa.sa_select_protected_tokens(sal_bar, k_tok, tok_idx=tok_idx, want_flag=False)
        rec(2)
        sa.sa_build_block_mask(t["q_a"], t["k_a"], plan.scale, w.block_a, w.k_keep_a, None,
                               kv_idx=kv_idx, kv_cnt=kv_cnt, ws=ws_mask)
        rec(3)
        sa.sa_sparse_attention(t["q_a"], t["k_a"], v_a, plan.scale, w.block_a, kv_idx,
                               kv_cnt, o=o, ws=ws_attn)
        rec(4)
        sa.sa_protected_token_attention(t["q_a"], t["k_a"], v_a, plan.scale, tok_idx, o,
                                        ws=ws_tok)
        rec(5)

    return step, names, kv_idx, kv_cnt, k_tok


def time_audio_branch(plan, t, w, steps, warmup, torch, sa):
    """Times the audio branch call by call (HIP events, host launch gaps
    included in the wall time).  Returns (ms per branch, per-call ms,
    computed flops)."""
    step, names, kv_idx, kv_cnt, k_tok = make_audio_branch(plan, t, w, torch, sa)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        step(ev[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_call = {n: sum(ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(steps)) / steps
                for j, n in enumerate(names)}
    flops = (computed_flops(kv_idx.cpu().numpy(), kv_cnt.cpu().numpy(), w.L_a, w.block_a, w.d)
             + 4.0 * w.d * k_tok * w.L_a * w.B * w.H)
    return wall * 1e3 / steps, per_call, flops


def time_graph(fn, steps, warmup, torch):
    """fn's kernels captured once into a HIP graph (torch.cuda.CUDAGraph) and
    replayed: (ms per replay from HIP events, ms per replay of wall time).
    The library allocates nothing and records no memory set, so the graph
    holds only its kernels."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(max(1, warmup)):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fn()
    torch.cuda.synchronize()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return e0.elapsed_time(e1) / steps, wall * 1e3 / steps


def error_by_rank(plan, t, w, x, di, dc, k_tok, torch, sa):
    """A synthetic analogue of the paper's Fig. 4: the error of vanilla
    sparse attention, block protection and token protection against the
    dense run (every list full), per video token, against the token's rank
    in the a->v saliency.  All outputs come from the library; the error of a
    token is ||O_x - O_dense||_2 averaged over heads, divided by the mean of
    ||O_dense||_2 over all (head, token) rows (one global scale: the dense
    rows of near-uniform attention have tiny norms, which makes per-row
    relative errors meaningless).  Returns the report dict."""
    B, H, L = w.B, w.H, w.L_v
    plan.cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"])
    sal = plan.sal_v_tok.clone()
    o_dense, _ = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], plan.scale, w.block,
                                        di, dc, ws=plan.ws)
    o_dense = o_dense.float()
    kv_idx, kv_cnt, _, _ = sa.sa_build_block_mask(t["q_v"], t["k_v"], plan.scale, w.block,
                                                  w.k_keep, None, ws=plan.ws)
    o_van, _ = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], plan.scale, w.block,
                                      kv_idx, kv_cnt, ws=plan.ws)
    tok_idx, tok_flag = sa.sa_select_protected_tokens(sal, k_tok)
    o_tok = o_van.clone()
    sa.sa_protected_token_attention(t["q_v"], t["k_v"], t["v_v"], plan.scale, tok_idx, o_tok)
    plan.select_protected()
    plan.build_block_mask(t["q_v"], t["k_v"])
    o_blk, _ = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], plan.scale, w.block,
                                      plan.kv_idx, plan.kv_cnt, ws=plan.ws)
    torch.cuda.synchronize()
    scale = float(o_dense.norm(dim=-1).mean())

    def err(o):
        return (o.float() - o_dense).norm(dim=-1).mean(dim=1) / scale  # [B, L]

    errs = {"vanilla": err(o_van), "block_protected": err(o_blk),
            "token_protected": err(o_tok)}
    rank = torch.argsort(torch.argsort(-sal, dim=1, stable=True), dim=1).float() / L
    edges = [0.0, 0.01, 0.05, 0.10, 0.25, 0.50, 1.0001]
    bins = []
    for lo, hi in zip(edges[:-1], edges[1:]):
        sel = (rank >= lo) & (rank < hi)
        bins.append({"rank_pct": f"{lo * 100:g}-{min(hi, 1.0) * 100:g}",
                     **{k: round(float(v[sel].mean()), 5) for k, v in errs.items()}})
    planted = torch.from_numpy(x["planted"]).cuda()
    return {"k_keep": w.k_keep, "k_prot_blocks": w.k_prot, "k_tok": k_tok,
            "metric": "per token: mean over heads of ||O - O_dense||_2, over the mean ||O_dense||_2",
            "by_saliency_rank": bins,
            "planted_tokens": {k: round(float(v[planted].mean()), 5) for k, v in errs.items()},
            "other_tokens": {k: round(float(v[~planted].mean()), 5) for k, v in errs.items()}}


def time_cross_attention(plan, t, w, steps, warmup, torch, sa):
    """The two cross-modal attention forwards (a->v: Q^a over K^v, V^v; v->a:
    Q^v over K^a, V^a) with their row LSEs, then the saliency of both
    directions from those LSEs (sa_cross_scores_from_lse), against the
    standalone saliency call.  V^a is drawn on the device.  Returns the
    report dict."""
    dev = t["q_a"].device
    g = torch.Generator(device="cuda").manual_seed(2)
    v_a = torch.randn(t["k_a"].shape, device=dev, generator=g).to(t["k_a"].dtype)
    B, H, L_v, L_a, d = w.B, w.H, w.L_v, w.L_a, w.d
    o_a = torch.empty_like(t["q_a"])
    o_v = torch.empty_like(t["q_v"])
    lse_a = torch.empty(B, H, L_a, dtype=torch.float32, device=dev)
    lse_v = torch.empty(B, H, L_v, dtype=torch.float32, device=dev)

    def ws(Lq, Lk):
        return torch.empty(max(1, sa.sa_workspace_size(sa.SA_CALL_CROSS_ATTENTION, B, H, Lq, Lk,
                                                       d, 0)), dtype=torch.uint8, device=dev)
    ws_a, ws_v = ws(L_a, L_v), ws(L_v, L_a)
    names = ["a2v_forward", "v2a_forward", "sa_cross_scores_from_lse", "sa_cross_scores",
             "sa_build_block_mask", "sa_cross_scores_pooled_from_lse",
             "sa_build_block_mask_pooled"]

    def step(e=None):
        rec = (lambda j: e[j].record()) if e else (lambda j: None)
        rec(0)
        sa.sa_cross_attention(t["q_a"], t["k_v"], t["v_v"], plan.scale, o=o_a, lse=lse_a,
                              ws=ws_a)
        rec(1)
        sa.sa_cross_attention(t["q_v"], t["k_a"], v_a, plan.scale, o=o_v, lse=lse_v, ws=ws_v)
        rec(2)
        sa.sa_cross_scores_from_lse(t["q_a"], t["k_v"], t["q_v"], t["k_a"], lse_a, lse_v,
                                    plan.scale, w.block, sal_v_tok=plan.sal_v_tok,
                                    sal_v_blk=plan.sal_v_blk, sal_a_tok=plan.sal_a_tok,
                                    ws=plan.ws)
        rec(3)
        plan.cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"])
        rec(4)
        plan.build_block_mask(t["q_v"], t["k_v"])
        rec(5)
        plan.cross_scores_pooled(t["q_a"], t["k_v"], t["q_v"], t["k_a"], lse_a=lse_a,
                                 lse_v=lse_v)
        rec(6)
        plan.build_block_mask_pooled()
        rec(7)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(8)] for _ in range(steps)]
    for i in range(steps):
        step(ev[i])
    torch.cuda.synchronize()
    ms = {n: sum(ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(steps)) / steps
          for j, n in enumerate(names)}
    flops = 4.0 * B * H * L_a * L_v * d  # each direction
    fwd_ms = ms["a2v_forward"] + ms["v2a_forward"]
    return {"per_call_ms": {k: round(v, 4) for k, v in ms.items()},
            "forward_tflop_each": round(flops / 1e12, 4),
            "a2v_forward_tflops": round(flops / (ms["a2v_forward"] * 1e-3) / 1e12, 1),
            "v2a_forward_tflops": round(flops / (ms["v2a_forward"] * 1e-3) / 1e12, 1),
            "forwards_plus_saliency_ms": round(fwd_ms + ms["sa_cross_scores_from_lse"], 4),
            "forwards_plus_standalone_saliency_ms": round(fwd_ms + ms["sa_cross_scores"], 4),
            # steps 1-2 on top of the forwards: saliency from their LSEs and the
            # block mask, with the mask call pooling Q^v, K^v itself, or with the
            # means pooled inside the saliency streams
            "saliency_plus_mask_ms": round(ms["sa_cross_scores_from_lse"]
                                           + ms["sa_build_block_mask"], 4),
            "saliency_plus_mask_pooled_ms": round(ms["sa_cross_scores_pooled_from_lse"]
                                                  + ms["sa_build_block_mask_pooled"], 4)}


def time_cache_indicator(w, steps, torch, sa):
    """The cache-reuse indicator (Eq. (12)-(15)) on block outputs of the
    workload's size (C = H*d channels per token, its dtype): current and
    cached video and audio outputs, 5 % protected token rows, both saliency
    maps.  Returns (ms per call, algorithmic bytes)."""
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    C = w.H * w.d
    g = torch.Generator(device="cuda").manual_seed(0)
    yv = torch.randn(w.B, w.L_v, C, device="cuda", generator=g).to(dt)
    yvh = torch.randn(w.B, w.L_v, C, device="cuda", generator=g).to(dt)
    ya = torch.randn(w.B, w.L_a, C, device="cuda", generator=g).to(dt)
    yah = torch.randn(w.B, w.L_a, C, device="cuda", generator=g).to(dt)
    flag = (torch.rand(w.B, w.L_v, device="cuda", generator=g) < 0.05).to(torch.uint8)
    sb = torch.rand(w.B, w.L_v, device="cuda", generator=g)
    sh = torch.rand(w.B, w.L_v, device="cuda", generator=g)
    out = torch.empty(6, dtype=torch.float32, device="cuda")
    call = lambda: sa.sa_cache_indicator(yv, yvh, prot_flag=flag, y_a=ya, y_a_hat=yah,
                                         s_bar=sb, s_hat=sh, out=out)
    call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    es = yv.element_size()
    nbytes = (2 * w.B * w.L_v * C + 2 * w.B * w.L_a * C) * es + w.B * w.L_v * (1 + 2 * 4)
    del yv, yvh, ya, yah
    torch.cuda.empty_cache()
    return e0.elapsed_time(e1) / steps, nbytes


def time_attention(plan, t, kv_idx, kv_cnt, steps, torch, sa):
    sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], plan.scale, plan.block,
                           kv_idx, kv_cnt, o=plan.o, ws=plan.ws)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], plan.scale, plan.block,
                               kv_idx, kv_cnt, o=plan.o, ws=plan.ws)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


# Inputs of the CPU baseline, set before the worker pool is forked so that the
# workers share them (copy-on-write) and never hold any GPU state.
_CPU_X = None


def _cpu_pool_init():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)  # one BLAS thread per worker
    except Exception:  # pragma: no cover
        pass


def _cpu_head(task):
    """The oracle's steps for one (b, h) slab of the layer: the a->v and v->a
    saliency of that head, its pooled-QK block mask and its sparse attention
    on the GPU's lists.  Returns the seconds it took."""
    import numpy as np
    import oracle
    b, h, scale, block, k_keep, n_b, kv_idx_bh, kv_cnt_bh = task
    x = _CPU_X
    sl = lambda k: x[k][b:b + 1, h:h + 1]
    t0 = time.perf_counter()
    oracle.cross_scores(sl("q_a"), sl("k_v"), scale, sl("q_v"), sl("k_a"))
    oracle.block_mask(sl("q_v"), sl("k_v"), scale, block, k_keep,
                      np.zeros((1, n_b), dtype=np.uint8))
    oracle.masked_attention(sl("q_v"), sl("k_v"), sl("v_v"), scale, block,
                            kv_idx_bh[None, None], kv_cnt_bh[None, None])
    return time.perf_counter() - t0


def cpu_workers():
    """Worker count: the CPUs this process may run on, at most 16 (the host
    share of one GPU)."""
    return max(1, min(len(os.sched_getaffinity(0)), 16))


def make_cpu_pool(x):
    """Fork the worker pool of the CPU baseline; called before torch touches
    the GPU."""
    import multiprocessing as mp
    global _CPU_X
    _CPU_X = x
    return mp.get_context("fork").Pool(cpu_workers(), initializer=_cpu_pool_init)


def cpu_baseline(w, pool, kv_idx, kv_cnt):
    """The oracle as it stands, timed on the whole layer: every (b, h) slab on
    a pool of worker processes with one BLAS thread each.  Returns the dict
    of the report."""
    import numpy as np
    tasks = [(b, h, w.scale, w.block, w.k_keep, w.n_b, np.ascontiguousarray(kv_idx[b, h]),
              np.ascontiguousarray(kv_cnt[b, h])) for b in range(w.B) for h in range(w.H)]
    t0 = time.perf_counter()
    per_head = pool.map(_cpu_head, tasks, chunksize=1)
    layer_s = time.perf_counter() - t0
    dense = 4.0 * w.B * w.H * w.L_v ** 2 * w.d
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in fh
                              if ln.startswith("model name")), cpu_model)
    except OSError:  # pragma: no cover
        pass
    return {"value": round(dense / layer_s / 1e12, 6), "unit": "TFLOP/s",
            "cores": cpu_workers(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "kind": "oracle", "cpu_model": cpu_model, "numpy": np.__version__,
            "ms_per_layer": round(layer_s * 1e3, 1),
            "cpu_seconds": round(float(sum(per_head)), 1),
            "sample": (f"the whole {w.name} layer: {w.B * w.H} (b, h) slabs, each the "
                       f"saliency in both directions, the pooled-QK block mask and the "
                       f"sparse attention on the GPU's lists, on {cpu_workers()} worker "
                       f"processes with one BLAS thread each")}


def run_sweep(path, steps, torch, sa, synth, LayerPlan):
    """Density x protection sweep at the Ovi-like shape: attention-kernel time
    of each cell against the same kernel with every list full."""
    base = synth.WORKLOADS["ovi_bf16"]
    with open(path, "a") as f:
        for seed in (0, 1, 2):
            x = synth.make_inputs(base.with_(seed=seed))
            t = {k: torch.from_numpy(x[k]).to(torch.bfloat16).cuda()
                 for k in ("q_v", "k_v", "v_v", "q_a", "k_a")}
            del x
            dense_ms = None
            for w in [s for s in synth.sweep_workloads() if s.seed == seed]:
                plan = LayerPlan(w.B, w.H, w.L_v, w.L_a, w.d, w.block, w.k_keep,
                                 w.k_prot, w.scale)
                plan.run(t["q_v"], t["k_v"], t["v_v"], t["q_a"], t["k_a"])
                ms = time_attention(plan, t, plan.kv_idx, plan.kv_cnt, steps, torch, sa)
                if dense_ms is None:
                    n_b = w.n_b
                    di = torch.arange(n_b, dtype=torch.int32, device="cuda").expand(
                        w.B, w.H, n_b, n_b).contiguous()
                    dc = torch.full((w.B, w.H, n_b), n_b, dtype=torch.int32, device="cuda")
                    dense_ms = time_attention(plan, t, di, dc, steps, torch, sa)
                cnt = plan.kv_cnt.cpu().numpy()
                frac = float(cnt.sum()) / (w.B * w.H * w.n_b * w.n_b)
                rec = {"cell": w.name, "density": w.density, "rho": w.rho, "seed": seed,
                       "k_keep": w.k_keep, "k_prot": w.k_prot, "block_fraction": frac,
                       "attn_ms": ms, "dense_attn_ms": dense_ms,
                       "speedup_vs_dense": dense_ms / ms, "ideal_1_over_f": 1.0 / frac}
                f.write(json.dumps(rec) + "\n")
                f.flush()
                print(json.dumps(rec), file=sys.stderr, flush=True)
                del plan
            del t
            torch.cuda.empty_cache()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the "
              "method's path is measured on one GPU's share at full shape.",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import synth

    w = synth.WORKLOADS[args.workload]
    print(f"bench: {w.name} B={w.B} H={w.H} L_v={w.L_v} L_a={w.L_a} d={w.d} "
          f"block={w.block} k_keep={w.k_keep} k_prot={w.k_prot}", file=sys.stderr,
          flush=True)
    x = synth.make_inputs(w)
    # the oracle's worker pool is forked before the GPU is initialised
    pool = None if args.no_cpu_baseline else make_cpu_pool(x)
    import torch
    import paper_2608_15522_amd as sa
    from paper_2608_15522_amd.layer import LayerPlan
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    t = {k: torch.from_numpy(x[k]).to(dt).cuda() for k in ("q_v", "k_v", "v_v", "q_a", "k_a")}
    plan = LayerPlan(w.B, w.H, w.L_v, w.L_a, w.d, w.block, w.k_keep, w.k_prot, w.scale,
                     dtype=dt)
    if args.calibrate_copy_mib > 0:
        nbytes = args.calibrate_copy_mib << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    ms_layer, per_call, per_call_median = time_layer(plan, t, args.steps, args.warmup, torch,
                                                     pooled=args.layer == "pooled")
    print(f"bench: layer {ms_layer:.3f} ms {per_call}", file=sys.stderr, flush=True)

    kv_idx = plan.kv_idx.cpu().numpy()
    kv_cnt = plan.kv_cnt.cpu().numpy()
    flops_attn = computed_flops(kv_idx, kv_cnt, w.L_v, w.block, w.d)
    dense_flops = 4.0 * w.B * w.H * w.L_v ** 2 * w.d
    n_b = w.n_b
    di = torch.arange(n_b, dtype=torch.int32, device="cuda").expand(w.B, w.H, n_b, n_b).contiguous()
    dc = torch.full((w.B, w.H, n_b), n_b, dtype=torch.int32, device="cuda")
    dense_ms = (time_attention(plan, t, di, dc, args.dense_steps, torch, sa)
                if args.dense_steps > 0 else None)
    attn_ms = per_call["sa_sparse_attention"]
    achieved = flops_attn / (attn_ms * 1e-3) / 1e12
    traffic, traffic_src = attention_traffic(w.name)
    res = {
        "metric": "ms/layer + effective TFLOP/s of protected sparse video attention (1 MI355X)",
        "value": round(dense_flops / (ms_layer * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_layer, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded Gaussian Q/K/V with planted audio-correlated video blocks)",
        "config": {"workload": w.name, "layer": args.layer, "B": w.B, "H": w.H, "L_v": w.L_v, "L_a": w.L_a,
                   "d": w.d, "block": w.block, "density": w.density, "k_keep": w.k_keep,
                   "k_prot": w.k_prot, "n_b": n_b},
        "per_call_ms": {k: round(v, 4) for k, v in per_call.items()},
        "per_call_median_ms": {k: round(v, 4) for k, v in per_call_median.items()},
        "attention": {
            "computed_tflop": round(flops_attn / 1e12, 4),
            "dense_tflop": round(dense_flops / 1e12, 4),
            "block_fraction": round(float(kv_cnt.sum()) / (w.B * w.H * n_b * n_b), 5),
            "ms": round(attn_ms, 4),
            "effective_dense_tflops": round(dense_flops / (attn_ms * 1e-3) / 1e12, 2),
            "dense_run_ms": round(dense_ms, 4) if dense_ms else None,
            "speedup_vs_dense_run": round(dense_ms / attn_ms, 3) if dense_ms else None,
        },
        "roofline": {"bound": "mfma", "kernel": ATTN_KERNEL,
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic, "traffic_unit": "bytes/launch",
                     "traffic_src": traffic_src,
                     "algorithmic_bytes": 4 * w.B * w.H * w.L_v * w.d * (2 if w.dtype == "bf16" else 4)},
    }
    if not args.no_mfma_probe:
        # The matrix cores' sustained rate on this device, with changing random
        # bf16 operands (the attention kernel's case) and with zero operands:
        # MFMA power, and with it the clock, depends on the operand bits.
        from paper_2608_15522_amd.binding import sa_bench_mfma_peak
        rnd_tf, rnd_ghz = sa_bench_mfma_peak(True)
        zero_tf, zero_ghz = sa_bench_mfma_peak(False)
        res["roofline"]["measured_peak"] = {
            "probe": "v_mfma_f32_32x32x16_bf16, 4 chains/wave, 4096 waves",
            "random_operands_tflops": round(rnd_tf, 1), "random_operands_ghz": round(rnd_ghz, 2),
            "zero_operands_tflops": round(zero_tf, 1), "zero_operands_ghz": round(zero_ghz, 2),
            "frac_of_random_operands": round(achieved / rnd_tf, 4)}
    if not args.no_pooled:
        pc_p, pc_0 = time_pooled_layer(plan, t, args.steps, args.warmup, torch)
        print(f"bench: pooled layer {pc_p}, plain layer {pc_0}", file=sys.stderr, flush=True)
        res["pooled_layer"] = {
            "timing": "medians, pooled and plain layers alternating step by step",
            "per_call_median_ms": {k: round(v, 4) for k, v in pc_p.items()},
            "plain_per_call_median_ms": {k: round(v, 4) for k, v in pc_0.items()},
            "layer_ms": round(sum(pc_p.values()), 4),
            "plain_layer_ms": round(sum(pc_0.values()), 4),
            "steps_1_2_ms": round(pc_p["sa_cross_scores_pooled"]
                                  + pc_p["sa_build_block_mask_pooled"], 4),
            "plain_steps_1_2_ms": round(pc_0["sa_cross_scores"]
                                        + pc_0["sa_build_block_mask"], 4)}
    if args.token_rho > 0:
        k_tok = synth.budget(args.token_rho, w.L_v)
        ms_tok, pc_tok, kvi_tok, kvc_tok = time_token_layer(
            plan, t, w, k_tok, args.token_alpha, args.steps, args.warmup, torch, sa)
        rows_flops = 4.0 * w.d * k_tok * w.L_v * w.B * w.H
        rows_ms = pc_tok["sa_protected_token_attention"]
        rows_tf = rows_flops / (rows_ms * 1e-3) / 1e12
        print(f"bench: token layer {ms_tok:.3f} ms {pc_tok}", file=sys.stderr, flush=True)
        res["token_protection"] = {
            "rho": args.token_rho, "k_tok": k_tok, "alpha": args.token_alpha,
            "ms_per_layer": round(ms_tok, 4),
            "value": round(dense_flops / (ms_tok * 1e-3) / 1e12, 3),
            "per_call_ms": {k: round(v, 4) for k, v in pc_tok.items()},
            "sparse_tflop": round(computed_flops(kvi_tok, kvc_tok, w.L_v, w.block, w.d) / 1e12, 4),
            "dense_rows_tflop": round(rows_flops / 1e12, 4),
            "dense_rows_kernels": "sparse_attn_bf16_kernel<128,128,true> + token_combine_kernel<128>",
            "dense_rows_tflops": round(rows_tf, 2),
            "dense_rows_frac_of_peak": round(rows_tf / PEAK_BF16_TFLOPS, 4)}
    if args.error_by_rank:
        res["error_by_rank"] = error_by_rank(plan, t, w, x, di, dc, synth.budget(w.rho, w.L_v),
                                             torch, sa)
    if not args.no_cross_attention:
        res["cross_attention"] = time_cross_attention(plan, t, w, args.steps, args.warmup,
                                                      torch, sa)
    if not args.no_audio_branch:
        ms_a, pc_a, flops_a = time_audio_branch(plan, t, w, args.steps, args.warmup, torch, sa)
        dense_a = 4.0 * w.B * w.H * w.L_a ** 2 * w.d
        res["audio_branch"] = {
            "L_a": w.L_a, "block_a": w.block_a, "k_keep_a": w.k_keep_a, "k_tok_a": w.k_tok_a,
            "ms": round(ms_a, 4), "per_call_ms": {k: round(v, 4) for k, v in pc_a.items()},
            "computed_tflop": round(flops_a / 1e12, 5),
            "effective_dense_tflops": round(dense_a / (ms_a * 1e-3) / 1e12, 2)}
    if not args.no_graph:
        # the same calls replayed from HIP graphs: no host launch gaps
        def layer():
            plan.run(t["q_v"], t["k_v"], t["v_v"], t["q_a"], t["k_a"])
        g_ms, g_wall = time_graph(layer, args.steps, args.warmup, torch)
        res["graph"] = {"layer_ms": round(g_ms, 4), "layer_wall_ms": round(g_wall, 4),
                        "layer_value": round(dense_flops / (g_ms * 1e-3) / 1e12, 3)}
        if not args.no_audio_branch:
            step_a = make_audio_branch(plan, t, w, torch, sa)[0]
            a_ms, a_wall = time_graph(step_a, args.steps, args.warmup, torch)
            res["graph"].update({"audio_branch_ms": round(a_ms, 4),
                                 "audio_branch_wall_ms": round(a_wall, 4)})
    if not args.no_cache_indicator:
        ci_ms, ci_bytes = time_cache_indicator(w, args.steps, torch, sa)
        ci_gbs = ci_bytes / (ci_ms * 1e-3) / 1e9
        res["cache_indicator"] = {
            "ms": round(ci_ms, 4), "channels": w.H * w.d, "bytes": ci_bytes,
            "bound": "hbm", "achieved_gbs": round(ci_gbs, 1), "peak_gbs": PEAK_HBM_GBS,
            "frac": round(ci_gbs / PEAK_HBM_GBS, 4)}
    if args.sweep:
        run_sweep(args.sweep, max(3, args.dense_steps), torch, sa, synth, LayerPlan)
    if not args.no_cpu_baseline:
        del t
        torch.cuda.empty_cache()
        res["cpu_baseline"] = cpu_baseline(w, pool, kv_idx, kv_cnt)
        pool.close()
        pool.join()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
