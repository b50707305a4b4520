"""GPU parity of the four C-ABI calls against the fp64 oracle, on seeded
synthetic inputs.  Small shapes span several tiles and ragged tails and are
compared element by element; edge cases use hand-built lists."""
import functools

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_15522_amd as sa
from sa_parity import (TOL_LSE, TOL_O, check_kv_lists, compare_layer, gpu_layer,
                       logit_ramp_inputs, to_dev)

pytestmark = pytest.mark.gpu

BASE = synth.WORKLOADS["ovi_bf16"]

# (name, workload overrides, k_keep, k_prot)
SMALL = [
    ("tiny_f32", synth.WORKLOADS["tiny_f32"], None, None),
    ("bf16_d128_b128_tail104_La200",
     BASE.with_(name="a", B=2, H=3, frames=10, rows=10, cols=10, L_a=200, n_plant=2), 2, 2),
    ("bf16_d128_b128_tail26",
     BASE.with_(name="b", H=2, frames=7, rows=10, cols=15, L_a=64, n_plant=1), 3, 1),
    ("bf16_d64_b64_tail60",
     BASE.with_(name="c", H=3, d=64, block=64, frames=7, rows=10, cols=10, L_a=130,
                n_plant=2), 3, 2),
    ("bf16_d128_b64_noprot",
     BASE.with_(name="d", H=2, block=64, frames=4, rows=10, cols=16, L_a=33, n_plant=2), 4, 0),
    ("bf16_d64_b128_allprot_La520",
     BASE.with_(name="e", B=2, H=1, d=64, frames=3, rows=10, cols=13, L_a=520, n_plant=1), 1, 4),
    ("bf16_single_block",
     BASE.with_(name="f", H=1, frames=7, rows=11, cols=1, L_a=5, n_plant=0), 1, 0),
    ("bf16_d128_La1100_three_slabs",
     BASE.with_(name="h", H=2, frames=3, rows=10, cols=14, L_a=1100, n_plant=1), 2, 1),
    ("f32_d128_b128",
     synth.WORKLOADS["tiny_f32"].with_(name="g", d=128, block=128, frames=5, rows=10,
                                       cols=20, L_a=70, n_plant=2), 2, 1),
    # B*H a multiple of 8: the attention launch places whole heads on XCDs
    # (the branch the full-size layers take); d 128, block 128, ragged tails
    ("bf16_d128_b128_BH8_tail10",
     BASE.with_(name="i", H=8, frames=5, rows=10, cols=77, L_a=96, n_plant=3), 7, 3),
    ("bf16_d128_b128_BH16_tail56",
     BASE.with_(name="j", B=2, H=8, frames=3, rows=12, cols=62, L_a=64, n_plant=2), 5, 2),
]


@pytest.mark.parametrize("name,w,k_keep,k_prot", SMALL, ids=[s[0] for s in SMALL])
def test_layer_parity_small(name, w, k_keep, k_prot):
    k_keep = w.k_keep if k_keep is None else k_keep
    k_prot = w.k_prot if k_prot is None else k_prot
    print(f"case {name}: B={w.B} H={w.H} d={w.d} L_v={w.L_v} L_a={w.L_a} "
          f"block={w.block} k_keep={k_keep} k_prot={k_prot}", flush=True)
    x = synth.make_inputs(w)
    g = gpu_layer(x, w, k_keep, k_prot)
    rep = compare_layer(x, w, g, k_keep, k_prot)
    print(name, rep, flush=True)


def test_no_audio_direction_skips_sal_a():
    w = SMALL[1][1]
    x = synth.make_inputs(w)
    g = gpu_layer(x, w, 2, 2, with_audio=False)
    assert g["sal_a_tok"] is None
    compare_layer(x, w, g, 2, 2, with_audio=False)


def _hand_lists(n_b, B, H, seed):
    rng = np.random.default_rng(seed)
    mask = rng.random((B, H, n_b, n_b)) < 0.35
    mask[..., 0] = True
    kv_idx, kv_cnt = oracle.kv_lists_from_mask(mask.astype(np.uint8))
    return kv_idx.astype(np.int32), kv_cnt.astype(np.int32)


@pytest.mark.parametrize("dtype,d,block", [("bf16", 128, 128), ("bf16", 64, 64),
                                           ("f32", 64, 64)])
def test_empty_and_invalid_list_entries(dtype, d, block):
    """kv_cnt = 0 gives zeros and lse = -inf; entries outside [0, n_b) and
    counts above n_b are ignored / clamped."""
    w = BASE.with_(name="h", H=2, d=d, block=block, frames=5, rows=10, cols=13,
                   dtype=dtype, n_plant=0)
    x = synth.make_inputs(w)
    n_b = w.n_b
    kv_idx, kv_cnt = _hand_lists(n_b, 1, 2, 3)
    kv_cnt[0, 0, 1] = 0
    kv_cnt[0, 1, 2] = 0
    # row (0,0,3): two bad entries after a valid list of two
    c = 2
    kv_idx[0, 0, 3, :] = -1
    kv_idx[0, 0, 3, :c + 2] = [0, 2, -5, n_b + 7]
    kv_cnt[0, 0, 3] = c + 2
    kv_cnt[0, 1, 4] = n_b + 100        # clamped to n_b (full row of -1 tails)
    t = {k: to_dev(x[k], dtype) for k in ("q_v", "k_v", "v_v")}
    o, lse = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, block,
                                    torch.from_numpy(kv_idx).cuda(),
                                    torch.from_numpy(kv_cnt).cuda(), want_lse=True)
    o = o.float().cpu().numpy()
    lse = lse.cpu().numpy()
    # the oracle's view of the same lists with the invalid entries dropped
    ref_idx = kv_idx.astype(np.int64).copy()
    ref_cnt = np.minimum(kv_cnt, n_b).astype(np.int64)
    ref_idx[0, 0, 3, c:c + 2] = -1
    ref_cnt[0, 0, 3] = c
    valid = ref_idx[0, 1, 4][(ref_idx[0, 1, 4] >= 0)]
    ref_cnt[0, 1, 4] = valid.size
    O_ref, lse_ref = oracle.masked_attention(x["q_v"], x["k_v"], x["v_v"], w.scale,
                                             block, ref_idx, ref_cnt)
    assert np.abs(o - O_ref).max() <= TOL_O[dtype]
    for (h, r) in ((0, 1), (1, 2)):
        sl = slice(r * block, (r + 1) * block)
        assert np.all(o[0, h, sl] == 0.0)
        assert np.all(np.isneginf(lse[0, h, sl]))
    fin = np.isfinite(lse_ref)
    assert np.abs(lse[fin] - lse_ref[fin]).max() <= TOL_LSE[dtype]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_masked_blocks_contribute_exactly_zero(dtype):
    """A key block in no list is NaN-poisoned in K and V: the output is
    bit-identical to the run on clean data."""
    w = BASE.with_(name="i", H=2, d=64, block=64, frames=4, rows=10, cols=16,
                   dtype=dtype, n_plant=0)
    x = synth.make_inputs(w)
    n_b = w.n_b
    kv_idx, kv_cnt = _hand_lists(n_b, 1, 2, 5)
    poisoned = 3
    mask = np.zeros((1, 2, n_b, n_b), dtype=np.uint8)
    for h in range(2):
        for r in range(n_b):
            mask[0, h, r, kv_idx[0, h, r, :kv_cnt[0, h, r]]] = 1
    mask[..., poisoned] = 0
    kv_idx, kv_cnt = (a.astype(np.int32) for a in oracle.kv_lists_from_mask(mask))
    di, dc = torch.from_numpy(kv_idx).cuda(), torch.from_numpy(kv_cnt).cuda()
    t = {k: to_dev(x[k], dtype) for k in ("q_v", "k_v", "v_v")}
    o_clean, _ = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, 64, di, dc)
    sl = slice(poisoned * 64, (poisoned + 1) * 64)
    t["k_v"][:, :, sl] = float("nan")
    t["v_v"][:, :, sl] = float("nan")
    o_pois, _ = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, 64, di, dc)
    assert torch.equal(o_clean, o_pois)
    assert torch.isfinite(o_pois.float()).all()


@pytest.mark.parametrize("dtype,d,block", [("bf16", 128, 128), ("f32", 64, 64)])
def test_dense_lists_match_dense_attention(dtype, d, block):
    w = BASE.with_(name="j", H=2, d=d, block=block, frames=3, rows=10, cols=29,
                   dtype=dtype, n_plant=0)
    x = synth.make_inputs(w)
    n_b = w.n_b
    kv_idx = np.tile(np.arange(n_b, dtype=np.int32), (1, 2, n_b, 1))
    kv_cnt = np.full((1, 2, n_b), n_b, dtype=np.int32)
    t = {k: to_dev(x[k], dtype) for k in ("q_v", "k_v", "v_v")}
    o, lse = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale, block,
                                    torch.from_numpy(kv_idx).cuda(),
                                    torch.from_numpy(kv_cnt).cuda(), want_lse=True)
    O_ref, lse_ref = oracle.dense_attention(x["q_v"], x["k_v"], x["v_v"], w.scale)
    assert np.abs(o.float().cpu().numpy() - O_ref).max() <= TOL_O[dtype]
    assert np.abs(lse.cpu().numpy() - lse_ref).max() <= TOL_LSE[dtype]


@pytest.mark.parametrize("profile", ["grow", "fall", "jump"])
@pytest.mark.parametrize("dtype,d,block", [("bf16", 128, 128), ("bf16", 64, 64),
                                           ("f32", 64, 64)])
def test_running_max_under_large_logit_changes(profile, dtype, d, block):
    """Logits that rise by ~98 log2 units along the keys (the running max is
    raised many times, in the steady-state loop and in the tail tiles), fall
    by as much (later tiles underflow), or jump by ~146 log2 units in the last
    50 keys (exp2 would overflow fp32 without raising the max first), against
    dense fp64 attention."""
    L, H = 2000, 2
    scale = float(np.float32(1.0 / np.sqrt(d)))
    q, k, v = logit_ramp_inputs(L, L, d, H, profile, dtype)
    print(f"case ramp {profile} {dtype} d={d} block={block} L={L}", flush=True)
    n_b = -(-L // block)
    kv_idx = np.tile(np.arange(n_b, dtype=np.int32), (1, H, n_b, 1))
    kv_cnt = np.full((1, H, n_b), n_b, dtype=np.int32)
    o, lse = sa.sa_sparse_attention(to_dev(q, dtype), to_dev(k, dtype), to_dev(v, dtype),
                                    scale, block, torch.from_numpy(kv_idx).cuda(),
                                    torch.from_numpy(kv_cnt).cuda(), want_lse=True)
    O_ref, lse_ref = oracle.dense_attention(q, k, v, scale)
    o = o.float().cpu().numpy()
    assert np.all(np.isfinite(o))
    o_err = float(np.abs(o - O_ref).max())
    l_err = float(np.abs(lse.cpu().numpy() - lse_ref).max())
    # fp32 logits carry a rounding error in proportion to their size (~110
    # here against ~1 in the unit-variance workloads), so the fp32 bounds
    # scale with the largest |logit| / 10; the bf16 bounds (set by the bf16
    # probabilities) hold as they are.
    big = max(float(np.abs(q[0, h].astype(np.float64) @ k[0, h].T.astype(np.float64)).max())
              for h in range(H)) * scale
    grow = 1.0 if dtype == "bf16" else max(1.0, big / 10.0)
    print(profile, dtype, dict(o_err=o_err, lse_err=l_err, max_logit=big), flush=True)
    assert o_err <= TOL_O[dtype] * grow and l_err <= TOL_LSE[dtype] * grow


def test_protected_rows_equal_the_dense_run_bitwise():
    """Eq. (11): a protected query block walks every key block in ascending
    order, exactly as the dense run of the same kernel does."""
    w = BASE.with_(name="k", H=2, frames=4, rows=10, cols=25, n_plant=2)
    x = synth.make_inputs(w)
    n_b = w.n_b
    t = {k: to_dev(x[k], "bf16") for k in ("q_v", "k_v", "v_v")}
    kv_idx, kv_cnt, _, _ = sa.sa_build_block_mask(
        t["q_v"], t["k_v"], w.scale, w.block, 2,
        torch.tensor([[0, 1, 0, 0, 1, 0, 0, 1]], dtype=torch.uint8, device="cuda"))
    o_sparse, _ = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale,
                                         w.block, kv_idx, kv_cnt)
    dense_idx = torch.arange(n_b, dtype=torch.int32, device="cuda").expand(1, 2, n_b, n_b).contiguous()
    dense_cnt = torch.full((1, 2, n_b), n_b, dtype=torch.int32, device="cuda")
    o_dense, _ = sa.sa_sparse_attention(t["q_v"], t["k_v"], t["v_v"], w.scale,
                                        w.block, dense_idx, dense_cnt)
    for r in (1, 4, 7):
        sl = slice(r * 128, min((r + 1) * 128, w.L_v))
        assert torch.equal(o_sparse[:, :, sl], o_dense[:, :, sl]), r
    assert not torch.equal(o_sparse[:, :, :128], o_dense[:, :, :128])


def test_exact_ties_follow_lower_index_first():
    """Q^a = 0 gives uniform saliency: blocks tie exactly, the lowest indices
    are protected and the short tail block ranks last.  Constant K gives equal
    pooled scores in every row: the first k_keep blocks are kept."""
    w = BASE.with_(name="l", H=2, frames=3, rows=10, cols=30, L_a=40, n_plant=0)
    x = synth.make_inputs(w)          # L_v = 900 -> 8 blocks, tail 4
    x["q_a"][:] = 0.0
    x["k_v"][:] = np.float32(0.5)
    g = gpu_layer(x, w, 3, 8)
    assert g["prot_idx"][0].tolist() == list(range(8))
    g = gpu_layer(x, w, 3, 5)
    assert g["prot_idx"][0].tolist() == [0, 1, 2, 3, 4]
    s_blk = g["sal_v_blk"][0]
    assert np.all(s_blk[:7] == s_blk[0]) and s_blk[7] < s_blk[0]
    unprot = g["prot_flag"][0] == 0
    for h in range(2):
        for r in np.nonzero(unprot)[0]:
            assert g["kv_idx"][0, h, r, :3].tolist() == [0, 1, 2]


def test_bitwise_reproducible_and_accumulate():
    w = SMALL[1][1]
    x = synth.make_inputs(w)
    a = gpu_layer(x, w, 2, 2)
    b = gpu_layer(x, w, 2, 2)
    for k in a:
        if a[k] is not None:
            assert np.array_equal(a[k], b[k], equal_nan=True), k
    t = {k: to_dev(x[k], "bf16") for k in ("q_v", "k_v", "q_a", "k_a")}
    tok, blk, aud = sa.sa_cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"],
                                       w.scale, w.block)
    tok2, blk2, aud2 = tok.clone(), blk.clone(), aud.clone()
    sa.sa_cross_scores(t["q_a"], t["k_v"], t["q_v"], t["k_a"], w.scale, w.block,
                       sal_v_tok=tok2, sal_v_blk=blk2, sal_a_tok=aud2, accumulate=True)
    assert torch.equal(tok2, 2 * tok) and torch.equal(blk2, 2 * blk)
    assert torch.equal(aud2, 2 * aud)


# the pooled means and mask rows are padded to 64 * E columns, E in
# {1, 2, 3, 4, 5, 6, 8, 10, 12, 16, 20, 24, 32}: one case per width beyond
# the powers of two, ragged tails, every list and G compared with the oracle
@pytest.mark.parametrize("n_b,E", [(150, 3), (300, 5), (370, 6), (480, 8), (600, 10),
                                   (640, 10), (700, 12), (1000, 16), (1100, 20), (1400, 24)])
def test_block_mask_at_padded_widths(n_b, E):
    w = BASE.with_(name=f"w{n_b}", H=2, d=64, block=64, frames=1, rows=1,
                   cols=64 * n_b - 21, L_a=16, n_plant=2)
    assert w.n_b == n_b and -(-n_b // 64) <= E
    k_keep = max(1, n_b // 7)
    print(f"case mask width n_b={n_b} E={E} k_keep={k_keep}", flush=True)
    x = synth.make_inputs(w)
    prot = np.zeros((1, n_b), dtype=np.uint8)
    prot[0, [0, n_b // 2, n_b - 1]] = 1
    t = {k: to_dev(x[k], "bf16") for k in ("q_v", "k_v")}
    kv_idx, kv_cnt, mask, scores = sa.sa_build_block_mask(
        t["q_v"], t["k_v"], w.scale, w.block, k_keep, torch.from_numpy(prot).cuda(),
        want_mask=True, want_scores=True)
    torch.cuda.synchronize()
    G = oracle.pooled_scores(x["q_v"], x["k_v"], w.scale, w.block)
    sc = scores.cpu().numpy()
    assert np.all(np.abs(sc - G) <= 2.0 ** -24 * np.abs(G) + 1e-12)
    check_kv_lists(kv_idx.cpu().numpy(), kv_cnt.cpu().numpy(), prot, G, k_keep,
                   mask.cpu().numpy())


@functools.lru_cache(maxsize=1)
def _mask_case(n_b):
    w = BASE.with_(name=f"x{n_b}", H=2, d=64, block=64, frames=1, rows=1,
                   cols=64 * n_b - 5, L_a=16, n_plant=2)
    x = synth.make_inputs(w)
    return w, x, oracle.pooled_scores(x["q_v"], x["k_v"], w.scale, w.block)


# the k-th order key is bounded by halving a key range; its extremes: the
# smallest key alone, all but the largest, and every key (the bound then lies
# between the largest real key and the padding keys of the row)
@pytest.mark.parametrize("n_b,k_keep", [(64, 1), (64, 63), (64, 64), (600, 1), (600, 599),
                                        (600, 600), (2000, 1), (2000, 1999), (2000, 2000)])
def test_block_mask_kth_extremes(n_b, k_keep):
    print(f"case mask k-th extremes n_b={n_b} k_keep={k_keep}", flush=True)
    w, x, G = _mask_case(n_b)
    assert w.n_b == n_b
    t = {k: to_dev(x[k], "bf16") for k in ("q_v", "k_v")}
    kv_idx, kv_cnt, mask, _ = sa.sa_build_block_mask(
        t["q_v"], t["k_v"], w.scale, w.block, k_keep, None, want_mask=True)
    torch.cuda.synchronize()
    idx, cnt = kv_idx.cpu().numpy(), kv_cnt.cpu().numpy()
    assert np.all(cnt == k_keep)
    check_kv_lists(idx, cnt, np.zeros((1, n_b), dtype=np.uint8), G, k_keep, mask.cpu().numpy())
    if k_keep == n_b:
        assert np.array_equal(idx, np.broadcast_to(np.arange(n_b, dtype=np.int32), idx.shape))
