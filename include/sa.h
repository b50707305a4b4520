/*
 * sa.h -- C ABI of the protected block-sparse video attention library
 * (libsa.so, MI355X / gfx950).
 *
 * The library implements one layer of the video hot path of
 * "Efficient Audio-Visual Generation via Synchrony-Aware Cross-Modal Sparse
 * Attention":
 *   1. sa_cross_scores      -- bidirectional audio-video cross-attention
 *                              saliency (Sec. 4.1, Eq. (1)-(2) and the
 *                              reverse direction stated after Eq. (2));
 *   2. sa_select_protected  -- protected query blocks by top-k of the block
 *                              saliency (Sec. 4.1 Eq. (3), Sec. 4.2 Eq. (8));
 *   3. sa_build_block_mask  -- sparse pattern S_m as pooled-QK block top-k,
 *                              with full rows for protected query blocks
 *                              (Sec. 4.2, Eq. (6) and (9));
 *   4. sa_sparse_attention  -- block-sparse flash attention over the
 *                              compacted key-block lists (Sec. 4.2,
 *                              Eq. (10)/(11); Eq. (5) when every list is full).
 * and the token-granular form of the protection:
 *   5. sa_saliency_ema              -- lagged saliency cache update (Eq. (4));
 *   6. sa_select_protected_tokens   -- protected query tokens by top-k of the
 *                                      token saliency (Eq. (3)/(8));
 *   7. sa_protected_token_attention -- dense rows of the protected tokens
 *                                      over the sparse output (Eq. (9)-(11));
 * the cross-modal attention forward whose row LSEs give the saliency:
 *   8. sa_cross_attention           -- dense cross-modal attention (Eq. (1));
 *   9. sa_cross_scores_from_lse     -- the saliency from its row LSEs;
 * and the cache-reuse decision:
 *  10. sa_cache_indicator           -- synchronization-aware cache-reuse
 *                                      indicator (Sec. 4.3, Eq. (12)-(15)).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensors are DEVICE pointers owned by the caller, contiguous, row-major
 *   [B, H, L, d] with d innermost, 16-byte aligned.  Q/K/V/O of one call share
 *   one dtype (SA_BF16 or SA_F32).  The library never allocates, frees or
 *   copies to the host.
 * - Calls are asynchronous on `stream` (a hipStream_t passed as void*;
 *   NULL = the default stream) and never synchronise the host.
 * - Return value: SA_OK or an SA_ERR_* code.  On any error nothing has been
 *   launched and nothing written; sa_last_error() gives a message
 *   (thread-local, valid until the next call on the same thread).
 *   SA_ERR_HIP reports a failed kernel launch (hipGetLastError).
 * - Budgets are plain integers; the caller computes ceil(ratio * count).
 * - Supported sizes: d in {64, 128}; block in {64, 128};
 *   1 <= n_b = ceil(L_v / block) <= 2048; L_a >= 1; B * H <= 65535 (larger
 *   products return SA_ERR_UNSUPPORTED).
 * - Results are bit-reproducible run to run (no floating-point atomics).
 * - Scratch memory ("workspace") is passed by the caller; its minimum size is
 *   sa_workspace_size(call, ...).  A smaller ws_bytes fails with
 *   SA_ERR_WORKSPACE.
 */
#ifndef SA_H_
#define SA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  SA_OK = 0,
  SA_ERR_INVALID_ARG = 1,  /* null pointer, bad size, bad budget, alignment */
  SA_ERR_UNSUPPORTED = 2,  /* d, block or dtype outside the supported set */
  SA_ERR_WORKSPACE = 3,    /* ws_bytes below sa_workspace_size(...) */
  SA_ERR_HIP = 4           /* a kernel launch failed */
};

enum { SA_BF16 = 0, SA_F32 = 1 };

enum {
  SA_CALL_CROSS_SCORES = 0,
  SA_CALL_BUILD_BLOCK_MASK = 1,
  SA_CALL_SPARSE_ATTENTION = 2,
  SA_CALL_SELECT_PROTECTED = 3,
  SA_CALL_CACHE_INDICATOR = 4,
  SA_CALL_TOKEN_ATTENTION = 5,
  SA_CALL_CROSS_ATTENTION = 6
};

/*
 * sa_cross_scores -- token and block saliency of one cross-attention layer.
 *
 * Sec. 4.1, Eq. (1): A^{a->v} = softmax(Q^a (K^v)^T * scale) over all L_v
 * video keys, per batch item and head.  Eq. (2): the video-token saliency is
 * the column mass of A^{a->v} summed over audio queries and heads, with Norm
 * taken as division by H * L_a (each softmax row sums to one, so the map sums
 * to one per batch item).  The reverse direction (v->a, the sentence after
 * Eq. (2)) gives the audio-token saliency with softmax over the L_a audio
 * keys, summed over video queries and heads, divided by H * L_v.  The block
 * saliency is the sum of the token saliency over each block of `block`
 * consecutive video tokens (the last block may be shorter).
 *
 *   q_a        [B,H,L_a,d]  audio queries (required)
 *   k_v        [B,H,L_v,d]  video keys (required)
 *   q_v        [B,H,L_v,d]  video queries; NULL skips the v->a direction
 *   k_a        [B,H,L_a,d]  audio keys; NULL iff q_v is NULL
 *   scale      softmax scale (normally 1/sqrt(d)), finite and > 0
 *   sal_v_tok  [B,L_v] f32 out, nullable
 *   sal_v_blk  [B,n_b] f32 out, required
 *   sal_a_tok  [B,L_a] f32 out, must be NULL iff q_v is NULL
 *   accumulate 0: outputs are overwritten; 1: the new values are added to
 *              what the outputs hold (sum over the layers of L_c)
 *   ws         workspace of at least sa_workspace_size(SA_CALL_CROSS_SCORES)
 */
int sa_cross_scores(const void* q_a, const void* k_v, const void* q_v,
                    const void* k_a, int B, int H, int L_v, int L_a, int d,
                    int dtype, float scale, int block, float* sal_v_tok,
                    float* sal_v_blk, float* sal_a_tok, int accumulate,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * sa_cross_attention -- the dense cross-modal attention forward of one layer
 * (the a->v and v->a attention of Eq. (1) and the sentence after Eq. (2)),
 * whose row log-sum-exps feed sa_cross_scores_from_lse.
 *
 * O = softmax(Q K^T * scale) V for every query of Q against all Lk keys:
 * Q^a against K^v, V^v (Lq = L_a, Lk = L_v) for the a->v direction, Q^v
 * against K^a, V^a (Lq = L_v, Lk = L_a) for v->a.  When Lq/128 row blocks
 * per head leave the chip short of work, the keys of each row block are cut
 * into up to 8 runs whose partial rows (f32) are merged in a fixed order.
 *
 *   q          [B,H,Lq,d] bf16; 1 <= Lq <= 262144
 *   k, v       [B,H,Lk,d] bf16; 1 <= Lk <= 262144
 *   o          [B,H,Lq,d] bf16 out (round to nearest even from fp32)
 *   lse        [B,H,Lq] f32 out, natural log of the softmax denominator of
 *              the scaled scores; nullable
 *   dtype      SA_BF16 only (SA_F32 returns SA_ERR_UNSUPPORTED)
 *   ws         workspace of at least sa_workspace_size(SA_CALL_CROSS_ATTENTION,
 *              B, H, Lq, Lk, d, 0) bytes (0: ws may be NULL)
 */
int sa_cross_attention(const void* q, const void* k, const void* v, void* o,
                       float* lse, int B, int H, int Lq, int Lk, int d,
                       int dtype, float scale, void* ws, size_t ws_bytes,
                       void* stream);

/*
 * sa_cross_scores_from_lse -- sa_cross_scores's outputs, given the row
 * log-sum-exps of the two cross-attention forwards (Sec. 4.1, Eq. (1)-(2)):
 * the saliency as a side output of attention the model computes anyway.
 *
 * The softmax of Eq. (1) is exp(scale * q.k - lse) with lse the row LSE of
 * that forward, so the first pass over the keys that sa_cross_scores needs
 * for it is skipped in both directions.  Arguments as in sa_cross_scores,
 * plus
 *   lse_a      [B,H,L_a] f32: lse of sa_cross_attention(Q^a, K^v, V^v)
 *   lse_v      [B,H,L_v] f32: lse of sa_cross_attention(Q^v, K^a, V^a);
 *              NULL iff q_v is NULL
 *   dtype      SA_BF16 only
 *   ws         workspace of at least sa_workspace_size(SA_CALL_CROSS_SCORES)
 * The results equal sa_cross_scores's up to the rounding of the given lse.
 */
int sa_cross_scores_from_lse(const void* q_a, const void* k_v, const void* q_v,
                             const void* k_a, const float* lse_a,
                             const float* lse_v, int B, int H, int L_v,
                             int L_a, int d, int dtype, float scale, int block,
                             float* sal_v_tok, float* sal_v_blk,
                             float* sal_a_tok, int accumulate, void* ws,
                             size_t ws_bytes, void* stream);

/*
 * sa_select_protected -- protected query blocks (Sec. 4.2, Eq. (8), at block
 * granularity; Sec. 4.1, Eq. (3)).
 *
 * Per batch item, the k_prot blocks of largest sal_blk; equal scores are
 * ordered by lower block index first.  The caller chooses which map is
 * ranked (the current one, or the lagged cache of Eq. (4)).
 *
 *   sal_blk    [B,n_b] f32 in (finite values)
 *   k_prot     0 <= k_prot <= n_b
 *   prot_idx   [B,k_prot] i32 out in rank order, nullable
 *   prot_flag  [B,n_b] u8 out, 1 = protected, required
 */
int sa_select_protected(const float* sal_blk, int B, int n_b, int k_prot,
                        int32_t* prot_idx, uint8_t* prot_flag, void* stream);

/*
 * sa_build_block_mask -- the protected block mask M~ of Eq. (9) as compacted
 * key-block lists (Sec. 4.2, Eq. (6) and (9)).
 *
 * The sparse pattern S_m is pooled-QK block top-k: Q and K are averaged over
 * each block of `block` tokens (the last block over its true length), the
 * pooled score is G[r,c] = scale * qbar_r . kbar_c, means and products in
 * fp64, and every query block r that is not protected keeps the k_keep key
 * blocks of largest G[r,:].  Equal scores go to the lower block index first;
 * the ranking compares the fp64 scores with their lowest 12 mantissa bits
 * dropped, so two scores within about 2^-40 relative of each other count as
 * equal.  A protected query block keeps every key block; protection adds
 * rows only.
 *
 *   q_v, k_v   [B,H,L_v,d] video queries and keys
 *   k_keep     1 <= k_keep <= n_b
 *   prot_flag  [B,n_b] u8 (nonzero = protected), shared by all heads;
 *              NULL = nothing protected
 *   kv_idx     [B,H,n_b,n_b] i32 out: kept key blocks of each query block in
 *              ascending order, first kv_cnt entries valid, the rest -1
 *   kv_cnt     [B,H,n_b] i32 out
 *   mask       [B,H,n_b,n_b] u8 out (1 = kept), nullable
 *   scores     [B,H,n_b,n_b] f32 out: the fp64 pooled scores G rounded once
 *              to fp32, nullable
 *   ws         workspace of at least sa_workspace_size(SA_CALL_BUILD_BLOCK_MASK)
 */
int sa_build_block_mask(const void* q_v, const void* k_v, int B, int H,
                        int L_v, int d, int dtype, float scale, int block,
                        int k_keep, const uint8_t* prot_flag, int32_t* kv_idx,
                        int32_t* kv_cnt, uint8_t* mask, float* scores,
                        void* ws, size_t ws_bytes, void* stream);

/*
 * Pooling fused into the saliency streams.  The mask's block means (Sec. 4.2,
 * Eq. (6)) are taken from the same Q^v and K^v that the saliency of Sec. 4.1
 * (Eq. (1)-(2) and the reverse direction) reads, so one pass over each serves
 * both: sa_cross_scores_pooled writes them, sa_build_block_mask_pooled ranks
 * them.  The pair gives the same lists as sa_cross_scores (or
 * sa_cross_scores_from_lse) followed by sa_build_block_mask: the means are
 * fp64 sums of the bf16 (or fp32) inputs divided once, as there, and such a
 * sum is exact (so independent of the order of the additions) whenever the
 * values of a block lie within 2^44 (bf16) or 2^28 (fp32) of each other in
 * magnitude.
 *
 * Layout of the means: qbar and kbar are each [B,H,d,n_pad] fp64 (block index
 * innermost), n_pad = sa_pool_columns(n_b); columns n_b .. n_pad-1 are never
 * written or read as scores.
 */

/* Columns n_pad of the pooled means for n_b blocks (0 if n_b is outside
 * [1, 2048]). */
int sa_pool_columns(int n_b);

/*
 * sa_cross_scores_pooled -- the saliency of sa_cross_scores (lse_a and lse_v
 * NULL) or of sa_cross_scores_from_lse (both given: the row LSEs of the two
 * sa_cross_attention forwards), plus the block means of Q^v and K^v.
 *
 * Both directions are computed (q_v, k_a, sal_a_tok are required).  With
 * bf16 inputs the means come from the streams of the column-mass passes:
 * K^v from the a->v pass (its first slab of audio queries), Q^v from the
 * rows each v->a workgroup holds.  fp32 inputs (standalone form only) pool
 * in a separate pass.  Other arguments and results as in sa_cross_scores.
 *
 *   lse_a, lse_v  [B,H,L_a], [B,H,L_v] f32, both NULL or both non-NULL
 *                 (non-NULL: SA_BF16 only)
 *   qbar, kbar    out, [B,H,d,sa_pool_columns(n_b)] fp64 each, 8-byte
 *                 aligned, not overlapping
 *   ws            workspace of at least sa_workspace_size(SA_CALL_CROSS_SCORES)
 */
int sa_cross_scores_pooled(const void* q_a, const void* k_v, const void* q_v,
                           const void* k_a, const float* lse_a,
                           const float* lse_v, int B, int H, int L_v, int L_a,
                           int d, int dtype, float scale, int block,
                           float* sal_v_tok, float* sal_v_blk,
                           float* sal_a_tok, int accumulate, double* qbar,
                           double* kbar, void* ws, size_t ws_bytes,
                           void* stream);

/*
 * sa_build_block_mask_pooled -- sa_build_block_mask from the block means that
 * sa_cross_scores_pooled wrote (Sec. 4.2, Eq. (6) and (9)): G, the ranking,
 * the protection and the outputs are those of sa_build_block_mask.  d, block
 * and L_v must be those of the pooling call.  No workspace.
 *
 *   qbar, kbar [B,H,d,sa_pool_columns(n_b)] fp64 in, 8-byte aligned
 */
int sa_build_block_mask_pooled(const double* qbar, const double* kbar, int B,
                               int H, int L_v, int d, float scale, int block,
                               int k_keep, const uint8_t* prot_flag,
                               int32_t* kv_idx, int32_t* kv_cnt,
                               uint8_t* mask, float* scores, void* stream);

/*
 * sa_sparse_attention -- protected block-sparse attention (Sec. 4.2,
 * Eq. (10) in its row form Eq. (11)).
 *
 * Query block r of head (b,h) attends to the tokens of key blocks
 * kv_idx[b,h,r,0:kv_cnt[b,h,r]] with an exact softmax (non-causal); a full
 * list gives dense attention, Eq. (5).  Keys past L do not exist.
 *
 *   q, k, v    [B,H,L,d] in dtype
 *   o          [B,H,L,d] out in dtype (round to nearest even from fp32)
 *   lse        [B,H,L] f32 out, natural-log log-sum-exp of the scaled
 *              logits of each row, nullable
 *   kv_idx     [B,H,n_b,n_b] i32; entries outside [0,n_b) are ignored
 *   kv_cnt     [B,H,n_b] i32, clamped to [0,n_b]; a row with no valid entry
 *              outputs zeros and lse = -inf
 *   ws         workspace of at least sa_workspace_size(SA_CALL_SPARSE_ATTENTION)
 */
int sa_sparse_attention(const void* q, const void* k, const void* v, void* o,
                        float* lse, int B, int H, int L, int d, int dtype,
                        float scale, int block, const int32_t* kv_idx,
                        const int32_t* kv_cnt, void* ws, size_t ws_bytes,
                        void* stream);

/*
 * sa_sparse_attention_noalloc -- sa_sparse_attention without a workspace
 * argument and without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid hipMalloc).
 *
 * Arguments, results and errors are those of sa_sparse_attention; the same
 * kernels run, so the outputs are bitwise those of sa_sparse_attention.  The
 * scratch (the launch order and schedule of the query blocks, two arrays of
 * B*H*n_b int32, and 8 row counters) lives in a 4 MiB array that the library
 * holds on each device it runs on until the process ends, so
 * B*H*n_b <= 524032; larger sizes fail with
 * SA_ERR_UNSUPPORTED before any launch.  Every element of the scratch that a
 * call reads is written by that call first (the row counters are set to zero
 * by a kernel of the same call), so nothing has to be cleared beforehand.
 * All calls on one device share the array: calls that overlap in time on one
 * device (on different streams, or from different threads) race and must be
 * serialised by the caller.  `stream` must belong to the current device.
 * The first call on a device looks up the array's device address
 * (hipGetSymbolAddress), which needs no allocation.
 */
int sa_sparse_attention_noalloc(const void* q, const void* k, const void* v,
                                void* o, float* lse, int B, int H, int L,
                                int d, int dtype, float scale, int block,
                                const int32_t* kv_idx, const int32_t* kv_cnt,
                                void* stream);

/*
 * sa_saliency_ema -- one update of the lagged saliency cache (Sec. 4.1,
 * Eq. (4)): sal_bar[i] = alpha * sal_bar[i] + (1 - alpha) * sal[i] for
 * i < n, in fp32.  The refresh schedule (every K denoising steps) is the
 * caller's; Eq. (4) gives no alpha, so it is an argument.
 *
 *   sal_bar    [n] f32 in/out
 *   sal        [n] f32 in; either the same buffer as sal_bar or disjoint
 *   alpha      0 <= alpha <= 1
 *   n          number of entries; 0 = nothing to do
 */
int sa_saliency_ema(float* sal_bar, const float* sal, size_t n, float alpha,
                    void* stream);

/*
 * sa_select_protected_tokens -- protected query tokens (Sec. 4.2, Eq. (8);
 * Sec. 4.1, Eq. (3)) at token granularity.
 *
 * Per batch item, the k_tok tokens of largest sal_tok (equal scores: lower
 * token index first), listed in ascending token order.  The set is shared by
 * all heads.
 *
 *   sal_tok    [B,L] f32 in (finite values), 1 <= L <= 262144
 *   k_tok      0 <= k_tok <= L (the caller computes ceil(rho * L))
 *   tok_idx    [B,k_tok] i32 out, ascending token order, nullable
 *   tok_flag   [B,L] u8 out, 1 = protected, nullable
 * At least one of tok_idx and tok_flag is non-NULL.  No workspace.
 */
int sa_select_protected_tokens(const float* sal_tok, int B, int L, int k_tok,
                               int32_t* tok_idx, uint8_t* tok_flag,
                               void* stream);

/*
 * sa_protected_token_attention -- dense attention rows of the protected
 * query tokens (Sec. 4.2, Eq. (11) first case: Eq. (9) keeps every key of a
 * protected query).
 *
 * For every head (b,h) and j < k_tok, token t = tok_idx[b,j] attends to all
 * L keys with an exact softmax, and row t of o (and of lse) is overwritten.
 * Run after sa_sparse_attention on lists built without block protection to
 * obtain Eq. (11) with protected tokens; every other row is left as it is.
 *
 *   q, k, v    [B,H,L,d] in dtype; 1 <= L <= 262144
 *   o          [B,H,L,d] in/out (round to nearest even from fp32)
 *   lse        [B,H,L] f32 in/out, nullable
 *   tok_idx    [B,k_tok] i32; entries outside [0,L) are skipped
 *   k_tok      0 <= k_tok <= L; 0 = nothing to do
 *   ws         workspace of at least sa_workspace_size(SA_CALL_TOKEN_ATTENTION,
 *              B, H, L, k_tok, d, 0) bytes (0 when the keys of a row are not
 *              split: then ws may be NULL).  With bf16 inputs the keys of each
 *              row may be cut into up to 8 runs whose partial rows (f32) are
 *              merged in a fixed order, so results do not depend on timing.
 */
int sa_protected_token_attention(const void* q, const void* k, const void* v,
                                 void* o, float* lse, int B, int H, int L,
                                 int d, int dtype, float scale,
                                 const int32_t* tok_idx, int k_tok, void* ws,
                                 size_t ws_bytes, void* stream);

/*
 * sa_cache_indicator -- synchronization-aware cache-reuse indicator of one
 * block at one denoising step (Sec. 4.3, Eq. (12)-(15)).
 *
 *   dv = ||Y^v - Yh^v||_1 / (||Y^v||_1 + eps)                     Eq. (12)
 *   da = the same for the audio outputs                             Eq. (12)
 *   dp = dv restricted to the rows of protected video tokens        Eq. (13)
 *   ds = 1 - <s_bar, s_hat> / (||s_bar||_2 ||s_hat||_2 + eps)       Eq. (14)
 *   sync = max(dv, da, lambda_p * dp, lambda_s * ds)                Eq. (15)
 *   reuse = sync < tau (decided on the fp32 value written to out[4])
 * Every norm runs over the whole output (all batch items and channels):
 * one decision per (step, block).  A NULL pair (audio, saliency, protected
 * flags) contributes 0 to the max.  The paper uses lambda_p = 0.5,
 * lambda_s = 0.1, tau = 0.2; eps is not given there.
 *
 *   y_v, y_v_hat   [B,L_v,C] in dtype: current and cached video block outputs
 *   prot_flag      [B,L_v] u8, nonzero = protected token row, nullable
 *   y_a, y_a_hat   [B,L_a,C] in dtype, both NULL or both non-NULL (L_a >= 1)
 *   s_bar, s_hat   [B,L_v] f32 current and cached saliency, both NULL or both
 *   C              channels per row, >= 8 and a multiple of 8; a
 *                  workgroup's share (ceil(B*L_v/1024) video rows, ceil(B*L_a/64)
 *                  audio rows) holds at most 2^32 - 1 chunks of 16 bytes, else
 *                  SA_ERR_INVALID_ARG
 *   out            [6] f32 out (device): dv, da, dp, ds, sync, reuse (1 or 0)
 *   ws             workspace of at least sa_workspace_size(SA_CALL_CACHE_INDICATOR)
 */
int sa_cache_indicator(const void* y_v, const void* y_v_hat,
                       const uint8_t* prot_flag, const void* y_a,
                       const void* y_a_hat, const float* s_bar,
                       const float* s_hat, int B, int L_v, int L_a, int C,
                       int dtype, float lambda_p, float lambda_s, float tau,
                       float eps, float* out, void* ws, size_t ws_bytes,
                       void* stream);

/*
 * Minimum workspace bytes of a call (SA_CALL_*) at the given sizes; L_a is
 * read by SA_CALL_CROSS_SCORES and SA_CALL_CACHE_INDICATOR (0 = no audio),
 * and SA_CALL_CACHE_INDICATOR reads B, L_v and L_a only.
 * SA_CALL_TOKEN_ATTENTION reads B, H, L_v (the sequence length L), d and
 * k_tok in the place of L_a; SA_CALL_CROSS_ATTENTION reads B, H, Lq in the
 * place of L_v, Lk in the place of L_a, and d; block is not read by either.  Returns 0 for sizes the
 * call rejects.
 * The figure covers both dtypes.
 */
size_t sa_workspace_size(int call, int B, int H, int L_v, int L_a, int d,
                         int block);

/* Message for the last non-OK return on this thread ("" if none). */
const char* sa_last_error(void);

/* Library ABI version (major * 100 + minor). */
int sa_version(void);

/*
 * Identity of the sources the library was built from: the first 16 hex
 * digits of a sha256 over the kernel sources, the internal headers and this
 * header ("unknown" for a build that did not supply it).  A caller that has
 * the sources can compare it before use; the Python binding does.
 */
const char* sa_build_id(void);

#ifdef __cplusplus
}
#endif

#endif /* SA_H_ */
