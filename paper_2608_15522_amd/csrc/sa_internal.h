// Host-side internals of libsa.so: workspace layout and kernel launchers.
// The public entry points (sa_api.hip) validate every argument, then call
// these launchers, which only enqueue kernels on the given stream.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sa {

// Tunables fixed at build time.
constexpr int kLseChunk = 1024;   // video keys per a->v log-sum-exp partial
constexpr int kQSlab = 512;       // queries per 16-wave workgroup slab
constexpr int kV2aChunk = 512;    // video queries per v->a workgroup
constexpr int kMaxBlocks = 2048;  // largest supported n_b
constexpr int kMaxPairs = 65535;  // largest B*H (a grid dimension indexes (b, h))

inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

// Workspace of sa_cross_scores (both dtypes are covered).
struct CrossWs {
  size_t lse_part;   // float2 [B,H,nchunk,L_a]  (m, l) partials, bf16 path
  size_t lse_a;      // float  [B,H,L_a]         a->v log2-sum-exp
  size_t colmass;    // float  [B,H,L_v]         per-head a->v column mass
  size_t lse_v;      // float  [B,H,L_v]         v->a log2-sum-exp, f32 path
  size_t v2a_part;   // float  [B,H,nchunk3,L_a] v->a column-mass partials
  size_t v2a_head;   // float  [B,H,L_a]         the same summed over chunks
  size_t total;
};

inline CrossWs cross_ws_layout(int B, int H, int L_v, int L_a) {
  CrossWs w{};
  const size_t nchunk = (L_v + kLseChunk - 1) / kLseChunk;
  const size_t nchunk3 = (L_v + kV2aChunk - 1) / kV2aChunk;
  size_t off = 0;
  w.lse_part = off; off += align_up(sizeof(float) * 2 * B * H * nchunk * L_a);
  w.lse_a = off;    off += align_up(sizeof(float) * B * H * L_a);
  w.colmass = off;  off += align_up(sizeof(float) * B * H * L_v);
  w.lse_v = off;    off += align_up(sizeof(float) * B * H * L_v);
  w.v2a_part = off; off += align_up(sizeof(float) * B * H * nchunk3 * L_a);
  w.v2a_head = off; off += align_up(sizeof(float) * B * H * L_a);
  w.total = off;
  return w;
}

// Column count of the pooled block means and of the mask rows: 64 * E, with
// E the smallest of the instantiated widths {1, 2, 3, 4, 5, 6, 8, 10, 12,
// 16, 20, 24, 32} that covers n_b (n_b <= 2048).
inline int mask_e(int n_b) {
  constexpr int kWidths[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 16, 20, 24, 32};
  const int need = (n_b + 63) / 64;
  for (int e : kWidths)
    if (e >= need) return e;
  return 32;
}
inline int mask_n_pad(int n_b) { return 64 * mask_e(n_b); }

struct MaskWs {
  size_t qbar;   // double [B,H,d,n_pad]  pooled query means, block index innermost
  size_t kbar;   // double [B,H,d,n_pad]  pooled key means, block index innermost
  size_t total;
};

inline MaskWs mask_ws_layout(int B, int H, int n_b, int d) {
  MaskWs w{};
  const size_t n_pad = static_cast<size_t>(mask_n_pad(n_b));
  size_t off = 0;
  w.qbar = off; off += align_up(sizeof(double) * B * H * d * n_pad);
  w.kbar = off; off += align_up(sizeof(double) * B * H * d * n_pad);
  w.total = off;
  return w;
}

struct AttnWs {
  size_t order;   // int [B,H,n_b]  query blocks of each head, heaviest first
  size_t sched;   // int [8][B*H/8][n_b]  per-XCD launch list (B*H a multiple of 8)
  size_t claim;   // int [8][64]  rows taken from each XCD's list (one per 256 bytes)
  size_t total;
};

inline AttnWs attn_ws_layout(int B, int H, int n_b, int /*d*/, int /*block*/) {
  AttnWs w{};
  size_t off = 0;
  w.order = off; off += align_up(sizeof(int32_t) * B * H * n_b);
  w.sched = off; off += align_up(sizeof(int32_t) * B * H * n_b);
  w.claim = off; off += align_up(sizeof(int32_t) * 8 * 64);
  w.total = off;
  return w;
}

// ---- launchers (defined in the kernel sources) ----------------------------
constexpr int kMaxTokens = kMaxBlocks * 128;  // longest token sequence (L)
// Cache-reuse indicator: 9 fp32 partial sums per workgroup of the first pass
// ([9][workgroups]); 1024 video workgroups fill one round of 256 CUs x 4.
inline int cache_workgroups_video(size_t rows_v) {
  return static_cast<int>(rows_v < 1024 ? rows_v : 1024);
}
inline int cache_workgroups_audio(size_t rows_a) {
  return static_cast<int>(rows_a < 64 ? rows_a : 64);
}
inline size_t cache_ws_bytes(int B, int L_v, int L_a) {
  const size_t nwg = static_cast<size_t>(cache_workgroups_video(static_cast<size_t>(B) * L_v)) +
                     cache_workgroups_audio(static_cast<size_t>(B) * (L_a > 0 ? L_a : 0));
  return align_up(nwg * 9 * sizeof(float));
}
void launch_cache_indicator(const void* y_v, const void* y_v_hat, const uint8_t* prot_flag,
                            const void* y_a, const void* y_a_hat, const float* s_bar,
                            const float* s_hat, int B, int L_v, int L_a, int C, int dtype,
                            float lambda_p, float lambda_s, float tau, float eps,
                            float* out, char* ws, hipStream_t s);
void launch_saliency_ema(float* s_bar, const float* s, size_t n, float alpha,
                         hipStream_t st);
void launch_select_protected_tokens(const float* sal_tok, int B, int L, int k_tok,
                                    int32_t* tok_idx, uint8_t* tok_flag, hipStream_t st);
// Protected-token rows run in workgroups of kTokRowBlock gathered rows.  The
// keys of a row are cut into n_split runs so that the launch fills the 512
// workgroup slots of the chip (256 CUs, 2 attention workgroups each) in
// whole rounds: n_split minimises rounds/n_split * (1 + 0.02*n_split), where
// the second factor prices each workgroup's fixed cost (pipeline fill, the
// partial row, its share of the combine); 1 <= n_split <= 8, and every run
// keeps at least 4 key blocks.
constexpr int kTokRowBlock = 128;
inline int token_attn_splits(int P, int k_tok, int n_b) {
  const long units = static_cast<long>(P) * ceil_div(k_tok, kTokRowBlock);
  int smax = n_b / 4;
  smax = smax < 1 ? 1 : (smax > 8 ? 8 : smax);
  int best = 1;
  double best_cost = 0.0;
  for (int s = 1; s <= smax; ++s) {
    const double rounds = static_cast<double>((units * s + 511) / 512);
    const double cost = rounds / s * (1.0 + 0.02 * s);
    if (s == 1 || cost < best_cost - 1e-9) {
      best = s;
      best_cost = cost;
    }
  }
  return best;
}
// Partial rows [n_split][B*H][k_tok][d] f32, then (m, l) [n_split][B*H][k_tok]
// float2; none with one split.
inline size_t token_attn_ws_bytes(int B, int H, int L, int d, int k_tok) {
  const int ns = token_attn_splits(B * H, k_tok, ceil_div(L, kTokRowBlock));
  if (ns <= 1 || k_tok <= 0) return 0;
  return align_up(static_cast<size_t>(ns) * B * H * k_tok * (static_cast<size_t>(d) * 4 + 8));
}
void launch_protected_token_attention_bf16(const uint16_t* q, const uint16_t* k,
                                           const uint16_t* v, uint16_t* o, float* lse,
                                           int B, int H, int L, int d, float scale,
                                           const int32_t* tok_idx, int k_tok, char* ws,
                                           hipStream_t s);
// Dense cross-modal attention (queries [B,H,Lq,d], keys/values [B,H,Lk,d]);
// the workspace is token_attn_ws_bytes(B, H, Lk, d, Lq).
void launch_cross_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                 uint16_t* o, float* lse, int B, int H, int Lq, int Lk, int d,
                                 float scale, char* ws, hipStream_t s);
void launch_protected_token_attention_f32(const float* q, const float* k, const float* v,
                                          float* o, float* lse, int B, int H, int L, int d,
                                          float scale, const int32_t* tok_idx, int k_tok,
                                          hipStream_t s);
void launch_cross_scores_bf16(const uint16_t* q_a, const uint16_t* k_v,
                              const uint16_t* q_v, const uint16_t* k_a, int B,
                              int H, int L_v, int L_a, int d, float scale,
                              int block, float* sal_v_tok, float* sal_v_blk,
                              float* sal_a_tok, int accumulate, double* qbar,
                              double* kbar, char* ws, hipStream_t s);
// Saliency from the row LSEs (natural log, [B,H,L_a] and [B,H,L_v]) of the
// two cross-attention forwards; the workspace is cross_ws_layout's.
void launch_cross_scores_from_lse_bf16(const uint16_t* q_a, const uint16_t* k_v,
                                       const uint16_t* q_v, const uint16_t* k_a,
                                       const float* lse_a, const float* lse_v, int B, int H,
                                       int L_v, int L_a, int d, float scale, int block,
                                       float* sal_v_tok, float* sal_v_blk, float* sal_a_tok,
                                       int accumulate, double* qbar, double* kbar, char* ws,
                                       hipStream_t s);
void launch_cross_scores_f32(const float* q_a, const float* k_v,
                             const float* q_v, const float* k_a, int B, int H,
                             int L_v, int L_a, int d, float scale, int block,
                             float* sal_v_tok, float* sal_v_blk,
                             float* sal_a_tok, int accumulate, char* ws,
                             hipStream_t s);
void launch_select_protected(const float* sal_blk, int B, int n_b, int k_prot,
                             int32_t* prot_idx, uint8_t* prot_flag,
                             hipStream_t s);
void launch_build_block_mask(const void* q_v, const void* k_v, int B, int H,
                             int L_v, int d, int dtype, float scale, int block,
                             int k_keep, const uint8_t* prot_flag,
                             int32_t* kv_idx, int32_t* kv_cnt, uint8_t* mask,
                             float* scores, char* ws, hipStream_t s);
// The pooling pass alone (K5): block means of q_v and k_v into qbar, kbar
// ([B,H,d,mask_n_pad(n_b)]).
void launch_block_pool(const void* q_v, const void* k_v, int B, int H, int L_v, int d,
                       int dtype, int block, double* qbar, double* kbar, hipStream_t s);
// The mask from given block means (K6 alone).
void launch_mask_from_means(const double* qbar, const double* kbar, int B, int H, int L_v,
                            int d, float scale, int block, int k_keep,
                            const uint8_t* prot_flag, int32_t* kv_idx, int32_t* kv_cnt,
                            uint8_t* mask, float* scores, hipStream_t s);
void launch_sparse_attention_bf16(const uint16_t* q, const uint16_t* k,
                                  const uint16_t* v, uint16_t* o, float* lse,
                                  int B, int H, int L, int d, float scale,
                                  int block, const int32_t* kv_idx,
                                  const int32_t* kv_cnt, char* ws,
                                  hipStream_t s);
void launch_sparse_attention_f32(const float* q, const float* k,
                                 const float* v, float* o, float* lse, int B,
                                 int H, int L, int d, float scale, int block,
                                 const int32_t* kv_idx, const int32_t* kv_cnt,
                                 char* ws, hipStream_t s);

}  // namespace sa
