// Public C ABI of libsa.so: argument validation, workspace sizing, error
// reporting, dispatch to the kernel launchers.  Every check runs on the host
// before any launch, so a rejected call writes nothing.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>

#include "../../include/sa.h"
#include "sa_device.h"
#include "sa_internal.h"

// Scratch of sa_sparse_attention_noalloc: each device holds its own copy of
// this array until the process ends.  Calls on one device share it.
constexpr size_t kStaticScratchBytes = static_cast<size_t>(4) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
char* g_scratch_ptr[kMaxScratchDevices];  // device address of scratch, per device

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int ok() {
  g_last_error.clear();
  return SA_OK;
}

int check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(SA_ERR_HIP, "%s: kernel launch failed: %s", what, hipGetErrorString(e));
  return ok();
}

bool aligned(const void* p, size_t a) {
  return (reinterpret_cast<uintptr_t>(p) % a) == 0;
}

// Shared shape checks; returns SA_OK or an error code with the message set.
int check_common(const char* fn, int B, int H, int L, int d, int dtype, float scale,
                 int block) {
  if (B < 1 || H < 1 || L < 1)
    return fail(SA_ERR_INVALID_ARG, "%s: B=%d H=%d L=%d must all be >= 1", fn, B, H, L);
  if (static_cast<long long>(B) * H > sa::kMaxPairs)  // one grid dimension per (b, h)
    return fail(SA_ERR_UNSUPPORTED, "%s: B*H=%lld exceeds %d", fn,
                static_cast<long long>(B) * H, sa::kMaxPairs);
  if (dtype != SA_BF16 && dtype != SA_F32)
    return fail(SA_ERR_UNSUPPORTED, "%s: dtype %d is neither SA_BF16 nor SA_F32", fn, dtype);
  if (d != 64 && d != 128)
    return fail(SA_ERR_UNSUPPORTED, "%s: head dim d=%d not in {64, 128}", fn, d);
  if (block != 64 && block != 128)
    return fail(SA_ERR_UNSUPPORTED, "%s: block=%d not in {64, 128}", fn, block);
  const long long n_b = (static_cast<long long>(L) + block - 1) / block;
  if (n_b > sa::kMaxBlocks)
    return fail(SA_ERR_UNSUPPORTED, "%s: n_b=%lld blocks exceeds %d", fn, n_b,
                sa::kMaxBlocks);
  if (!(scale > 0.f) || !isfinite(scale))
    return fail(SA_ERR_INVALID_ARG, "%s: scale=%g must be finite and > 0", fn,
                static_cast<double>(scale));
  return SA_OK;
}

int check_tensor(const char* fn, const char* name, const void* p, bool required,
                 size_t align) {
  if (p == nullptr) {
    if (required) return fail(SA_ERR_INVALID_ARG, "%s: %s is NULL", fn, name);
    return SA_OK;
  }
  if (!aligned(p, align))
    return fail(SA_ERR_INVALID_ARG, "%s: %s is not %zu-byte aligned", fn, name, align);
  return SA_OK;
}

int check_ws(const char* fn, const void* ws, size_t ws_bytes, size_t need) {
  if (ws_bytes < need)
    return fail(SA_ERR_WORKSPACE, "%s: workspace of %zu bytes is below the %zu required",
                fn, ws_bytes, need);
  if (need > 0 && ws == nullptr) return fail(SA_ERR_INVALID_ARG, "%s: ws is NULL", fn);
  if (need > 0 && !aligned(ws, 16))
    return fail(SA_ERR_INVALID_ARG, "%s: ws is not 16-byte aligned", fn);
  return SA_OK;
}

#ifndef SA_SRC_ID
#define SA_SRC_ID "unknown"
#endif

#define SA_TRY(expr)          \
  do {                        \
    const int rc_ = (expr);   \
    if (rc_ != SA_OK) return rc_; \
  } while (0)

int check_sparse_attention_args(const char* fn, const void* q, const void* k, const void* v,
                                const void* o, const float* lse, int B, int H, int L, int d,
                                int dtype, float scale, int block, const int32_t* kv_idx,
                                const int32_t* kv_cnt) {
  SA_TRY(check_common(fn, B, H, L, d, dtype, scale, block));
  SA_TRY(check_tensor(fn, "q", q, true, 16));
  SA_TRY(check_tensor(fn, "k", k, true, 16));
  SA_TRY(check_tensor(fn, "v", v, true, 16));
  SA_TRY(check_tensor(fn, "o", o, true, 16));
  SA_TRY(check_tensor(fn, "lse", lse, false, 4));
  SA_TRY(check_tensor(fn, "kv_idx", kv_idx, true, 4));
  SA_TRY(check_tensor(fn, "kv_cnt", kv_cnt, true, 4));
  return SA_OK;
}

void launch_sparse_attention(const void* q, const void* k, const void* v, void* o, float* lse,
                             int B, int H, int L, int d, int dtype, float scale, int block,
                             const int32_t* kv_idx, const int32_t* kv_cnt, char* ws,
                             hipStream_t s) {
  if (dtype == SA_BF16)
    sa::launch_sparse_attention_bf16(
        static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
        static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), lse, B, H, L, d,
        scale, block, kv_idx, kv_cnt, ws, s);
  else
    sa::launch_sparse_attention_f32(
        static_cast<const float*>(q), static_cast<const float*>(k),
        static_cast<const float*>(v), static_cast<float*>(o), lse, B, H, L, d, scale,
        block, kv_idx, kv_cnt, ws, s);
}

// The device address of `scratch` on the device that runs stream s, looked up
// on the first call on that device (with it current) and kept.  The array's
// host-side name is not a device address; only the address returned here is
// passed to kernels.
int static_scratch(const char* fn, hipStream_t s, char** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return fail(SA_ERR_HIP, "%s: hipGetDevice failed: %s", fn, hipGetErrorString(e));
  if (s != nullptr) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(s, &sdev);
    if (e != hipSuccess)
      return fail(SA_ERR_HIP, "%s: hipStreamGetDevice failed: %s", fn, hipGetErrorString(e));
    if (sdev != dev)
      return fail(SA_ERR_INVALID_ARG, "%s: the stream belongs to device %d, not to the "
                  "current device %d", fn, static_cast<int>(sdev), dev);
  }
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(SA_ERR_UNSUPPORTED, "%s: device %d outside [0, %d)", fn, dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(SA_ERR_HIP, "%s: hipGetSymbolAddress(scratch) failed on device %d: %s", fn,
                  dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return SA_OK;
}

}  // namespace

extern "C" {

int sa_version(void) { return 100; }

const char* sa_build_id(void) { return SA_SRC_ID; }

const char* sa_last_error(void) { return g_last_error.c_str(); }

size_t sa_workspace_size(int call, int B, int H, int L_v, int L_a, int d, int block) {
  if (call == SA_CALL_CACHE_INDICATOR)
    return (B < 1 || L_v < 1 || L_a < 0) ? 0 : sa::cache_ws_bytes(B, L_v, L_a);
  if (static_cast<long long>(B) * H > sa::kMaxPairs) return 0;
  if (call == SA_CALL_CROSS_ATTENTION) {  // L_v carries Lq, L_a carries Lk
    const int Lq = L_v, Lk = L_a;
    if (B < 1 || H < 1 || Lq < 1 || Lq > sa::kMaxTokens || Lk < 1 || Lk > sa::kMaxTokens ||
        (d != 64 && d != 128))
      return 0;
    return sa::token_attn_ws_bytes(B, H, Lk, d, Lq);
  }
  if (call == SA_CALL_TOKEN_ATTENTION) {  // L_a carries k_tok
    if (B < 1 || H < 1 || L_v < 1 || L_v > sa::kMaxTokens || (d != 64 && d != 128) ||
        L_a < 0 || L_a > L_v)
      return 0;
    return sa::token_attn_ws_bytes(B, H, L_v, d, L_a);
  }
  if (B < 1 || H < 1 || L_v < 1 || (d != 64 && d != 128) || (block != 64 && block != 128))
    return 0;
  // in 64 bits: L_v + block - 1 overflows int for L_v near INT_MAX
  if ((static_cast<long long>(L_v) + block - 1) / block > sa::kMaxBlocks) return 0;
  const int n_b = sa::ceil_div(L_v, block);
  switch (call) {
    case SA_CALL_CROSS_SCORES:
      if (L_a < 1) return 0;
      return sa::cross_ws_layout(B, H, L_v, L_a).total;
    case SA_CALL_BUILD_BLOCK_MASK:
      return sa::mask_ws_layout(B, H, n_b, d).total;
    case SA_CALL_SPARSE_ATTENTION:
      return sa::attn_ws_layout(B, H, n_b, d, block).total;
    case SA_CALL_SELECT_PROTECTED:
      return 0;
    default:
      return 0;
  }
}

int sa_cross_scores(const void* q_a, const void* k_v, const void* q_v, const void* k_a,
                    int B, int H, int L_v, int L_a, int d, int dtype, float scale,
                    int block, float* sal_v_tok, float* sal_v_blk, float* sal_a_tok,
                    int accumulate, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sa_cross_scores";
  SA_TRY(check_common(fn, B, H, L_v, d, dtype, scale, block));
  if (L_a < 1) return fail(SA_ERR_INVALID_ARG, "%s: L_a=%d must be >= 1", fn, L_a);
  if (accumulate != 0 && accumulate != 1)
    return fail(SA_ERR_INVALID_ARG, "%s: accumulate=%d must be 0 or 1", fn, accumulate);
  const bool rev = q_v != nullptr;
  if ((k_a != nullptr) != rev || (sal_a_tok != nullptr) != rev)
    return fail(SA_ERR_INVALID_ARG,
                "%s: q_v, k_a and sal_a_tok must be all NULL or all non-NULL", fn);
  SA_TRY(check_tensor(fn, "q_a", q_a, true, 16));
  SA_TRY(check_tensor(fn, "k_v", k_v, true, 16));
  SA_TRY(check_tensor(fn, "q_v", q_v, false, 16));
  SA_TRY(check_tensor(fn, "k_a", k_a, false, 16));
  SA_TRY(check_tensor(fn, "sal_v_tok", sal_v_tok, false, 4));
  SA_TRY(check_tensor(fn, "sal_v_blk", sal_v_blk, true, 4));
  SA_TRY(check_tensor(fn, "sal_a_tok", sal_a_tok, false, 4));
  SA_TRY(check_ws(fn, ws, ws_bytes, sa::cross_ws_layout(B, H, L_v, L_a).total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  if (dtype == SA_BF16)
    sa::launch_cross_scores_bf16(
        static_cast<const uint16_t*>(q_a), static_cast<const uint16_t*>(k_v),
        static_cast<const uint16_t*>(q_v), static_cast<const uint16_t*>(k_a), B, H, L_v,
        L_a, d, scale, block, sal_v_tok, sal_v_blk, sal_a_tok, accumulate, nullptr, nullptr,
        w, s);
  else
    sa::launch_cross_scores_f32(
        static_cast<const float*>(q_a), static_cast<const float*>(k_v),
        static_cast<const float*>(q_v), static_cast<const float*>(k_a), B, H, L_v, L_a,
        d, scale, block, sal_v_tok, sal_v_blk, sal_a_tok, accumulate, w, s);
  return check_launch(fn);
}

int sa_cross_scores_from_lse(const void* q_a, const void* k_v, const void* q_v,
                             const void* k_a, const float* lse_a, const float* lse_v, int B,
                             int H, int L_v, int L_a, int d, int dtype, float scale, int block,
                             float* sal_v_tok, float* sal_v_blk, float* sal_a_tok,
                             int accumulate, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sa_cross_scores_from_lse";
  SA_TRY(check_common(fn, B, H, L_v, d, dtype, scale, block));
  if (dtype != SA_BF16)
    return fail(SA_ERR_UNSUPPORTED, "%s: only SA_BF16 inputs are supported", fn);
  if (L_a < 1) return fail(SA_ERR_INVALID_ARG, "%s: L_a=%d must be >= 1", fn, L_a);
  if (accumulate != 0 && accumulate != 1)
    return fail(SA_ERR_INVALID_ARG, "%s: accumulate=%d must be 0 or 1", fn, accumulate);
  const bool rev = q_v != nullptr;
  if ((k_a != nullptr) != rev || (sal_a_tok != nullptr) != rev || (lse_v != nullptr) != rev)
    return fail(SA_ERR_INVALID_ARG,
                "%s: q_v, k_a, lse_v and sal_a_tok must be all NULL or all non-NULL", fn);
  SA_TRY(check_tensor(fn, "q_a", q_a, true, 16));
  SA_TRY(check_tensor(fn, "k_v", k_v, true, 16));
  SA_TRY(check_tensor(fn, "q_v", q_v, false, 16));
  SA_TRY(check_tensor(fn, "k_a", k_a, false, 16));
  SA_TRY(check_tensor(fn, "lse_a", lse_a, true, 4));
  SA_TRY(check_tensor(fn, "lse_v", lse_v, false, 4));
  SA_TRY(check_tensor(fn, "sal_v_tok", sal_v_tok, false, 4));
  SA_TRY(check_tensor(fn, "sal_v_blk", sal_v_blk, true, 4));
  SA_TRY(check_tensor(fn, "sal_a_tok", sal_a_tok, false, 4));
  SA_TRY(check_ws(fn, ws, ws_bytes, sa::cross_ws_layout(B, H, L_v, L_a).total));
  sa::launch_cross_scores_from_lse_bf16(
      static_cast<const uint16_t*>(q_a), static_cast<const uint16_t*>(k_v),
      static_cast<const uint16_t*>(q_v), static_cast<const uint16_t*>(k_a), lse_a, lse_v, B, H,
      L_v, L_a, d, scale, block, sal_v_tok, sal_v_blk, sal_a_tok, accumulate, nullptr, nullptr,
      static_cast<char*>(ws), static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

int sa_pool_columns(int n_b) {
  if (n_b < 1 || n_b > sa::kMaxBlocks) return 0;
  return sa::mask_n_pad(n_b);
}

int sa_cross_scores_pooled(const void* q_a, const void* k_v, const void* q_v, const void* k_a,
                           const float* lse_a, const float* lse_v, int B, int H, int L_v,
                           int L_a, int d, int dtype, float scale, int block, float* sal_v_tok,
                           float* sal_v_blk, float* sal_a_tok, int accumulate, double* qbar,
                           double* kbar, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sa_cross_scores_pooled";
  SA_TRY(check_common(fn, B, H, L_v, d, dtype, scale, block));
  if (L_a < 1) return fail(SA_ERR_INVALID_ARG, "%s: L_a=%d must be >= 1", fn, L_a);
  if (accumulate != 0 && accumulate != 1)
    return fail(SA_ERR_INVALID_ARG, "%s: accumulate=%d must be 0 or 1", fn, accumulate);
  const bool from_lse = lse_a != nullptr;
  if ((lse_v != nullptr) != from_lse)
    return fail(SA_ERR_INVALID_ARG, "%s: lse_a and lse_v must be both NULL or both non-NULL",
                fn);
  if (from_lse && dtype != SA_BF16)
    return fail(SA_ERR_UNSUPPORTED, "%s: the LSE form takes SA_BF16 inputs only", fn);
  SA_TRY(check_tensor(fn, "q_a", q_a, true, 16));
  SA_TRY(check_tensor(fn, "k_v", k_v, true, 16));
  SA_TRY(check_tensor(fn, "q_v", q_v, true, 16));
  SA_TRY(check_tensor(fn, "k_a", k_a, true, 16));
  SA_TRY(check_tensor(fn, "lse_a", lse_a, false, 4));
  SA_TRY(check_tensor(fn, "lse_v", lse_v, false, 4));
  SA_TRY(check_tensor(fn, "sal_v_tok", sal_v_tok, false, 4));
  SA_TRY(check_tensor(fn, "sal_v_blk", sal_v_blk, true, 4));
  SA_TRY(check_tensor(fn, "sal_a_tok", sal_a_tok, true, 4));
  SA_TRY(check_tensor(fn, "qbar", qbar, true, 8));
  SA_TRY(check_tensor(fn, "kbar", kbar, true, 8));
  const size_t nmean = static_cast<size_t>(B) * H * d * sa::mask_n_pad(sa::ceil_div(L_v, block));
  if (qbar < kbar + nmean && kbar < qbar + nmean)
    return fail(SA_ERR_INVALID_ARG, "%s: qbar and kbar overlap (each holds %zu doubles)", fn,
                nmean);
  SA_TRY(check_ws(fn, ws, ws_bytes, sa::cross_ws_layout(B, H, L_v, L_a).total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  const uint16_t* qa16 = static_cast<const uint16_t*>(q_a);
  const uint16_t* kv16 = static_cast<const uint16_t*>(k_v);
  const uint16_t* qv16 = static_cast<const uint16_t*>(q_v);
  const uint16_t* ka16 = static_cast<const uint16_t*>(k_a);
  if (from_lse) {
    sa::launch_cross_scores_from_lse_bf16(qa16, kv16, qv16, ka16, lse_a, lse_v, B, H, L_v, L_a,
                                          d, scale, block, sal_v_tok, sal_v_blk, sal_a_tok,
                                          accumulate, qbar, kbar, w, s);
  } else if (dtype == SA_BF16) {
    sa::launch_cross_scores_bf16(qa16, kv16, qv16, ka16, B, H, L_v, L_a, d, scale, block,
                                 sal_v_tok, sal_v_blk, sal_a_tok, accumulate, qbar, kbar, w, s);
  } else {  // the fp32 correctness path pools in a pass of its own
    sa::launch_cross_scores_f32(
        static_cast<const float*>(q_a), static_cast<const float*>(k_v),
        static_cast<const float*>(q_v), static_cast<const float*>(k_a), B, H, L_v, L_a, d,
        scale, block, sal_v_tok, sal_v_blk, sal_a_tok, accumulate, w, s);
    sa::launch_block_pool(q_v, k_v, B, H, L_v, d, dtype, block, qbar, kbar, s);
  }
  return check_launch(fn);
}

int sa_cross_attention(const void* q, const void* k, const void* v, void* o, float* lse,
                       int B, int H, int Lq, int Lk, int d, int dtype, float scale, void* ws,
                       size_t ws_bytes, void* stream) {
  const char* fn = "sa_cross_attention";
  SA_TRY(check_common(fn, B, H, Lk, d, dtype, scale, 128));
  if (dtype != SA_BF16)
    return fail(SA_ERR_UNSUPPORTED, "%s: only SA_BF16 inputs are supported", fn);
  if (Lq < 1 || Lq > sa::kMaxTokens)
    return fail(SA_ERR_INVALID_ARG, "%s: Lq=%d outside [1, %d]", fn, Lq, sa::kMaxTokens);
  SA_TRY(check_tensor(fn, "q", q, true, 16));
  SA_TRY(check_tensor(fn, "k", k, true, 16));
  SA_TRY(check_tensor(fn, "v", v, true, 16));
  SA_TRY(check_tensor(fn, "o", o, true, 16));
  SA_TRY(check_tensor(fn, "lse", lse, false, 4));
  SA_TRY(check_ws(fn, ws, ws_bytes, sa::token_attn_ws_bytes(B, H, Lk, d, Lq)));
  sa::launch_cross_attention_bf16(static_cast<const uint16_t*>(q),
                                  static_cast<const uint16_t*>(k),
                                  static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o),
                                  lse, B, H, Lq, Lk, d, scale, static_cast<char*>(ws),
                                  static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

int sa_select_protected(const float* sal_blk, int B, int n_b, int k_prot,
                        int32_t* prot_idx, uint8_t* prot_flag, void* stream) {
  const char* fn = "sa_select_protected";
  if (B < 1 || n_b < 1)
    return fail(SA_ERR_INVALID_ARG, "%s: B=%d n_b=%d must be >= 1", fn, B, n_b);
  if (n_b > sa::kMaxBlocks)
    return fail(SA_ERR_UNSUPPORTED, "%s: n_b=%d exceeds %d", fn, n_b, sa::kMaxBlocks);
  if (k_prot < 0 || k_prot > n_b)
    return fail(SA_ERR_INVALID_ARG, "%s: k_prot=%d outside [0, n_b=%d]", fn, k_prot, n_b);
  SA_TRY(check_tensor(fn, "sal_blk", sal_blk, true, 4));
  SA_TRY(check_tensor(fn, "prot_idx", prot_idx, false, 4));
  SA_TRY(check_tensor(fn, "prot_flag", prot_flag, true, 1));
  sa::launch_select_protected(sal_blk, B, n_b, k_prot, prot_idx, prot_flag,
                              static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

int sa_build_block_mask(const void* q_v, const void* k_v, int B, int H, int L_v, int d,
                        int dtype, float scale, int block, int k_keep,
                        const uint8_t* prot_flag, int32_t* kv_idx, int32_t* kv_cnt,
                        uint8_t* mask, float* scores, void* ws, size_t ws_bytes,
                        void* stream) {
  const char* fn = "sa_build_block_mask";
  SA_TRY(check_common(fn, B, H, L_v, d, dtype, scale, block));
  const int n_b = sa::ceil_div(L_v, block);
  if (k_keep < 1 || k_keep > n_b)
    return fail(SA_ERR_INVALID_ARG, "%s: k_keep=%d outside [1, n_b=%d]", fn, k_keep, n_b);
  SA_TRY(check_tensor(fn, "q_v", q_v, true, 16));
  SA_TRY(check_tensor(fn, "k_v", k_v, true, 16));
  SA_TRY(check_tensor(fn, "prot_flag", prot_flag, false, 1));
  SA_TRY(check_tensor(fn, "kv_idx", kv_idx, true, 4));
  SA_TRY(check_tensor(fn, "kv_cnt", kv_cnt, true, 4));
  SA_TRY(check_tensor(fn, "mask", mask, false, 1));
  SA_TRY(check_tensor(fn, "scores", scores, false, 4));
  SA_TRY(check_ws(fn, ws, ws_bytes, sa::mask_ws_layout(B, H, n_b, d).total));
  sa::launch_build_block_mask(q_v, k_v, B, H, L_v, d, dtype, scale, block, k_keep,
                              prot_flag, kv_idx, kv_cnt, mask, scores,
                              static_cast<char*>(ws), static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

int sa_build_block_mask_pooled(const double* qbar, const double* kbar, int B, int H, int L_v,
                               int d, float scale, int block, int k_keep,
                               const uint8_t* prot_flag, int32_t* kv_idx, int32_t* kv_cnt,
                               uint8_t* mask, float* scores, void* stream) {
  const char* fn = "sa_build_block_mask_pooled";
  SA_TRY(check_common(fn, B, H, L_v, d, SA_BF16, scale, block));
  const int n_b = sa::ceil_div(L_v, block);
  if (k_keep < 1 || k_keep > n_b)
    return fail(SA_ERR_INVALID_ARG, "%s: k_keep=%d outside [1, n_b=%d]", fn, k_keep, n_b);
  SA_TRY(check_tensor(fn, "qbar", qbar, true, 8));
  SA_TRY(check_tensor(fn, "kbar", kbar, true, 8));
  SA_TRY(check_tensor(fn, "prot_flag", prot_flag, false, 1));
  SA_TRY(check_tensor(fn, "kv_idx", kv_idx, true, 4));
  SA_TRY(check_tensor(fn, "kv_cnt", kv_cnt, true, 4));
  SA_TRY(check_tensor(fn, "mask", mask, false, 1));
  SA_TRY(check_tensor(fn, "scores", scores, false, 4));
  sa::launch_mask_from_means(qbar, kbar, B, H, L_v, d, scale, block, k_keep, prot_flag, kv_idx,
                             kv_cnt, mask, scores, static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

int sa_sparse_attention(const void* q, const void* k, const void* v, void* o, float* lse,
                        int B, int H, int L, int d, int dtype, float scale, int block,
                        const int32_t* kv_idx, const int32_t* kv_cnt, void* ws,
                        size_t ws_bytes, void* stream) {
  const char* fn = "sa_sparse_attention";
  SA_TRY(check_sparse_attention_args(fn, q, k, v, o, lse, B, H, L, d, dtype, scale, block,
                                     kv_idx, kv_cnt));
  const int n_b = sa::ceil_div(L, block);
  SA_TRY(check_ws(fn, ws, ws_bytes, sa::attn_ws_layout(B, H, n_b, d, block).total));
  launch_sparse_attention(q, k, v, o, lse, B, H, L, d, dtype, scale, block, kv_idx, kv_cnt,
                          static_cast<char*>(ws), static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

int sa_sparse_attention_noalloc(const void* q, const void* k, const void* v, void* o,
                                float* lse, int B, int H, int L, int d, int dtype, float scale,
                                int block, const int32_t* kv_idx, const int32_t* kv_cnt,
                                void* stream) {
  const char* fn = "sa_sparse_attention_noalloc";
  SA_TRY(check_sparse_attention_args(fn, q, k, v, o, lse, B, H, L, d, dtype, scale, block,
                                     kv_idx, kv_cnt));
  const int n_b = sa::ceil_div(L, block);
  const size_t need = sa::attn_ws_layout(B, H, n_b, d, block).total;
  if (need > kStaticScratchBytes)
    return fail(SA_ERR_UNSUPPORTED,
                "%s: B=%d H=%d n_b=%d needs %zu bytes of scratch, above the %zu bytes the "
                "library holds per device; call sa_sparse_attention with a workspace "
                "instead", fn, B, H, n_b, need, kStaticScratchBytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = nullptr;
  SA_TRY(static_scratch(fn, s, &ws));
  launch_sparse_attention(q, k, v, o, lse, B, H, L, d, dtype, scale, block, kv_idx, kv_cnt,
                          ws, s);
  return check_launch(fn);
}

int sa_saliency_ema(float* sal_bar, const float* sal, size_t n, float alpha, void* stream) {
  const char* fn = "sa_saliency_ema";
  if (!(alpha >= 0.f && alpha <= 1.f))
    return fail(SA_ERR_INVALID_ARG, "%s: alpha=%g outside [0, 1]", fn,
                static_cast<double>(alpha));
  SA_TRY(check_tensor(fn, "sal_bar", sal_bar, true, 4));
  SA_TRY(check_tensor(fn, "sal", sal, true, 4));
  if (sal != sal_bar && sal < sal_bar + n && sal_bar < sal + n)
    return fail(SA_ERR_INVALID_ARG, "%s: sal and sal_bar overlap without being equal", fn);
  if (n == 0) return ok();
  sa::launch_saliency_ema(sal_bar, sal, n, alpha, static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

int sa_select_protected_tokens(const float* sal_tok, int B, int L, int k_tok,
                               int32_t* tok_idx, uint8_t* tok_flag, void* stream) {
  const char* fn = "sa_select_protected_tokens";
  if (B < 1 || L < 1) return fail(SA_ERR_INVALID_ARG, "%s: B=%d L=%d must be >= 1", fn, B, L);
  if (L > sa::kMaxTokens)
    return fail(SA_ERR_UNSUPPORTED, "%s: L=%d exceeds %d", fn, L, sa::kMaxTokens);
  if (k_tok < 0 || k_tok > L)
    return fail(SA_ERR_INVALID_ARG, "%s: k_tok=%d outside [0, L=%d]", fn, k_tok, L);
  if (tok_idx == nullptr && tok_flag == nullptr)
    return fail(SA_ERR_INVALID_ARG, "%s: tok_idx and tok_flag are both NULL", fn);
  SA_TRY(check_tensor(fn, "sal_tok", sal_tok, true, 4));
  SA_TRY(check_tensor(fn, "tok_idx", tok_idx, false, 4));
  SA_TRY(check_tensor(fn, "tok_flag", tok_flag, false, 1));
  sa::launch_select_protected_tokens(sal_tok, B, L, k_tok, tok_idx, tok_flag,
                                     static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

int sa_protected_token_attention(const void* q, const void* k, const void* v, void* o,
                                 float* lse, int B, int H, int L, int d, int dtype,
                                 float scale, const int32_t* tok_idx, int k_tok, void* ws,
                                 size_t ws_bytes, void* stream) {
  const char* fn = "sa_protected_token_attention";
  SA_TRY(check_common(fn, B, H, L, d, dtype, scale, 128));
  if (k_tok < 0 || k_tok > L)
    return fail(SA_ERR_INVALID_ARG, "%s: k_tok=%d outside [0, L=%d]", fn, k_tok, L);
  SA_TRY(check_tensor(fn, "q", q, true, 16));
  SA_TRY(check_tensor(fn, "k", k, true, 16));
  SA_TRY(check_tensor(fn, "v", v, true, 16));
  SA_TRY(check_tensor(fn, "o", o, true, 16));
  SA_TRY(check_tensor(fn, "lse", lse, false, 4));
  SA_TRY(check_tensor(fn, "tok_idx", tok_idx, k_tok > 0, 4));
  SA_TRY(check_ws(fn, ws, ws_bytes, sa::token_attn_ws_bytes(B, H, L, d, k_tok)));
  if (k_tok == 0) return ok();
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == SA_BF16)
    sa::launch_protected_token_attention_bf16(
        static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
        static_cast<const uint16_t*>(v), static_cast<uint16_t*>(o), lse, B, H, L, d, scale,
        tok_idx, k_tok, static_cast<char*>(ws), s);
  else
    sa::launch_protected_token_attention_f32(
        static_cast<const float*>(q), static_cast<const float*>(k),
        static_cast<const float*>(v), static_cast<float*>(o), lse, B, H, L, d, scale,
        tok_idx, k_tok, s);
  return check_launch(fn);
}

int sa_cache_indicator(const void* y_v, const void* y_v_hat, const uint8_t* prot_flag,
                       const void* y_a, const void* y_a_hat, const float* s_bar,
                       const float* s_hat, int B, int L_v, int L_a, int C, int dtype,
                       float lambda_p, float lambda_s, float tau, float eps, float* out,
                       void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "sa_cache_indicator";
  if (B < 1 || L_v < 1)
    return fail(SA_ERR_INVALID_ARG, "%s: B=%d L_v=%d must be >= 1", fn, B, L_v);
  if (dtype != SA_BF16 && dtype != SA_F32)
    return fail(SA_ERR_UNSUPPORTED, "%s: dtype %d is neither SA_BF16 nor SA_F32", fn, dtype);
  if (C < 8 || C % 8 != 0)
    return fail(SA_ERR_INVALID_ARG, "%s: C=%d must be >= 8 and a multiple of 8", fn, C);
  if ((y_a == nullptr) != (y_a_hat == nullptr))
    return fail(SA_ERR_INVALID_ARG, "%s: y_a and y_a_hat must be both NULL or both non-NULL",
                fn);
  if (y_a != nullptr && L_a < 1)
    return fail(SA_ERR_INVALID_ARG, "%s: L_a=%d must be >= 1 with audio outputs", fn, L_a);
  if ((s_bar == nullptr) != (s_hat == nullptr))
    return fail(SA_ERR_INVALID_ARG, "%s: s_bar and s_hat must be both NULL or both non-NULL",
                fn);
  if (!(lambda_p >= 0.f) || !isfinite(lambda_p) || !(lambda_s >= 0.f) || !isfinite(lambda_s) ||
      !isfinite(tau) || !(eps >= 0.f) || !isfinite(eps))
    return fail(SA_ERR_INVALID_ARG,
                "%s: lambda_p=%g lambda_s=%g must be finite and >= 0, tau=%g finite, "
                "eps=%g finite and >= 0", fn, static_cast<double>(lambda_p),
                static_cast<double>(lambda_s), static_cast<double>(tau),
                static_cast<double>(eps));
  SA_TRY(check_tensor(fn, "y_v", y_v, true, 16));
  SA_TRY(check_tensor(fn, "y_v_hat", y_v_hat, true, 16));
  SA_TRY(check_tensor(fn, "prot_flag", prot_flag, false, 1));
  SA_TRY(check_tensor(fn, "y_a", y_a, false, 16));
  SA_TRY(check_tensor(fn, "y_a_hat", y_a_hat, false, 16));
  SA_TRY(check_tensor(fn, "s_bar", s_bar, false, 4));
  SA_TRY(check_tensor(fn, "s_hat", s_hat, false, 4));
  SA_TRY(check_tensor(fn, "out", out, true, 4));
  const int la = y_a != nullptr ? L_a : 0;
  // a workgroup indexes its span of 16-byte chunks with 32 bits
  const size_t cpr = static_cast<size_t>(C) / (dtype == SA_BF16 ? 8 : 4);
  const size_t rv = static_cast<size_t>(B) * L_v, ra = static_cast<size_t>(B) * la;
  const size_t wv = sa::cache_workgroups_video(rv), wa = sa::cache_workgroups_audio(ra);
  if ((rv + wv - 1) / wv * cpr > 0xffffffffull ||
      (wa > 0 && (ra + wa - 1) / wa * cpr > 0xffffffffull))
    return fail(SA_ERR_INVALID_ARG, "%s: B=%d L_v=%d L_a=%d C=%d is too large", fn, B, L_v,
                la, C);
  SA_TRY(check_ws(fn, ws, ws_bytes, sa::cache_ws_bytes(B, L_v, la)));
  sa::launch_cache_indicator(y_v, y_v_hat, prot_flag, y_a, y_a_hat, s_bar, s_hat, B, L_v, la,
                             C, dtype, lambda_p, lambda_s, tau, eps, out,
                             static_cast<char*>(ws), static_cast<hipStream_t>(stream));
  return check_launch(fn);
}

}  // extern "C"
