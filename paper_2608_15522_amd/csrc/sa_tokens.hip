// Token-granular protection (Sec. 4.1 Eq. (3)/(8) at token level) and the
// lagged saliency update (Eq. (4)).
//
// K8 saliency_ema: s_bar = alpha * s_bar + (1 - alpha) * s, elementwise fp32.
// K9 select_tokens: per batch item one 1024-thread workgroup finds the
//    k_tok-th smallest order key (value descending, index ascending) of the
//    L token saliencies by a bitwise search from the top bit: each step counts
//    the keys under the fixed prefix (per-thread count, wave sum, one barrier
//    with alternating LDS slots) and stops once a single key shares the
//    prefix.  Thread t owns tokens [t*C, (t+1)*C), C = ceil(L/1024), so an
//    exclusive scan of the per-thread counts in thread order writes the kept
//    tokens in ascending order.
// The dense attention rows of the protected tokens are the gather variant of
// the attention kernel (sa_attn.hip).
#include "sa_device.h"
#include "sa_internal.h"

namespace sa {
namespace {

// ---- K8 ---------------------------------------------------------------------
__global__ void __launch_bounds__(256)
saliency_ema_kernel(float* __restrict__ s_bar, const float* __restrict__ s, size_t n,
                    float alpha) {
  const float beta = 1.0f - alpha;
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += static_cast<size_t>(gridDim.x) * blockDim.x)
    s_bar[i] = fmaf(alpha, s_bar[i], beta * s[i]);
}

// ---- K9 ---------------------------------------------------------------------
constexpr int kTokThreads = 1024;
constexpr int kTokWaves = kTokThreads / 64;
constexpr int kTokRegs = 32;  // tokens per thread kept in registers (L <= 32768)

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Exclusive prefix of `v` over the workgroup in thread order, and the total.
// Ends with a barrier after the LDS slots are read.
__device__ __forceinline__ int block_exclusive_scan(int v, int* wave_tot, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(incl, o, 64);
    if (lane >= o) incl += u;
  }
  if (lane == 63) wave_tot[wave] = incl;
  __syncthreads();
  int base = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kTokWaves; ++w) {
    const int t = wave_tot[w];
    if (w < wave) base += t;
    total += t;
  }
  __syncthreads();
  return base + incl - v;
}

template <bool REGS>
__global__ void __launch_bounds__(kTokThreads)
select_tokens_kernel(const float* __restrict__ sal, int L, int k_tok,
                     int32_t* __restrict__ tok_idx, uint8_t* __restrict__ tok_flag) {
  __shared__ int cnt_sh[2][kTokWaves];
  __shared__ int wave_tot[kTokWaves];
  const int b = blockIdx.x;
  const float* s = sal + static_cast<size_t>(b) * L;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = ceil_div(L, kTokThreads);
  const int i0 = min(tid * C, L), i1 = min(i0 + C, L);

  // value part of the order key: larger saliency -> smaller key
  uint32_t vk[REGS ? kTokRegs : 1];
  if constexpr (REGS) {
#pragma unroll
    for (int j = 0; j < kTokRegs; ++j) vk[j] = i0 + j < i1 ? ~float_order_key(s[i0 + j]) : 0u;
  }
  auto key_of = [&](int j) -> uint64_t {  // token i0 + j (< i1)
    const uint32_t v = REGS ? vk[REGS ? j : 0] : ~float_order_key(s[i0 + j]);
    return (static_cast<uint64_t>(v) << 32) | static_cast<uint32_t>(i0 + j);
  };
  auto count_under = [&](uint64_t sel, uint64_t prefix) {
    int c = 0;
    if constexpr (REGS) {
#pragma unroll
      for (int j = 0; j < kTokRegs; ++j) c += (i0 + j < i1) && ((key_of(j) & sel) == prefix);
    } else {
      for (int j = 0; j < i1 - i0; ++j) c += (key_of(j) & sel) == prefix;
    }
    return c;
  };

  // 0 < k_tok < L: keep <=> (key & fixed) <= prefix once the search ends;
  // k_tok == L keeps every token and k_tok == 0 none (no search)
  uint64_t prefix = 0, fixed = 0;
  if (k_tok > 0 && k_tok < L) {
    int below = 0, size = L;
    for (int bit = 63, step = 0; bit >= 0 && size > 1; --bit, ++step) {
      const uint64_t sel = fixed | (1ull << bit);
      const int c = wave_sum(count_under(sel, prefix));
      if (lane == 0) cnt_sh[step & 1][wave] = c;
      __syncthreads();
      int cnt = 0;
#pragma unroll
      for (int w = 0; w < kTokWaves; ++w) cnt += cnt_sh[step & 1][w];
      if (below + cnt < k_tok) {
        below += cnt;
        size -= cnt;
        prefix |= 1ull << bit;
      } else {
        size = cnt;
      }
      fixed = sel;
    }
  }
  auto kept = [&](int j) {
    if (k_tok == 0) return false;
    if (k_tok == L) return true;
    return (key_of(j) & fixed) <= prefix;
  };

  int mine = 0;
  if constexpr (REGS) {
#pragma unroll
    for (int j = 0; j < kTokRegs; ++j) mine += (i0 + j < i1) && kept(j);
  } else {
    for (int j = 0; j < i1 - i0; ++j) mine += kept(j);
  }
  int total = 0;
  int pos = block_exclusive_scan(mine, wave_tot, total);
  int32_t* out = tok_idx != nullptr ? tok_idx + static_cast<size_t>(b) * k_tok : nullptr;
  uint8_t* flag = tok_flag != nullptr ? tok_flag + static_cast<size_t>(b) * L : nullptr;
  for (int j = 0; j < i1 - i0; ++j) {
    const bool on = kept(j);
    // exactly k_tok keys are kept (the keys are distinct); the bound only
    // keeps the writes inside tok_idx whatever the input values are
    if (on && out != nullptr && pos < k_tok) out[pos++] = i0 + j;
    if (flag != nullptr) flag[i0 + j] = on ? 1 : 0;
  }
}

}  // namespace

void launch_saliency_ema(float* s_bar, const float* s, size_t n, float alpha, hipStream_t st) {
  const size_t blocks = n / 256 + 1 < 4096 ? n / 256 + 1 : 4096;
  hipLaunchKernelGGL(saliency_ema_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     st, s_bar, s, n, alpha);
}

void launch_select_protected_tokens(const float* sal_tok, int B, int L, int k_tok,
                                    int32_t* tok_idx, uint8_t* tok_flag, hipStream_t st) {
  if (L <= kTokThreads * kTokRegs)
    hipLaunchKernelGGL(select_tokens_kernel<true>, dim3(B), dim3(kTokThreads), 0, st, sal_tok,
                       L, k_tok, tok_idx, tok_flag);
  else
    hipLaunchKernelGGL(select_tokens_kernel<false>, dim3(B), dim3(kTokThreads), 0, st,
                       sal_tok, L, k_tok, tok_idx, tok_flag);
}

}  // namespace sa
