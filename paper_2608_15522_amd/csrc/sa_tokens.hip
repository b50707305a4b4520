// Token-granular protection (Sec. 4.1 Eq. (3)/(8) at token level) and the
// lagged saliency update (Eq. (4)).
//
// K8 saliency_ema: s_bar = alpha * s_bar + (1 - alpha) * s, elementwise fp32.
// K9 select_tokens: per batch item one workgroup (one wave up to L = 2048,
//    else 1024 threads) finds the k_tok-th smallest value key T (saliency
//    descending) of the L tokens by a radix search: the bits that every key
//    shares are decided by one AND/OR
//    reduction, then each step decides two bits from the key counts of the
//    prefix group per digit (DPP wave sums, one barrier with alternating LDS
//    slots), until one key is left in the group.  Tokens tied at T are taken
//    in index order.  Each wave owns a contiguous range of tokens (in
//    registers up to L = 32768), read 64 consecutive tokens at a time,
//    so ballot prefix counts and one scan of the per-wave totals write the
//    kept tokens in ascending order.  Once the prefix group holds at most
//    16384 keys they are copied to LDS and later steps scan only them.
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
constexpr int kTokCand = 16384;  // LDS candidates once the prefix group fits

// Exclusive prefix of `v` over the workgroup (NW waves) in thread order, and
// the total.  Ends with a barrier after the LDS slots are read.
template <int NW>
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
  for (int w = 0; w < NW; ++w) {
    const int t = wave_tot[w];
    if (w < wave) base += t;
    total += t;
  }
  __syncthreads();
  return base + incl - v;
}

// Exclusive prefix over the NW waves of a per-wave value (given by every
// lane of the wave); ends with a barrier after the LDS slots are read.
template <int NW>
__device__ __forceinline__ int wave_exclusive_base(int v, int* wave_tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_tot[wave] = v;
  __syncthreads();
  int base = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w)
    if (w < wave) base += wave_tot[w];
  __syncthreads();
  return base;
}

// The order key of a token is its value key: the fp32 saliency mapped to a
// monotone integer and inverted, so that a larger saliency is a smaller key.
// The k_tok-th smallest value key T is found first; tokens with a key below T
// are kept, and of the tokens whose key equals T the lowest indices fill the
// remaining places (larger saliency first, then lower index).
// NT threads (NW = NT/64 waves); wave w owns the tokens [w*S, (w+1)*S),
// S = ceil(L/NW); lane l holds tokens w*S + 64 j + l.  R > 0: the keys stay
// in registers (64 R >= S); R == 0: they are read from global memory on
// every pass.  Only the 1024-thread form copies candidates to LDS.
template <int R, int NT>
__global__ void __launch_bounds__(NT)
select_tokens_kernel(const float* __restrict__ sal, int L, int k_tok,
                     int32_t* __restrict__ tok_idx, uint8_t* __restrict__ tok_flag) {
  constexpr int NW = NT / 64;
  constexpr bool kCompact = NW > 1;
  __shared__ uint32_t cand[kCompact ? kTokCand : 1];
  __shared__ uint32_t cnt_sh[2][NW][4];
  __shared__ uint32_t red_sh[NW][2];
  __shared__ int wave_tot[NW];
  const int b = blockIdx.x;
  const float* s = sal + static_cast<size_t>(b) * L;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int S = ceil_div(L, NW);
  const int w0 = min(wave * S, L), w1 = min(w0 + S, L);
  const int J = R > 0 ? R : ceil_div(S, 64);
  const uint64_t lanes_below = (1ull << lane) - 1ull;

  constexpr int RR = R > 0 ? R : 1;
  uint32_t vk[RR];
  if constexpr (R > 0) {
    // unconditional loads at a clamped index, so that all of them are in
    // flight at once
    float x[R];
#pragma unroll
    for (int j = 0; j < R; ++j) x[j] = s[min(w0 + 64 * j + lane, L - 1)];
#pragma unroll
    for (int j = 0; j < R; ++j) vk[j] = w0 + 64 * j + lane < w1 ? ~float_order_key(x[j]) : 0u;
  }
  // f(key, token, valid) for j = 0 .. J-1, the same j on every lane
  auto for_all = [&](auto f) {
    if constexpr (R > 0) {
#pragma unroll
      for (int j = 0; j < R; ++j) {
        const int i = w0 + 64 * j + lane;
        f(vk[j], i, i < w1);
      }
    } else {
      for (int j = 0; j < J; ++j) {
        const int i = w0 + 64 * j + lane;
        const bool ok = i < w1;
        const float x = s[min(i, L - 1)];
        f(ok ? ~float_order_key(x) : 0u, i, ok);
      }
    }
  };
  auto for_keys = [&](auto f) {
    for_all([&](uint32_t key, int, bool ok) {
      if (ok) f(key);
    });
  };

  // Search for T, for 0 < k_tok < L.  `fixed` marks the decided bits of T,
  // `prefix` their values; `below` keys lie under the prefix group and
  // `size` keys share it.  k_tok == L keeps every token, k_tok == 0 none.
  uint32_t prefix = 0, fixed = 0;
  int below = 0, size = L;
  if (k_tok > 0 && k_tok < L) {
    // bits that every key shares are decided at once
    uint32_t a = 0xffffffffu, o = 0u;
    for_keys([&](uint32_t key) { a &= key; o |= key; });
    a = __reduce_and_sync(~0ull, a);
    o = __reduce_or_sync(~0ull, o);
    if (lane == 0) {
      red_sh[wave][0] = a;
      red_sh[wave][1] = o;
    }
    __syncthreads();
    a = 0xffffffffu;
    o = 0u;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      a &= red_sh[w][0];
      o |= red_sh[w][1];
    }
    const uint32_t diff = a ^ o;
    int hb = diff != 0u ? 31 - __clz(diff) : -1;  // highest undecided bit
    fixed = hb >= 0 ? ~static_cast<uint32_t>((2ull << hb) - 1ull) : 0xffffffffu;
    prefix = a & fixed;
    bool in_lds = false;
    int n_cand = 0;
    // two bits per step: count the keys of the prefix group by digit
    for (int step = 0; hb >= 0 && size > 1; ++step) {
      if (kCompact && !in_lds && size <= kTokCand) {
        // the group's keys go to LDS and later steps scan only them
        int mine_c = 0;
        for_keys([&](uint32_t key) { mine_c += (key & fixed) == prefix; });
        int tot = 0;
        int at = block_exclusive_scan<NW>(mine_c, wave_tot, tot);
        for_keys([&](uint32_t key) {
          if ((key & fixed) == prefix) cand[at++] = key;
        });
        __syncthreads();
        in_lds = true;
        n_cand = size;
      }
      const int lo = hb > 0 ? hb - 1 : 0;
      uint32_t c0 = 0u, c1 = 0u, c2 = 0u;
      auto count = [&](uint32_t key) {
        const bool in = (key & fixed) == prefix;
        const uint32_t dg = (key >> lo) & 3u;
        c0 += in && dg == 0u;
        c1 += in && dg == 1u;
        c2 += in && dg == 2u;
      };
      if (in_lds) {
        // all slots of this thread at once; reads stay inside `cand`
        constexpr int U = kCompact ? kTokCand / NT : 1;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int i = tid + u * NT;
          const uint32_t key = cand[min(i, kTokCand - 1)];
          if (i < n_cand) count(key);
        }
      } else {
        for_keys(count);
      }
      c0 = __reduce_add_sync(~0ull, c0);
      c1 = __reduce_add_sync(~0ull, c1);
      c2 = __reduce_add_sync(~0ull, c2);
      if (lane == 0) {
        cnt_sh[step & 1][wave][0] = c0;
        cnt_sh[step & 1][wave][1] = c1;
        cnt_sh[step & 1][wave][2] = c2;
      }
      __syncthreads();
      int n0 = 0, n1 = 0, n2 = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        n0 += static_cast<int>(cnt_sh[step & 1][w][0]);
        n1 += static_cast<int>(cnt_sh[step & 1][w][1]);
        n2 += static_cast<int>(cnt_sh[step & 1][w][2]);
      }
      uint32_t dsel;
      if (below + n0 >= k_tok) {
        dsel = 0u;
        size = n0;
      } else if (below + n0 + n1 >= k_tok) {
        dsel = 1u;
        below += n0;
        size = n1;
      } else if (below + n0 + n1 + n2 >= k_tok) {
        dsel = 2u;
        below += n0 + n1;
        size = n2;
      } else {
        dsel = 3u;
        size -= n0 + n1 + n2;
        below += n0 + n1 + n2;
      }
      const uint32_t width = hb > 0 ? 3u : 1u;
      fixed |= width << lo;
      prefix |= dsel << lo;
      hb = lo - 1;
    }
  }
  // size > 1 here only if every bit is decided: `size` keys equal T, and the
  // k_tok - below lowest-index ones among them are kept
  const bool ties = k_tok > 0 && k_tok < L && size > 1;
  const int need = k_tok - below;
  auto is_tie = [&](uint32_t key, bool ok) { return ties && ok && key == prefix; };
  auto kept = [&](uint32_t key, bool ok, int tie_rank) {
    if (!ok || k_tok == 0) return false;
    if (k_tok == L) return true;
    if (!ties) return (key & fixed) <= prefix;
    return key < prefix || (key == prefix && tie_rank < need);
  };
  // tokens before this wave's range that tie at T, and that are kept
  int tie_wave = 0;
  if (ties) {  // uniform over the workgroup
    for_all([&](uint32_t key, int, bool ok) { tie_wave += __popcll(__ballot(is_tie(key, ok))); });
  }
  const int tie_base = ties ? wave_exclusive_base<NW>(tie_wave, wave_tot) : 0;
  int kept_wave = 0;
  {
    int tr = tie_base;
    for_all([&](uint32_t key, int, bool ok) {
      const uint64_t tb = __ballot(is_tie(key, ok));
      const bool on = kept(key, ok, tr + __popcll(tb & lanes_below));
      tr += __popcll(tb);
      kept_wave += __popcll(__ballot(on));
    });
  }
  int pos = wave_exclusive_base<NW>(kept_wave, wave_tot);
  int32_t* out = tok_idx != nullptr ? tok_idx + static_cast<size_t>(b) * k_tok : nullptr;
  uint8_t* flag = tok_flag != nullptr ? tok_flag + static_cast<size_t>(b) * L : nullptr;
  int tr = tie_base;
  for_all([&](uint32_t key, int i, bool ok) {
    const uint64_t tb = __ballot(is_tie(key, ok));
    const bool on = kept(key, ok, tr + __popcll(tb & lanes_below));
    tr += __popcll(tb);
    const uint64_t kb = __ballot(on);
    const int p = pos + __popcll(kb & lanes_below);
    pos += __popcll(kb);
    // exactly k_tok tokens are kept; the bound only keeps the writes inside
    // tok_idx whatever the input values are
    if (on && out != nullptr && p < k_tok) out[p] = i;
    if (ok && flag != nullptr) flag[i] = on ? 1 : 0;
  });
}

}  // namespace

void launch_saliency_ema(float* s_bar, const float* s, size_t n, float alpha, hipStream_t st) {
  const size_t blocks = n / 256 + 1 < 4096 ? n / 256 + 1 : 4096;
  hipLaunchKernelGGL(saliency_ema_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     st, s_bar, s, n, alpha);
}

void launch_select_protected_tokens(const float* sal_tok, int B, int L, int k_tok,
                                    int32_t* tok_idx, uint8_t* tok_flag, hipStream_t st) {
  const dim3 grid(B);
#define SA_SELECT(R, NT)                                                                 \
  hipLaunchKernelGGL((select_tokens_kernel<R, NT>), grid, dim3(NT), 0, st, sal_tok, L, k_tok, \
                     tok_idx, tok_flag)
  if (L <= 512) {  // one wave: tokens per lane ceil(L/64)
    SA_SELECT(8, 64);
  } else if (L <= 2048) {
    SA_SELECT(32, 64);
  } else {  // 16 waves: tokens per lane ceil(ceil(L/16)/64)
    const int J = ceil_div(ceil_div(L, 16), 64);
    if (J <= 4)
      SA_SELECT(4, 1024);
    else if (J <= 16)
      SA_SELECT(16, 1024);
    else if (J <= 32)
      SA_SELECT(32, 1024);
    else
      SA_SELECT(0, 1024);
  }
#undef SA_SELECT
}

}  // namespace sa
