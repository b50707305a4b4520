// Protected selection and the protected block mask.
//
// K4 select_protected (Sec. 4.2, Eq. (8) at block granularity): per batch
//    item one workgroup sorts the block saliencies in LDS with a bitonic
//    network on 64-bit keys (value descending, index ascending) and takes
//    the first k_prot.
// K5 block_pool: per (b,h, block) the mean of Q and of K over the valid
//    tokens of the block, accumulated in fp64 (16-byte loads, fixed-order LDS
//    reduction); the sums of bf16/fp32 inputs are exact.
// K6 mask_build (Sec. 4.2, Eq. (6) and (9)): per (b,h) and a group of query
//    blocks, the pooled scores G = scale * qbar kbar^T by fp64 FMA (a few
//    hundred MFLOP per layer; fp32 would misrank scores closer than ~1e-6,
//    and pooled-score gaps are that small), then per row either the full list
//    (protected row) or the top-k_keep blocks: one wave finds the k-th
//    smallest order key (value descending, index ascending) by a bitwise
//    search with ballots and compacts the blocks at or below it into an
//    ascending list.
#include "sa_device.h"
#include "sa_internal.h"

namespace sa {
namespace {

// ---- K4 ---------------------------------------------------------------------
__global__ void __launch_bounds__(1024)
select_protected_kernel(const float* __restrict__ sal_blk, int n_b, int k_prot,
                        int n_pad, int32_t* __restrict__ prot_idx,
                        uint8_t* __restrict__ prot_flag) {
  __shared__ uint64_t keys[kMaxBlocks];
  __shared__ uint8_t flag[kMaxBlocks];
  const int b = blockIdx.x;
  const float* s = sal_blk + static_cast<size_t>(b) * n_b;
  for (int i = threadIdx.x; i < n_pad; i += blockDim.x) {
    keys[i] = i < n_b ? desc_value_asc_index_key(s[i], static_cast<uint32_t>(i))
                      : ~0ull;
    if (i < n_b) flag[i] = 0;
  }
  bitonic_sort_lds(keys, n_pad);
  for (int i = threadIdx.x; i < k_prot; i += blockDim.x) {
    const uint32_t c = static_cast<uint32_t>(keys[i] & 0xffffffffu);
    flag[c] = 1;
    if (prot_idx != nullptr) prot_idx[static_cast<size_t>(b) * k_prot + i] = c;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < n_b; i += blockDim.x)
    prot_flag[static_cast<size_t>(b) * n_b + i] = flag[i];
}

// ---- K5 ---------------------------------------------------------------------
template <typename T> struct Elem;
template <> struct Elem<uint16_t> {
  static constexpr int kPer16B = 8;
  __device__ static void unpack(u32x4 v, double* out) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out[2 * i] = static_cast<double>(__uint_as_float(v[i] << 16));
      out[2 * i + 1] = static_cast<double>(__uint_as_float(v[i] & 0xffff0000u));
    }
  }
};
template <> struct Elem<float> {
  static constexpr int kPer16B = 4;
  __device__ static void unpack(u32x4 v, double* out) {
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = static_cast<double>(__uint_as_float(v[i]));
  }
};

// Grid (n_b, P), 256 threads.  out[pair][c][:] = mean of the rows of block c,
// in fp64: the sums of bf16 or fp32 inputs are exact, the mean is rounded
// once.
template <typename T, int D>
__global__ void __launch_bounds__(256)
block_pool_kernel(const T* __restrict__ q, const T* __restrict__ k,
                  double* __restrict__ qbar, double* __restrict__ kbar, int L,
                  int block) {
  constexpr int EPC = Elem<T>::kPer16B;       // elements per 16-byte chunk
  constexpr int CPR = D / EPC;                // chunks per row
  constexpr int RG = 256 / CPR;               // row groups
  __shared__ double part[RG][D];
  const int c = blockIdx.x;
  const size_t pair = blockIdx.y;
  const int n_b = gridDim.x;
  const int row0 = c * block;
  const int len = min(block, L - row0);
  const int cc = threadIdx.x % CPR, rg = threadIdx.x / CPR;
  for (int which = 0; which < 2; ++which) {
    const T* src = (which == 0 ? q : k) + pair * L * D;
    double acc[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[e] = 0.0;
    for (int r = rg; r < len; r += RG) {
      double v[EPC];
      Elem<T>::unpack(ldg16(src + static_cast<size_t>(row0 + r) * D + cc * EPC), v);
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[e] += v[e];
    }
#pragma unroll
    for (int e = 0; e < EPC; ++e) part[rg][cc * EPC + e] = acc[e];
    __syncthreads();
    if (threadIdx.x < D) {
      double sum = 0.0;
      for (int i = 0; i < RG; ++i) sum += part[i][threadIdx.x];
      double* dst = (which == 0 ? qbar : kbar);
      dst[(pair * n_b + c) * D + threadIdx.x] = sum / static_cast<double>(len);
    }
    __syncthreads();
  }
}

// ---- K6 ---------------------------------------------------------------------
constexpr int kMaskThreads = 256;  // 4 waves

// k-th smallest (1-based, 1 <= k <= number of keys) of the E x 64 keys held
// by one wave (E per lane), all distinct: bits are fixed from the top, each
// step counting the keys that share the fixed prefix and have a 0 next.
template <int E>
__device__ __forceinline__ uint64_t wave_kth_smallest(const uint64_t* keys, int k) {
  uint64_t prefix = 0;
  int below = 0;
  for (int bit = 63; bit >= 0; --bit) {
    const uint64_t hi = ~((2ull << bit) - 1ull);  // bits above `bit`
    const uint64_t sel = hi | (1ull << bit);
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) cnt += __popcll(__ballot((keys[e] & sel) == prefix));
    if (below + cnt < k) {
      below += cnt;
      prefix |= 1ull << bit;
    }
  }
  return prefix;
}

// Grid (ceil(n_b / ROWS), P), 256 threads; template E = n_pad / 64 (n_pad the
// next power of two >= n_b, at least 64).  Column col = 64*e + lane of a row
// lives in register e of lane `lane`.  Each wave owns RW rows.
template <int D, int E>
__global__ void __launch_bounds__(kMaskThreads)
mask_build_kernel(const double* __restrict__ qbar, const double* __restrict__ kbar,
                  const uint8_t* __restrict__ prot_flag, int H, int n_b, int k_keep,
                  double scale, int32_t* __restrict__ kv_idx, int32_t* __restrict__ kv_cnt,
                  uint8_t* __restrict__ mask, float* __restrict__ scores) {
  constexpr int NPAD = 64 * E;
  constexpr int RW = E >= 8 ? 1 : 8 / E;          // rows per wave
  constexpr int ROWS = 4 * RW;                     // rows per workgroup
  constexpr int DCH = (8192 / NPAD) < D ? (8192 / NPAD) : D;  // d values per 64 KB stage
  constexpr int KSS = NPAD + 1;                    // padded row: conflict-free stores
  constexpr int PER = DCH * NPAD / kMaskThreads;   // staged values per thread
  __shared__ double ks[DCH * KSS];
  __shared__ double qs[ROWS * D];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t pair = blockIdx.y;
  const int b = static_cast<int>(pair / H);
  const int r0 = blockIdx.x * ROWS;
  const double* qb = qbar + pair * n_b * D;
  const double* kb = kbar + pair * n_b * D;

  for (int i = tid; i < ROWS * D; i += kMaskThreads) {
    const int rr = i / D;
    qs[i] = r0 + rr < n_b ? qb[static_cast<size_t>(r0) * D + i] : 0.0;
  }
  double acc[RW][E];
#pragma unroll
  for (int rr = 0; rr < RW; ++rr)
#pragma unroll
    for (int e = 0; e < E; ++e) acc[rr][e] = 0.0;
  for (int d0 = 0; d0 < D; d0 += DCH) {
    // kbar[col][d0 .. d0+DCH) -> ks[dd][col]: every load of the stage is
    // issued before the first store (DCH consecutive threads read one row)
    double v[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = tid + kMaskThreads * j;
      const int col = i / DCH, dd = i % DCH;
      v[j] = col < n_b ? kb[static_cast<size_t>(col) * D + d0 + dd] : 0.0;
    }
    __syncthreads();  // the previous stage has been consumed
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = tid + kMaskThreads * j;
      ks[(i % DCH) * KSS + i / DCH] = v[j];
    }
    __syncthreads();
#pragma unroll 4
    for (int dd = 0; dd < DCH; ++dd) {
      double kv[E];
#pragma unroll
      for (int e = 0; e < E; ++e) kv[e] = ks[dd * KSS + 64 * e + lane];
#pragma unroll
      for (int rr = 0; rr < RW; ++rr) {
        const double qv = qs[(wave * RW + rr) * D + d0 + dd];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[rr][e] = fma(qv, kv[e], acc[rr][e]);
      }
    }
  }

  const uint64_t below_mask = (1ull << lane) - 1ull;
#pragma unroll
  for (int rr = 0; rr < RW; ++rr) {
    const int r = r0 + wave * RW + rr;
    if (r >= n_b) break;  // uniform across the wave
    const size_t row = pair * n_b + r;
    int32_t* out_idx = kv_idx + row * n_b;
    uint64_t keys[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int col = 64 * e + lane;
      const double gval = acc[rr][e] * scale;
      keys[e] = col < n_b ? desc_double_asc_index_key(gval, static_cast<uint32_t>(col)) : ~0ull;
      if (scores != nullptr && col < n_b) scores[row * n_b + col] = static_cast<float>(gval);
    }
    const bool prot = prot_flag != nullptr && prot_flag[static_cast<size_t>(b) * n_b + r] != 0;
    if (prot) {
      for (int col = lane; col < n_b; col += 64) {
        out_idx[col] = col;
        if (mask != nullptr) mask[row * n_b + col] = 1;
      }
      if (lane == 0) kv_cnt[row] = n_b;
      continue;
    }
    const uint64_t kth = wave_kth_smallest<E>(keys, k_keep);
    int base = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int col = 64 * e + lane;
      const bool on = keys[e] <= kth;  // padding keys (~0) are never at or below it
      const uint64_t m = __ballot(on);
      if (on) out_idx[base + __popcll(m & below_mask)] = col;
      base += __popcll(m);
      if (mask != nullptr && col < n_b) mask[row * n_b + col] = on ? 1 : 0;
    }
    for (int i = k_keep + lane; i < n_b; i += 64) out_idx[i] = -1;
    if (lane == 0) kv_cnt[row] = k_keep;
  }
}

template <int D>
void launch_mask_build(int E, dim3 grid, hipStream_t s, const double* qbar,
                       const double* kbar, const uint8_t* prot_flag, int H, int n_b,
                       int k_keep, double sc, int32_t* kv_idx, int32_t* kv_cnt,
                       uint8_t* mask, float* scores) {
#define SA_MASK_CASE(EV)                                                                 \
  case EV:                                                                               \
    hipLaunchKernelGGL((mask_build_kernel<D, EV>), grid, dim3(kMaskThreads), 0, s, qbar,  \
                       kbar, prot_flag, H, n_b, k_keep, sc, kv_idx, kv_cnt, mask, scores);  \
    break;
  switch (E) {
    SA_MASK_CASE(1)
    SA_MASK_CASE(2)
    SA_MASK_CASE(4)
    SA_MASK_CASE(8)
    SA_MASK_CASE(16)
    SA_MASK_CASE(32)
    default: break;
  }
#undef SA_MASK_CASE
}

inline int mask_rows_per_wg(int E) { return 4 * (E >= 8 ? 1 : 8 / E); }

}  // namespace

void launch_select_protected(const float* sal_blk, int B, int n_b, int k_prot,
                             int32_t* prot_idx, uint8_t* prot_flag,
                             hipStream_t s) {
  const int n_pad = next_pow2(n_b);
  hipLaunchKernelGGL(select_protected_kernel, dim3(B), dim3(1024), 0, s, sal_blk, n_b,
                     k_prot, n_pad, prot_idx, prot_flag);
}

void launch_build_block_mask(const void* q_v, const void* k_v, int B, int H,
                             int L_v, int d, int dtype, float scale, int block,
                             int k_keep, const uint8_t* prot_flag,
                             int32_t* kv_idx, int32_t* kv_cnt, uint8_t* mask,
                             float* scores, char* ws, hipStream_t s) {
  const int n_b = ceil_div(L_v, block);
  const int P = B * H;
  const MaskWs lay = mask_ws_layout(B, H, n_b, d);
  double* qbar = reinterpret_cast<double*>(ws + lay.qbar);
  double* kbar = reinterpret_cast<double*>(ws + lay.kbar);
  const dim3 pgrid(n_b, P);
  if (dtype == 0) {
    const uint16_t* q = static_cast<const uint16_t*>(q_v);
    const uint16_t* k = static_cast<const uint16_t*>(k_v);
    if (d == 128)
      hipLaunchKernelGGL((block_pool_kernel<uint16_t, 128>), pgrid, dim3(256), 0, s, q, k,
                         qbar, kbar, L_v, block);
    else
      hipLaunchKernelGGL((block_pool_kernel<uint16_t, 64>), pgrid, dim3(256), 0, s, q, k,
                         qbar, kbar, L_v, block);
  } else {
    const float* q = static_cast<const float*>(q_v);
    const float* k = static_cast<const float*>(k_v);
    if (d == 128)
      hipLaunchKernelGGL((block_pool_kernel<float, 128>), pgrid, dim3(256), 0, s, q, k,
                         qbar, kbar, L_v, block);
    else
      hipLaunchKernelGGL((block_pool_kernel<float, 64>), pgrid, dim3(256), 0, s, q, k,
                         qbar, kbar, L_v, block);
  }
  const int n_pad = next_pow2(n_b) < 64 ? 64 : next_pow2(n_b);
  const int E = n_pad / 64;
  const dim3 mgrid(ceil_div(n_b, mask_rows_per_wg(E)), P);
  const double sc = static_cast<double>(scale);
  if (d == 128)
    launch_mask_build<128>(E, mgrid, s, qbar, kbar, prot_flag, H, n_b, k_keep, sc, kv_idx,
                           kv_cnt, mask, scores);
  else
    launch_mask_build<64>(E, mgrid, s, qbar, kbar, prot_flag, H, n_b, k_keep, sc, kv_idx,
                          kv_cnt, mask, scores);
}

}  // namespace sa
