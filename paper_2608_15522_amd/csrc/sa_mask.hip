// Protected selection and the protected block mask.
//
// K4 select_protected (Sec. 4.2, Eq. (8) at block granularity): per batch
//    item one workgroup sorts the block saliencies in LDS with a bitonic
//    network on 64-bit keys (value descending, index ascending) and takes
//    the first k_prot.
// K5 block_pool: per (b,h, block) the mean of Q and of K over the valid
//    tokens of the block, accumulated in fp64 (16-byte loads, fixed-order LDS
//    reduction); the sums of bf16/fp32 inputs are exact.
// K6 mask_build (Sec. 4.2, Eq. (6) and (9)): per (b,h) and up to 8 query
//    blocks, the pooled scores G = scale * qbar kbar^T by fp64 FMA (a few
//    hundred MFLOP per layer; fp32 would misrank scores closer than ~1e-6,
//    and pooled-score gaps are that small), then per row either the full list
//    (protected row) or the top-k_keep of an LDS bitonic sort of the row's
//    keys, compacted into an ascending list with a workgroup prefix sum.
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
constexpr int kMaskThreads = 256;
constexpr int kRowsPerWg = 8;  // upper bound of the rows handled per workgroup

// Rows per workgroup so that the per-row key arrays take at most 32 KB.
inline int mask_rows_per_wg(int n_pad) {
  const int r = 4096 / n_pad;
  return r < 1 ? 1 : (r > kRowsPerWg ? kRowsPerWg : r);
}

// Dynamic LDS: keys[rows][n_pad] u64 | qbar rows [rows][D] f64 |
// sel[n_pad] u8 | scan[kMaskThreads] i32.
template <int D>
__global__ void __launch_bounds__(kMaskThreads)
mask_build_kernel(const double* __restrict__ qbar, const double* __restrict__ kbar,
                  const uint8_t* __restrict__ prot_flag, int H, int n_b,
                  int n_pad, int rows, int k_keep, double scale,
                  int32_t* __restrict__ kv_idx, int32_t* __restrict__ kv_cnt,
                  uint8_t* __restrict__ mask, float* __restrict__ scores) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint64_t* keys_all = reinterpret_cast<uint64_t*>(smem);
  double* qs = reinterpret_cast<double*>(keys_all + static_cast<size_t>(rows) * n_pad);
  uint8_t* sel = reinterpret_cast<uint8_t*>(qs + rows * D);
  int* scan = reinterpret_cast<int*>(sel + ((n_pad + 15) & ~15));

  const int tid = threadIdx.x;
  const size_t pair = blockIdx.y;
  const int b = static_cast<int>(pair / H);
  const int r0 = blockIdx.x * rows;
  const int nr = min(rows, n_b - r0);
  const double* qb = qbar + pair * n_b * D;
  const double* kb = kbar + pair * n_b * D;

  for (int e = tid; e < nr * D; e += kMaskThreads) qs[e] = qb[static_cast<size_t>(r0) * D + e];
  __syncthreads();
  // pooled scores in fp64, one key block per thread, d-sequential FMA; the
  // sort keys of every row and the optional fp32 copy of G are written here
  for (int col = tid; col < n_pad; col += kMaskThreads) {
    if (col >= n_b) {
      for (int rr = 0; rr < nr; ++rr) keys_all[rr * n_pad + col] = ~0ull;
      continue;
    }
    double acc[kRowsPerWg];
#pragma unroll
    for (int rr = 0; rr < kRowsPerWg; ++rr) acc[rr] = 0.0;
    const double* kr = kb + static_cast<size_t>(col) * D;
    for (int e = 0; e < D; ++e) {
      const double kv = kr[e];
#pragma unroll
      for (int rr = 0; rr < kRowsPerWg; ++rr)
        if (rr < nr) acc[rr] = fma(qs[rr * D + e], kv, acc[rr]);
    }
#pragma unroll
    for (int rr = 0; rr < kRowsPerWg; ++rr) {
      if (rr < nr) {
        const double gval = acc[rr] * scale;
        keys_all[rr * n_pad + col] = desc_double_asc_index_key(gval, static_cast<uint32_t>(col));
        if (scores != nullptr)
          scores[(pair * n_b + r0 + rr) * n_b + col] = static_cast<float>(gval);
      }
    }
  }
  __syncthreads();

  const int per = ceil_div(n_b, kMaskThreads);  // entries per thread in the scan
  for (int rr = 0; rr < nr; ++rr) {
    const int r = r0 + rr;
    const size_t row = pair * n_b + r;
    const bool prot = prot_flag != nullptr && prot_flag[static_cast<size_t>(b) * n_b + r] != 0;
    int32_t* out_idx = kv_idx + row * n_b;
    if (prot) {
      for (int col = tid; col < n_b; col += kMaskThreads) {
        out_idx[col] = col;
        if (mask != nullptr) mask[row * n_b + col] = 1;
      }
      if (tid == 0) kv_cnt[row] = n_b;
      continue;  // uniform across the workgroup
    }
    uint64_t* keys = keys_all + static_cast<size_t>(rr) * n_pad;
    for (int i = tid; i < n_pad; i += kMaskThreads) sel[i] = 0;
    bitonic_sort_lds(keys, n_pad);
    for (int i = tid; i < k_keep; i += kMaskThreads)
      sel[static_cast<uint32_t>(keys[i] & 0xfffu)] = 1;
    __syncthreads();
    // exclusive prefix count of sel over ascending column index
    const int lo = tid * per, hi = min(lo + per, n_b);
    int local = 0;
    for (int i = lo; i < hi; ++i) local += sel[i];
    scan[tid] = local;
    __syncthreads();
    for (int off = 1; off < kMaskThreads; off <<= 1) {
      const int v = tid >= off ? scan[tid - off] : 0;
      __syncthreads();
      scan[tid] += v;
      __syncthreads();
    }
    int pos = scan[tid] - local;
    for (int i = lo; i < hi; ++i) {
      if (sel[i]) out_idx[pos++] = i;
    }
    for (int i = k_keep + tid; i < n_b; i += kMaskThreads) out_idx[i] = -1;
    if (mask != nullptr)
      for (int col = tid; col < n_b; col += kMaskThreads) mask[row * n_b + col] = sel[col];
    if (tid == 0) kv_cnt[row] = k_keep;
    __syncthreads();
  }
}

}  // namespace

size_t mask_build_lds_bytes(int n_b, int d) {
  const int n_pad = next_pow2(n_b);
  const int rows = mask_rows_per_wg(n_pad);
  size_t off = sizeof(uint64_t) * static_cast<size_t>(rows) * n_pad;
  off += sizeof(double) * rows * d;
  off += (n_pad + 15) & ~15;
  off += sizeof(int) * kMaskThreads;
  return off;
}

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
  const int n_pad = next_pow2(n_b);
  const size_t lds = mask_build_lds_bytes(n_b, d);
  const int rows = mask_rows_per_wg(n_pad);
  const dim3 mgrid(ceil_div(n_b, rows), P);
  const double sc = static_cast<double>(scale);
  if (d == 128)
    hipLaunchKernelGGL(mask_build_kernel<128>, mgrid, dim3(kMaskThreads), lds, s, qbar,
                       kbar, prot_flag, H, n_b, n_pad, rows, k_keep, sc, kv_idx,
                       kv_cnt, mask, scores);
  else
    hipLaunchKernelGGL(mask_build_kernel<64>, mgrid, dim3(kMaskThreads), lds, s, qbar,
                       kbar, prot_flag, H, n_b, n_pad, rows, k_keep, sc, kv_idx,
                       kv_cnt, mask, scores);
}

}  // namespace sa
