// Protected selection and the protected block mask.
//
// K4 select_protected (Sec. 4.2, Eq. (8) at block granularity): per batch
//    item one workgroup sorts the block saliencies in LDS with a bitonic
//    network on 64-bit keys (value descending, index ascending) and takes
//    the first k_prot.
// K5 block_pool: per (b,h) and 8 consecutive blocks the mean of Q and of K
//    over the valid tokens of each block, accumulated in fp64 (16-byte loads,
//    fixed-order LDS reduction; the sums are exact, see block_pool_kernel),
//    stored as [d][n_pad] (block index innermost).
// K6 mask_build (Sec. 4.2, Eq. (6) and (9)): per (b,h) and 16 query blocks
//    (rows padded to 64 * E columns, E <= 10; 8 or 4 blocks for wider
//    rows), the pooled scores G = scale * qbar kbar^T in fp64, on the
//    matrix cores (v_mfma_f64_16x16x4f64) up to 640 columns and by vector
//    FMAs beyond (a few GFLOP per layer; fp32 would misrank scores closer
//    than ~1e-6, and pooled-score gaps are that small), then per row
//    either the full list (protected row) or the top-k_keep blocks: one
//    wave bounds the k-th smallest order key (value descending, index
//    ascending) by halving a key range, counting with ballots, and compacts
//    the blocks below the bound into an ascending list.
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

constexpr int kMaxPoolBlock = 128;  // largest supported block

// Grid (ceil(n_b / kPoolBlocks), P), 256 threads.  out[pair][:][c] (layout
// [d][n_pad]) = mean of the rows of block c, in fp64: a sum of at most 128
// values is exact in fp64 whenever their magnitudes lie within 2^44 (bf16
// inputs, 8 significant bits) or 2^28 (fp32, 24 bits) of each other, so the
// result does not depend on the order of the additions, and the mean is
// rounded once.  Per block, thread
// (rg, cc) loads 16-byte chunk cc of rows rg, rg + RG, ... of both matrices
// and the RG partial sums of each element are added in a fixed order; the
// means of the workgroup's blocks are written as runs of consecutive
// columns.
constexpr int kPoolBlocks = 8;  // blocks per block_pool workgroup

template <typename T, int D>
__global__ void __launch_bounds__(256)
block_pool_kernel(const T* __restrict__ q, const T* __restrict__ k,
                  double* __restrict__ qbar, double* __restrict__ kbar, int L,
                  int block, int n_b, int n_pad) {
  constexpr int EPC = Elem<T>::kPer16B;       // elements per 16-byte chunk
  constexpr int CPR = D / EPC;                // chunks per row
  constexpr int RG = 256 / CPR;               // row groups
  constexpr int NR = kMaxPoolBlock / RG;      // rows per thread, at most
  __shared__ double part[2][RG][EPC][CPR];    // element e of chunk cc: consecutive cc
  __shared__ double mean[2][D][kPoolBlocks];
  const int c0 = blockIdx.x * kPoolBlocks;
  const size_t pair = blockIdx.y;
  const int nblk = min(kPoolBlocks, n_b - c0);
  const int cc = threadIdx.x % CPR, rg = threadIdx.x / CPR;
  // One block in registers at a time: at 110 VGPRs three workgroups share a
  // CU (as many as the LDS holds) and hide each other's loads; a second
  // buffer for block j+1 took 174 VGPRs, two workgroups per CU, and left the
  // 768-workgroup Ovi-like grid 1.5 rounds long (90 against 81 us).
  auto load_block = [&](int j, u32x4 (&dst)[2][NR]) {
    const int row0 = (c0 + j) * block;
    const int len = j < nblk ? min(block, L - row0) : 0;
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      const T* src = (which == 0 ? q : k) + pair * L * D;
#pragma unroll
      for (int i = 0; i < NR; ++i) {
        const int r = rg + RG * i;
        dst[which][i] = r < len ? ldg16_nt(src + static_cast<size_t>(row0 + r) * D + cc * EPC)
                                : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  u32x4 raw[2][NR];
  for (int j = 0; j < nblk; ++j) {
    const int row0 = (c0 + j) * block;
    const int len = min(block, L - row0);
    load_block(j, raw);
    __syncthreads();  // the previous block's partial sums have been read
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      double acc[EPC];
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[e] = 0.0;
#pragma unroll
      for (int i = 0; i < NR; ++i) {
        if (rg + RG * i >= len) break;
        double v[EPC];
        Elem<T>::unpack(raw[which][i], v);
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[e] += v[e];
      }
#pragma unroll
      for (int e = 0; e < EPC; ++e) part[which][rg][e][cc] = acc[e];
    }
    __syncthreads();
    for (int t = threadIdx.x; t < 2 * D; t += 256) {
      const int which = t / D, dd = t % D;
      double sum = 0.0;
      for (int i = 0; i < RG; ++i) sum += part[which][i][dd % EPC][dd / EPC];
      mean[which][dd][j] = sum / static_cast<double>(len);
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t < 2 * D * kPoolBlocks; t += 256) {
    const int j = t % kPoolBlocks, dd = (t / kPoolBlocks) % D, which = t / (kPoolBlocks * D);
    if (j < nblk) {
      double* dst = (which == 0 ? qbar : kbar);
      dst[(pair * D + dd) * n_pad + c0 + j] = mean[which][dd][j];
    }
  }
}

// ---- K6 ---------------------------------------------------------------------
// Row widths up to 640 columns compute G on the matrix cores
// (v_mfma_f64_16x16x4f64, fp64 products and sums like the vector path);
// wider rows use fp64 FMAs on the vector ALUs.
__host__ __device__ constexpr bool mask_uses_mfma(int E) { return E <= 10; }

// Waves per mask workgroup.  Matrix-core path: 16 up to 384 columns (one
// row per wave in the selection; at <= 64 VGPRs two workgroups fill a CU's
// 32 wave slots), 8 for 512 and 640 columns, which with at most 113 VGPRs
// lets two 16-row workgroups of 64-80 KB share a CU (at 5 waves and 144
// VGPRs a CU held one, and the n_b = 591 mask took 290 instead of 205 us; at
// 8 waves 153 us, at 16 waves, one workgroup per CU, 205 us).  Vector path:
// a divisor of E from 4 up, so that every wave computes the scores of as
// many 64-column groups; 4 when E has no such divisor up to 6.
__host__ __device__ constexpr int mask_waves(int E) {
  return mask_uses_mfma(E) ? (E <= 6 ? 16 : 8)
                           : (E % 4 == 0 ? 4 : (E % 5 == 0 ? 5 : (E % 6 == 0 ? 6 : 4)));
}

// Query-block rows per mask workgroup: 16 on the matrix-core path (its tile
// height; the rows of G fill at most 80 KB of LDS); on the vector path 8,
// and 4 from n_pad = 1280 on, where the rows would not fit otherwise.
__host__ __device__ constexpr int mask_rows_per_wg(int E) {
  return mask_uses_mfma(E) ? 16 : (E >= 20 ? 4 : 8);
}

// Bound of the k smallest (1 <= k <= number of real keys) of the E x 64 keys
// held by one wave (E per lane): returns T such that exactly k keys are < T.
// Real keys are distinct; padding keys are ~0 and never below a real one.
// The search halves a key range [lo, lo + 2^w) that holds the k-th smallest
// key: one compare per key against the midpoint, counted with ballots, tells
// which half holds it.  It stops once the range holds that key alone.
template <int E>
__device__ __forceinline__ uint64_t wave_kth_bound(const uint64_t* keys, int k) {
  uint64_t lo = 0;
  int below = 0, size = 64 * E;  // keys below lo / in the range
  int w = 64;
  do {
    --w;
    const uint64_t mid = lo | (1ull << w);
    int cnt = 0;  // keys below mid
#pragma unroll
    for (int e = 0; e < E; ++e) cnt += __popcll(__ballot(keys[e] < mid));
    if (cnt < k) {
      size -= cnt - below;
      below = cnt;
      lo = mid;
    } else {
      size = cnt - below;
    }
  } while (w > 0 && size > 1);
  return lo + (1ull << w);
}

typedef double f64x4 __attribute__((ext_vector_type(4)));

// Buffer resource over n_bytes from base (gfx9 raw buffer, bounds-checked:
// loads past n_bytes return 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const double* base, int n_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<double*>(base), 0, n_bytes, 0x00020000);
}
__device__ __forceinline__ double buffer_load_f64(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}

// 1-D grid of 8 * ceil(P / 8) * ceil(n_b / R) workgroups of mask_waves(E)
// waves; template E = n_pad / 64.  Workgroup w runs on XCD w % 8
// (round-robin dispatch) and takes (b,h) pair (w % 8) + 8 * ((w / 8) / nrt)
// and row tile (w / 8) % nrt, so all tiles of a pair share one XCD's L2
// (workgroups past P exit).  Pooled means are [d][n_pad] per (b,h).
// Phase 1, the rows r0 .. r0+R-1 of G = scale * qbar kbar^T into LDS:
//  * matrix-core path (R = 16): wave w takes the pairs of 16-column tiles
//    w, w+W, ...; per 4 d-steps one A fragment (query means) and one B
//    fragment per tile come from global memory, PD steps ahead, and each
//    tile takes one v_mfma_f64_16x16x4f64 (n_pad / 16 tiles in all).
//  * vector path: the workgroup's query means are copied to LDS as [d][R];
//    wave w takes the 64-column groups w, w+W, ..., one column per lane: the
//    lane's key means are loaded KP d-steps ahead and each feeds R fp64 FMAs
//    whose query operands are broadcast LDS reads.
// Rows >= n_b and columns >= n_b hold padding and are discarded.  Phase 2:
// wave w takes rows w, w+W, ... with column col = 64*e + lane in register e
// of lane `lane`, and either emits the full list (protected row) or the
// top-k_keep blocks.
template <int D, int E>
__global__ void __launch_bounds__(64 * mask_waves(E)) __attribute__((amdgpu_waves_per_eu(4)))
mask_build_kernel(const double* __restrict__ qbar, const double* __restrict__ kbar,
                  const uint8_t* __restrict__ prot_flag, int H, int n_b, int k_keep,
                  double scale, int32_t* __restrict__ kv_idx, int32_t* __restrict__ kv_cnt,
                  uint8_t* __restrict__ mask, float* __restrict__ scores, int P) {
  constexpr int NPAD = 64 * E;
  constexpr bool MF = mask_uses_mfma(E);
  constexpr int R = mask_rows_per_wg(E);
  constexpr int kMaskWaves = mask_waves(E);
  constexpr int kMaskThreads = 64 * kMaskWaves;
  // rows of G, then (vector path) the query means as [d][R]
  __shared__ __attribute__((aligned(16))) double lds[R * NPAD + (MF ? 0 : D * R)];
  double(*gs)[NPAD] = reinterpret_cast<double(*)[NPAD]>(lds);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nrt = ceil_div(n_b, R);
  const int wg = blockIdx.x;
  const int pair_i = (wg % 8) + 8 * ((wg / 8) / nrt);
  if (pair_i >= P) return;  // uniform: the whole workgroup exits
  const size_t pair = static_cast<size_t>(pair_i);
  const int b = pair_i / H;
  const int r0 = ((wg / 8) % nrt) * R;
  const double* qp = qbar + pair * D * NPAD + r0;
  const double* kp = kbar + pair * D * NPAD;
  const __amdgpu_buffer_rsrc_t krs = buffer_rsrc(kp, D * NPAD * 8);

  if constexpr (MF) {
    // A[i][kk] (query block r0+i, d = 4k+kk) sits in lane i + 16kk, B[kk][j]
    // (d = 4k+kk, key block c0+j) in lane j + 16kk, and D[i][j] in lane
    // j + 16(i % 4), element i / 4.
    const __amdgpu_buffer_rsrc_t qrs = buffer_rsrc(qp, (D * NPAD - r0) * 8);
    const int lo = lane & 15, hi = lane >> 4;
    const int frag = (hi * NPAD + lo) * 8;  // byte offset of the lane's element in a 4-d slab
    constexpr int KS = D / 4;               // k-steps
    constexpr int PD = 4;                   // k-steps of fragments in flight
    constexpr int TG = 2;                   // 16-column tiles per pass of a wave
    constexpr int T = NPAD / 16;
    constexpr int NG = T / TG;
#pragma unroll 1
    for (int g = wave; g < NG; g += kMaskWaves) {
      const int c0 = 16 * TG * g;
      f64x4 acc[TG];
#pragma unroll
      for (int t = 0; t < TG; ++t) acc[t] = f64x4{0.0, 0.0, 0.0, 0.0};
      double aq[PD], bq[PD][TG];
      auto load_ab = [&](int k) {
        aq[k % PD] = buffer_load_f64(qrs, frag, 4 * k * NPAD * 8);
#pragma unroll
        for (int t = 0; t < TG; ++t)
          bq[k % PD][t] = buffer_load_f64(krs, frag + (c0 + 16 * t) * 8, 4 * k * NPAD * 8);
      };
#pragma unroll
      for (int p = 0; p < PD; ++p) load_ab(p);
#pragma unroll
      for (int k = 0; k < KS; ++k) {
#pragma unroll
        for (int t = 0; t < TG; ++t)
          acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(aq[k % PD], bq[k % PD][t], acc[t], 0, 0, 0);
        if (k + PD < KS) load_ab(k + PD);
      }
#pragma unroll
      for (int t = 0; t < TG; ++t)
#pragma unroll
        for (int v = 0; v < 4; ++v) gs[hi + 4 * v][c0 + 16 * t + lo] = acc[t][v] * scale;
    }
  } else {
    constexpr int KP = 8;  // d-steps of key values in flight per lane
    static_assert(D % (2 * KP) == 0 && R % 2 == 0, "chunking");
    double(*qs)[R] = reinterpret_cast<double(*)[R]>(lds + R * NPAD);
    for (int i = tid; i < D * R; i += kMaskThreads) qs[i / R][i % R] = qp[(i / R) * NPAD + i % R];
    __syncthreads();
#pragma unroll 1
    for (int cg = wave; cg < E; cg += kMaskWaves) {
      const int col = 64 * cg + lane;
      double acc[R];
#pragma unroll
      for (int i = 0; i < R; ++i) acc[i] = 0.0;
      // key values of chunk c (KP d-steps) alternate between ka and kb
      auto load_chunk = [&](double* kv, int c) {
#pragma unroll
        for (int j = 0; j < KP; ++j) kv[j] = buffer_load_f64(krs, col * 8, (c * KP + j) * NPAD * 8);
      };
      // The FMAs of each d-step are pinned before the query reads of the
      // next: left free, the compiler hoisted every LDS read of two chunks
      // above their FMAs and spilled them.
      auto use_chunk = [&](const double* kv, int c) {
#pragma unroll
        for (int j = 0; j < KP; ++j) {
          const double* qrow = qs[c * KP + j];
#pragma unroll
          for (int i = 0; i < R; i += 2) {
            const double2 qq = *reinterpret_cast<const double2*>(qrow + i);
            acc[i] = fma(qq.x, kv[j], acc[i]);
            acc[i + 1] = fma(qq.y, kv[j], acc[i + 1]);
          }
#pragma unroll
          for (int i = 0; i < R; ++i) asm volatile("" : "+v"(acc[i])::"memory");
        }
      };
      double ka[KP], kb[KP];
      load_chunk(ka, 0);
#pragma unroll 1
      for (int c = 0; c < D / KP; c += 2) {
        load_chunk(kb, c + 1);
        use_chunk(ka, c);
        if (c + 2 < D / KP) load_chunk(ka, c + 2);
        use_chunk(kb, c + 1);
      }
#pragma unroll
      for (int i = 0; i < R; ++i) gs[i][col] = acc[i] * scale;
    }
  }
  __syncthreads();

  const uint64_t below_mask = (1ull << lane) - 1ull;
  for (int i = wave; i < R; i += kMaskWaves) {
    const int r = r0 + i;
    if (r >= n_b) break;  // uniform across the wave
    const size_t row = pair * n_b + r;
    int32_t* out_idx = kv_idx + row * n_b;
    uint64_t keys[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int col = 64 * e + lane;
      const double gval = col < n_b ? gs[i][col] : 0.0;
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
    const uint64_t bound = wave_kth_bound<E>(keys, k_keep);
    int base = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int col = 64 * e + lane;
      const bool on = keys[e] < bound;  // padding keys (~0) never pass
      const uint64_t m = __ballot(on);
      if (on) out_idx[base + __popcll(m & below_mask)] = col;
      base += __popcll(m);
      if (mask != nullptr && col < n_b) mask[row * n_b + col] = on ? 1 : 0;
    }
    for (int j = k_keep + lane; j < n_b; j += 64) out_idx[j] = -1;
    if (lane == 0) kv_cnt[row] = k_keep;
  }
}

template <int D>
void launch_mask_build(int E, dim3 grid, hipStream_t s, const double* qbar,
                       const double* kbar, const uint8_t* prot_flag, int P, int H, int n_b,
                       int k_keep, double sc, int32_t* kv_idx, int32_t* kv_cnt,
                       uint8_t* mask, float* scores) {
#define SA_MASK_CASE(EV)                                                                 \
  case EV:                                                                               \
    hipLaunchKernelGGL((mask_build_kernel<D, EV>), grid, dim3(64 * mask_waves(EV)), 0, s,  \
                       qbar,                                                              \
                       kbar, prot_flag, H, n_b, k_keep, sc, kv_idx, kv_cnt, mask, scores, \
                       P);                                                                \
    break;
  switch (E) {
    SA_MASK_CASE(1)
    SA_MASK_CASE(2)
    SA_MASK_CASE(3)
    SA_MASK_CASE(4)
    SA_MASK_CASE(5)
    SA_MASK_CASE(6)
    SA_MASK_CASE(8)
    SA_MASK_CASE(10)
    SA_MASK_CASE(12)
    SA_MASK_CASE(16)
    SA_MASK_CASE(20)
    SA_MASK_CASE(24)
    SA_MASK_CASE(32)
    default: break;
  }
#undef SA_MASK_CASE
}


}  // namespace

void launch_select_protected(const float* sal_blk, int B, int n_b, int k_prot,
                             int32_t* prot_idx, uint8_t* prot_flag,
                             hipStream_t s) {
  const int n_pad = next_pow2(n_b);
  hipLaunchKernelGGL(select_protected_kernel, dim3(B), dim3(1024), 0, s, sal_blk, n_b,
                     k_prot, n_pad, prot_idx, prot_flag);
}

void launch_block_pool(const void* q_v, const void* k_v, int B, int H, int L_v, int d,
                       int dtype, int block, double* qbar, double* kbar, hipStream_t s) {
  const int n_b = ceil_div(L_v, block);
  const int n_pad = mask_n_pad(n_b);
  const dim3 pgrid(ceil_div(n_b, kPoolBlocks), B * H);
  if (dtype == 0) {
    const uint16_t* q = static_cast<const uint16_t*>(q_v);
    const uint16_t* k = static_cast<const uint16_t*>(k_v);
    if (d == 128)
      hipLaunchKernelGGL((block_pool_kernel<uint16_t, 128>), pgrid, dim3(256), 0, s, q, k,
                         qbar, kbar, L_v, block, n_b, n_pad);
    else
      hipLaunchKernelGGL((block_pool_kernel<uint16_t, 64>), pgrid, dim3(256), 0, s, q, k,
                         qbar, kbar, L_v, block, n_b, n_pad);
  } else {
    const float* q = static_cast<const float*>(q_v);
    const float* k = static_cast<const float*>(k_v);
    if (d == 128)
      hipLaunchKernelGGL((block_pool_kernel<float, 128>), pgrid, dim3(256), 0, s, q, k,
                         qbar, kbar, L_v, block, n_b, n_pad);
    else
      hipLaunchKernelGGL((block_pool_kernel<float, 64>), pgrid, dim3(256), 0, s, q, k,
                         qbar, kbar, L_v, block, n_b, n_pad);
  }
}

void launch_mask_from_means(const double* qbar, const double* kbar, int B, int H, int L_v,
                            int d, float scale, int block, int k_keep,
                            const uint8_t* prot_flag, int32_t* kv_idx, int32_t* kv_cnt,
                            uint8_t* mask, float* scores, hipStream_t s) {
  const int n_b = ceil_div(L_v, block);
  const int P = B * H;
  const int E = mask_n_pad(n_b) / 64;
  const dim3 mgrid(8 * ceil_div(P, 8) * ceil_div(n_b, mask_rows_per_wg(E)));
  const double sc = static_cast<double>(scale);
  if (d == 128)
    launch_mask_build<128>(E, mgrid, s, qbar, kbar, prot_flag, P, H, n_b, k_keep, sc, kv_idx,
                           kv_cnt, mask, scores);
  else
    launch_mask_build<64>(E, mgrid, s, qbar, kbar, prot_flag, P, H, n_b, k_keep, sc, kv_idx,
                          kv_cnt, mask, scores);
}

void launch_build_block_mask(const void* q_v, const void* k_v, int B, int H,
                             int L_v, int d, int dtype, float scale, int block,
                             int k_keep, const uint8_t* prot_flag,
                             int32_t* kv_idx, int32_t* kv_cnt, uint8_t* mask,
                             float* scores, char* ws, hipStream_t s) {
  const MaskWs lay = mask_ws_layout(B, H, ceil_div(L_v, block), d);
  double* qbar = reinterpret_cast<double*>(ws + lay.qbar);
  double* kbar = reinterpret_cast<double*>(ws + lay.kbar);
  launch_block_pool(q_v, k_v, B, H, L_v, d, dtype, block, qbar, kbar, s);
  launch_mask_from_means(qbar, kbar, B, H, L_v, d, scale, block, k_keep, prot_flag, kv_idx,
                         kv_cnt, mask, scores, s);
}

}  // namespace sa
