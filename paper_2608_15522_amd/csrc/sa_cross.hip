// Cross-modal saliency (Sec. 4.1, Eq. (1)-(2) and the reverse v->a
// direction).
//
// a->v: s^v_i = 1/(H*L_a) * sum_h sum_j softmax_i(scale * q^a_j . k^v_i).
//   K1 a2v_lse_partial : per (b,h, 1024-key chunk, 512-query slab) a 16-wave
//                        workgroup; wave w owns 32 audio queries and computes
//                        S^T = K^v Q^a^T tiles with bf16 MFMA, so a lane owns
//                        one audio query and keeps a lane-local online
//                        (max, sum) over its keys; partials go to workspace.
//   K1b lse_combine    : fixed-order merge of the chunk partials (log2 units).
//   K2 a2v_colmass     : per (b, 128 video keys, group of 4 heads) a 16-wave
//                        workgroup; wave w owns 32 audio queries and computes
//                        S = Q^a K^v^T so a lane owns one video key column and
//                        sums exp2(S*c - lse) over its rows, heads and query
//                        slabs; the 32 lane/wave partials per key are added
//                        in a fixed order.  No atomics: every output element
//                        has one writer, so results are reproducible.
//   K2b a2v_finalize   : sum over head groups, divide by H*L_a, block sums.
// v->a: s^a_j = 1/(H*L_v) * sum_h sum_i softmax_j(scale * q^v_i . k^a_j).
//   K3 v2a_colmass     : per (b,h, 512 video queries); pass 1 with S^T gives
//                        each video query its log-sum-exp (lane-local), pass 2
//                        recomputes S and reduces the column mass of every
//                        64-key audio tile across the workgroup.
//   K3b v2a_chunk_sum  : fixed-order sum over video chunks per head, then
//       v2a_finalize   : fixed-order sum over heads, / (H*L_v).
// fp32 inputs use plain per-thread kernels with the same outputs.
#include "sa_device.h"
#include "sa_internal.h"

namespace sa {
namespace {

constexpr int kCT = 64;  // keys per LDS tile in K1/K3

// Load a [64 x D] bf16 tile (rows >= row_end zero-filled) into swizzled LDS
// with all threads of the workgroup.  Row r, 16-byte chunk cc lands at chunk
// cc ^ (r & (CPR-1)).
template <int D, int NT>
__device__ __forceinline__ void load_rows_to_regs(const uint16_t* base, int row0,
                                                  int row_end, u32x4* reg) {
  constexpr int CPR = D / 8;
  constexpr int CH = (kCT * CPR + NT - 1) / NT;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int qq = threadIdx.x + NT * i;
    const int row = qq / CPR, cc = qq % CPR;
    reg[i] = (qq < kCT * CPR && row0 + row < row_end)
                 ? ldg16(base + static_cast<size_t>(row0 + row) * D + cc * 8)
                 : u32x4{0u, 0u, 0u, 0u};
  }
}
template <int D, int NT>
__device__ __forceinline__ void store_rows_to_lds(uint16_t* lds, const u32x4* reg) {
  constexpr int CPR = D / 8;
  constexpr int CH = (kCT * CPR + NT - 1) / NT;
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int qq = threadIdx.x + NT * i;
    if (qq < kCT * CPR) {
      const int row = qq / CPR, cc = qq % CPR;
      stg16(lds + row * D + ((cc ^ (row & (CPR - 1))) * 8), reg[i]);
    }
  }
}
// Operand fragment of row `row` (of a swizzled [rows x D] LDS tile) for k-step kc.
template <int D>
__device__ __forceinline__ u32x4 lds_frag(const uint16_t* lds, int row, int kc, int g) {
  constexpr int CPR = D / 8;
  const int ch = 2 * kc + g;
  return *reinterpret_cast<const u32x4*>(lds + row * D + ((ch ^ (row & (CPR - 1))) * 8));
}

template <int D>
__device__ __forceinline__ void load_qfrag(const uint16_t* base, int row, int nrows,
                                           int g, u32x4* qf) {
#pragma unroll
  for (int kc = 0; kc < D / 16; ++kc)
    qf[kc] = row < nrows ? ldg16(base + static_cast<size_t>(row) * D + 16 * kc + 8 * g)
                         : u32x4{0u, 0u, 0u, 0u};
}

// ---- K1 ---------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(1024)
a2v_lse_partial_kernel(const uint16_t* __restrict__ q_a,
                       const uint16_t* __restrict__ k_v,
                       float2* __restrict__ part, int L_v, int L_a, int nchunk,
                       float c) {
  constexpr int NT = 1024, KC = D / 16;
  constexpr int CH = (kCT * (D / 8) + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][kCT * D];
  const int chunk = blockIdx.x, slab = blockIdx.y, pair = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 5, n = lane & 31;
  const int j = slab * kQSlab + wave * 32 + n;
  const bool wave_on = slab * kQSlab + wave * 32 < L_a;
  const int key_begin = chunk * kLseChunk;
  const int key_end = min(key_begin + kLseChunk, L_v);
  const int ntiles = ceil_div(key_end - key_begin, kCT);
  const uint16_t* kh = k_v + static_cast<size_t>(pair) * L_v * D;

  u32x4 qf[KC];
  load_qfrag<D>(q_a + static_cast<size_t>(pair) * L_a * D, j, L_a, g, qf);
  float m = -INFINITY, l = 0.f;
  u32x4 reg[CH];
  load_rows_to_regs<D, NT>(kh, key_begin, key_end, reg);
  store_rows_to_lds<D, NT>(Ks[0], reg);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int key0 = key_begin + t * kCT;
    if (t + 1 < ntiles) load_rows_to_regs<D, NT>(kh, key0 + kCT, key_end, reg);
    if (wave_on) {
      f32x16 s0 = zero16(), s1 = zero16();
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        s0 = mfma32x32x16(lds_frag<D>(Ks[buf], n, kc, g), qf[kc], s0);
        s1 = mfma32x32x16(lds_frag<D>(Ks[buf], 32 + n, kc, g), qf[kc], s1);
      }
      if (key0 + kCT > key_end) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          if (key0 + crow(i, g) >= key_end) s0[i] = -INFINITY;
          if (key0 + 32 + crow(i, g) >= key_end) s1[i] = -INFINITY;
        }
      }
      float mx = s0[0];
#pragma unroll
      for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s0[i]);
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s1[i]);
      const float m_new = fmaxf(m, mx * c);
      if (m_new > -INFINITY) {
        float rs = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i)
          rs += fast_exp2(fmaf(s0[i], c, -m_new)) + fast_exp2(fmaf(s1[i], c, -m_new));
        l = fmaf(l, fast_exp2(m - m_new), rs);
        m = m_new;
      }
    }
    if (t + 1 < ntiles) store_rows_to_lds<D, NT>(Ks[buf ^ 1], reg);
    __syncthreads();
  }
  // merge the two lanes that hold the same audio query
  const float m2 = swap_halves(m), l2 = swap_halves(l);
  const float mm = fmaxf(m, m2);
  float lt = 0.f;
  if (mm > -INFINITY) lt = l * fast_exp2(m - mm) + l2 * fast_exp2(m2 - mm);
  if (g == 0 && j < L_a)
    part[(static_cast<size_t>(pair) * nchunk + chunk) * L_a + j] = make_float2(mm, lt);
}

// lse2[pair][j] = log2(sum over chunks of l * 2^m), merged in chunk order.
__global__ void lse_combine_kernel(const float2* __restrict__ part,
                                   float* __restrict__ lse2, int P, int L_a,
                                   int nchunk) {
  const size_t t = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<size_t>(P) * L_a) return;
  const size_t pair = t / L_a, j = t % L_a;
  const float2* p = part + pair * nchunk * L_a + j;
  float M = -INFINITY;
  for (int ch = 0; ch < nchunk; ++ch) M = fmaxf(M, p[static_cast<size_t>(ch) * L_a].x);
  float S = 0.f;
  for (int ch = 0; ch < nchunk; ++ch) {
    const float2 v = p[static_cast<size_t>(ch) * L_a];
    if (v.y > 0.f) S += v.y * fast_exp2(v.x - M);
  }
  lse2[t] = M + __log2f(S);
}

// ---- K2 ---------------------------------------------------------------------
// Column mass of one (batch, head) pair over a chunk of kColChunk video keys.
// 8 waves; wave w owns audio queries 64*w .. 64*w+63 of the current 512-query
// slab (two 32-row MFMA blocks), so every K operand read from LDS feeds two
// MFMAs.  S = Q^a K^v^T puts one video key per lane column: the lane sums
// exp2(S*c - lse) over its query rows and adds the result to its own slot of
// an LDS partial array (one writer per slot, so the order is fixed); the 16
// partials of a key (2 lane halves x 8 waves) are added in order at the end.
// Query rows past L_a carry lse = +inf, so their probabilities are exactly 0;
// keys past L_v only reach their own columns, which are not written.
constexpr int kColChunk = 512;   // video keys per K2 workgroup
constexpr int kColWaves = 8;     // 64 audio queries per wave

template <int D>
__global__ void __launch_bounds__(kColWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
a2v_colmass_kernel(const uint16_t* __restrict__ q_a,
                   const uint16_t* __restrict__ k_v,
                   const float* __restrict__ lse2, float* __restrict__ colmass,
                   int H, int L_v, int L_a, float c) {
  constexpr int NT = kColWaves * 64, KC = D / 16, CPR = D / 8;
  constexpr int CH = (kCT * CPR + NT - 1) / NT;   // 16-byte chunks per thread per tile
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][kCT * D];
  __shared__ float red[kColWaves * 2][kColChunk];
  const int chunk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 5, n = lane & 31;
  const int key0 = chunk * kColChunk;
  const int key_end = min(key0 + kColChunk, L_v);
  const size_t pair = static_cast<size_t>(b) * H + h;
  const uint16_t* kh = k_v + pair * L_v * D;
  const uint16_t* qh = q_a + pair * L_a * D;
  const float* lh = lse2 + pair * L_a;
  const int nslab = ceil_div(L_a, kQSlab);
  const int ntiles = ceil_div(key_end - key0, kCT);
  float* myred = red[2 * wave + g];
  for (int i = n; i < kColChunk; i += 32) myred[i] = 0.f;

  for (int slab = 0; slab < nslab; ++slab) {
    const int jb = slab * kQSlab + wave * 64;   // first query row of this wave
    u32x4 qf[2][KC];
    load_qfrag<D>(qh, jb + n, L_a, g, qf[0]);
    load_qfrag<D>(qh, jb + 32 + n, L_a, g, qf[1]);
    float lr[2][16];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int jj = jb + 32 * qb + crow(i, g);
        lr[qb][i] = jj < L_a ? lh[jj] : INFINITY;
      }
    u32x4 reg[CH];
    load_rows_to_regs<D, NT>(kh, key0, key_end, reg);
    __syncthreads();  // the previous slab is done with both buffers
    store_rows_to_lds<D, NT>(Ks[0], reg);
    __syncthreads();
#pragma unroll 1
    for (int t = 0; t < ntiles; ++t) {
      const int buf = t & 1;
      if (t + 1 < ntiles) load_rows_to_regs<D, NT>(kh, key0 + (t + 1) * kCT, key_end, reg);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s0 = zero16(), s1 = zero16();
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) {
          const u32x4 kf = lds_frag<D>(Ks[buf], 32 * kb + n, kc, g);
          s0 = mfma32x32x16(qf[0][kc], kf, s0);
          s1 = mfma32x32x16(qf[1][kc], kf, s1);
        }
        float cs = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i)
          cs += fast_exp2(fmaf(s0[i], c, -lr[0][i])) + fast_exp2(fmaf(s1[i], c, -lr[1][i]));
        myred[t * kCT + 32 * kb + n] += cs;
      }
      if (t + 1 < ntiles) store_rows_to_lds<D, NT>(Ks[buf ^ 1], reg);
      __syncthreads();
    }
  }
  __syncthreads();
  for (int kk = threadIdx.x; kk < kColChunk; kk += NT) {
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kColWaves * 2; ++w) sum += red[w][kk];
    if (key0 + kk < L_v) colmass[pair * L_v + key0 + kk] = sum;
  }
}

// ---- K3 ---------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(1024)
v2a_colmass_kernel(const uint16_t* __restrict__ q_v,
                   const uint16_t* __restrict__ k_a, float* __restrict__ part,
                   int L_v, int L_a, int nchunk, float c) {
  constexpr int NT = 1024, KC = D / 16;
  constexpr int CH = (kCT * (D / 8) + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][kCT * D];
  __shared__ float lse_w[16][32];
  __shared__ float red[16][2][kCT];
  const int chunk = blockIdx.x, pair = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 5, n = lane & 31;
  const int ibase = chunk * kV2aChunk + wave * 32;
  const bool wave_on = ibase < L_v;
  const uint16_t* kah = k_a + static_cast<size_t>(pair) * L_a * D;
  const int ntiles = ceil_div(L_a, kCT);

  u32x4 qf[KC];
  load_qfrag<D>(q_v + static_cast<size_t>(pair) * L_v * D, ibase + n, L_v, g, qf);
  u32x4 reg[CH];

  // pass 1: log-sum-exp of every video query over all audio keys
  float m = -INFINITY, l = 0.f;
  load_rows_to_regs<D, NT>(kah, 0, L_a, reg);
  store_rows_to_lds<D, NT>(Ks[0], reg);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int key0 = t * kCT;
    if (t + 1 < ntiles) load_rows_to_regs<D, NT>(kah, key0 + kCT, L_a, reg);
    if (wave_on) {
      f32x16 s0 = zero16(), s1 = zero16();
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        s0 = mfma32x32x16(lds_frag<D>(Ks[buf], n, kc, g), qf[kc], s0);
        s1 = mfma32x32x16(lds_frag<D>(Ks[buf], 32 + n, kc, g), qf[kc], s1);
      }
      if (key0 + kCT > L_a) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          if (key0 + crow(i, g) >= L_a) s0[i] = -INFINITY;
          if (key0 + 32 + crow(i, g) >= L_a) s1[i] = -INFINITY;
        }
      }
      float mx = s0[0];
#pragma unroll
      for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s0[i]);
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s1[i]);
      const float m_new = fmaxf(m, mx * c);
      if (m_new > -INFINITY) {
        float rs = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i)
          rs += fast_exp2(fmaf(s0[i], c, -m_new)) + fast_exp2(fmaf(s1[i], c, -m_new));
        l = fmaf(l, fast_exp2(m - m_new), rs);
        m = m_new;
      }
    }
    if (t + 1 < ntiles) store_rows_to_lds<D, NT>(Ks[buf ^ 1], reg);
    __syncthreads();
  }
  {
    const float m2 = swap_halves(m), l2 = swap_halves(l);
    const float mm = fmaxf(m, m2);
    float lt = 0.f;
    if (mm > -INFINITY) lt = l * fast_exp2(m - mm) + l2 * fast_exp2(m2 - mm);
    // rows past L_v get +inf: their probabilities are exactly 0
    if (g == 0) lse_w[wave][n] = (ibase + n < L_v) ? mm + __log2f(lt) : INFINITY;
  }
  __syncthreads();
  float lr[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) lr[i] = lse_w[wave][crow(i, g)];

  // pass 2: column mass of each 64-key audio tile
  load_rows_to_regs<D, NT>(kah, 0, L_a, reg);
  store_rows_to_lds<D, NT>(Ks[0], reg);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int key0 = t * kCT;
    if (t + 1 < ntiles) load_rows_to_regs<D, NT>(kah, key0 + kCT, L_a, reg);
    float cs0 = 0.f, cs1 = 0.f;
    if (wave_on) {
      f32x16 s0 = zero16(), s1 = zero16();
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        s0 = mfma32x32x16(qf[kc], lds_frag<D>(Ks[buf], n, kc, g), s0);
        s1 = mfma32x32x16(qf[kc], lds_frag<D>(Ks[buf], 32 + n, kc, g), s1);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        cs0 += fast_exp2(fmaf(s0[i], c, -lr[i]));
        cs1 += fast_exp2(fmaf(s1[i], c, -lr[i]));
      }
    }
    red[wave][g][n] = cs0;
    red[wave][g][32 + n] = cs1;
    if (t + 1 < ntiles) store_rows_to_lds<D, NT>(Ks[buf ^ 1], reg);
    __syncthreads();
    if (threadIdx.x < kCT && key0 + static_cast<int>(threadIdx.x) < L_a) {
      const int kk = threadIdx.x;
      float sum = 0.f;
      for (int w = 0; w < 16; ++w) sum += red[w][0][kk] + red[w][1][kk];
      part[(static_cast<size_t>(pair) * nchunk + chunk) * L_a + key0 + kk] = sum;
    }
    __syncthreads();
  }
}

// ---- finalize ---------------------------------------------------------------
// sal_v_tok / sal_v_blk from column-mass partials [B][nsum][L_v] (per head,
// or one partial holding every head), summed in order: grid (n_b, B), block
// threads = `block` (one per token of the video block).
__global__ void __launch_bounds__(128)
a2v_finalize_kernel(const float* __restrict__ colmass, float* __restrict__ sal_v_tok,
                    float* __restrict__ sal_v_blk, int L_v, int nsum,
                    float inv_norm, int accumulate) {
  __shared__ float red[128];
  const int c = blockIdx.x, b = blockIdx.y, n_b = gridDim.x;
  const int i = c * blockDim.x + threadIdx.x;
  float v = 0.f;
  if (i < L_v) {
    for (int gi = 0; gi < nsum; ++gi)
      v += colmass[(static_cast<size_t>(b) * nsum + gi) * L_v + i];
    v *= inv_norm;
    if (sal_v_tok != nullptr) {
      float* dst = sal_v_tok + static_cast<size_t>(b) * L_v + i;
      *dst = accumulate ? *dst + v : v;
    }
  }
  red[threadIdx.x] = v;
  __syncthreads();
  for (int s = blockDim.x / 2; s > 0; s >>= 1) {
    if (static_cast<int>(threadIdx.x) < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    float* dst = sal_v_blk + static_cast<size_t>(b) * n_b + c;
    *dst = accumulate ? *dst + red[0] : red[0];
  }
}

// head_sum[pair][j] = sum over video chunks of part[pair][chunk][j]: grid
// (ceil(L_a/64), P), 256 threads = 4 chunk phases x 64 audio keys, then a
// fixed-order sum of the 4 phases.
__global__ void __launch_bounds__(256)
v2a_chunk_sum_kernel(const float* __restrict__ part, float* __restrict__ head_sum,
                     int L_a, int nchunk) {
  __shared__ float red[4][64];
  const int j = blockIdx.x * 64 + (threadIdx.x & 63);
  const int ph = threadIdx.x >> 6;
  const size_t pair = blockIdx.y;
  float v = 0.f;
  if (j < L_a)
    for (int ch = ph; ch < nchunk; ch += 4)
      v += part[(pair * nchunk + ch) * L_a + j];
  red[ph][threadIdx.x & 63] = v;
  __syncthreads();
  if (ph == 0 && j < L_a)
    head_sum[pair * L_a + j] = (red[0][threadIdx.x] + red[1][threadIdx.x]) +
                               (red[2][threadIdx.x] + red[3][threadIdx.x]);
}

// sal_a_tok[b][j] = sum over nparts of part / (H*L_v), fixed order.
__global__ void v2a_finalize_kernel(const float* __restrict__ part,
                                    float* __restrict__ sal_a_tok, int B,
                                    int nparts, int L_a, float inv_norm,
                                    int accumulate) {
  const size_t t = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<size_t>(B) * L_a) return;
  const size_t b = t / L_a, j = t % L_a;
  float v = 0.f;
  for (int p = 0; p < nparts; ++p)
    v += part[(b * nparts + p) * L_a + j];
  v *= inv_norm;
  sal_a_tok[t] = accumulate ? sal_a_tok[t] + v : v;
}

// ---- fp32 path --------------------------------------------------------------
// Row log2-sum-exp of scale*Q K^T over all keys: one thread per query row.
template <int D>
__global__ void __launch_bounds__(128)
row_lse2_f32_kernel(const float* __restrict__ qm, const float* __restrict__ km,
                    float* __restrict__ lse2, int P, int Lq, int Lk, float c) {
  const size_t t = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<size_t>(P) * Lq) return;
  const size_t pair = t / Lq;
  const float* qr = qm + t * D;
  const float* kh = km + pair * Lk * D;
  float qv[D];
#pragma unroll
  for (int e = 0; e < D; ++e) qv[e] = qr[e];
  float m = -INFINITY, l = 0.f;
  for (int i = 0; i < Lk; ++i) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) s = fmaf(qv[e], kh[static_cast<size_t>(i) * D + e], s);
    s *= c;
    const float m_new = fmaxf(m, s);
    l = l * exp2f(m - m_new) + exp2f(s - m_new);
    m = m_new;
  }
  lse2[t] = m + log2f(l);
}

// Column mass: out[b][i] = sum_h sum_j 2^(c * q_j . k_i - lse2[b,h,j]) for
// key i; one thread per (b, key).
template <int D>
__global__ void __launch_bounds__(128)
colmass_f32_kernel(const float* __restrict__ qm, const float* __restrict__ km,
                   const float* __restrict__ lse2, float* __restrict__ out, int B,
                   int H, int Lq, int Lk, float c) {
  const size_t t = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<size_t>(B) * Lk) return;
  const size_t b = t / Lk, i = t % Lk;
  float acc = 0.f;
  for (int h = 0; h < H; ++h) {
    const size_t pair = b * H + h;
    float kv[D];
#pragma unroll
    for (int e = 0; e < D; ++e) kv[e] = km[(pair * Lk + i) * D + e];
    const float* qh = qm + pair * Lq * D;
    for (int j = 0; j < Lq; ++j) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < D; ++e) s = fmaf(qh[static_cast<size_t>(j) * D + e], kv[e], s);
      acc += exp2f(s * c - lse2[pair * Lq + j]);
    }
  }
  out[t] = acc;
}

template <int D>
void cross_bf16(const uint16_t* q_a, const uint16_t* k_v, const uint16_t* q_v,
                const uint16_t* k_a, int B, int H, int L_v, int L_a, float scale,
                int block, float* sal_v_tok, float* sal_v_blk, float* sal_a_tok,
                int accumulate, char* ws, hipStream_t s) {
  const CrossWs lay = cross_ws_layout(B, H, L_v, L_a);
  const float c = scale * kLog2e;
  const int P = B * H;
  const int nchunk = ceil_div(L_v, kLseChunk);
  const int nslab = ceil_div(L_a, kQSlab);
  float2* lse_part = reinterpret_cast<float2*>(ws + lay.lse_part);
  float* lse_a = reinterpret_cast<float*>(ws + lay.lse_a);
  float* colmass = reinterpret_cast<float*>(ws + lay.colmass);
  hipLaunchKernelGGL(a2v_lse_partial_kernel<D>, dim3(nchunk, nslab, P), dim3(1024), 0, s,
                     q_a, k_v, lse_part, L_v, L_a, nchunk, c);
  const size_t nlse = static_cast<size_t>(P) * L_a;
  hipLaunchKernelGGL(lse_combine_kernel, dim3((nlse + 255) / 256), dim3(256), 0, s,
                     lse_part, lse_a, P, L_a, nchunk);
  hipLaunchKernelGGL(a2v_colmass_kernel<D>, dim3(ceil_div(L_v, kColChunk), H, B),
                     dim3(kColWaves * 64), 0, s, q_a, k_v, lse_a, colmass, H, L_v, L_a, c);
  const int n_b = ceil_div(L_v, block);
  hipLaunchKernelGGL(a2v_finalize_kernel, dim3(n_b, B), dim3(block), 0, s, colmass,
                     sal_v_tok, sal_v_blk, L_v, H,
                     1.0f / (static_cast<float>(H) * static_cast<float>(L_a)), accumulate);
  if (q_v != nullptr) {
    float* v2a_part = reinterpret_cast<float*>(ws + lay.v2a_part);
    const int nchunk3 = ceil_div(L_v, kV2aChunk);
    float* v2a_head = reinterpret_cast<float*>(ws + lay.v2a_head);
    hipLaunchKernelGGL(v2a_colmass_kernel<D>, dim3(nchunk3, P), dim3(1024), 0, s, q_v,
                       k_a, v2a_part, L_v, L_a, nchunk3, c);
    hipLaunchKernelGGL(v2a_chunk_sum_kernel, dim3(ceil_div(L_a, 64), P), dim3(256), 0, s,
                       v2a_part, v2a_head, L_a, nchunk3);
    const size_t na = static_cast<size_t>(B) * L_a;
    hipLaunchKernelGGL(v2a_finalize_kernel, dim3((na + 255) / 256), dim3(256), 0, s,
                       v2a_head, sal_a_tok, B, H, L_a,
                       1.0f / (static_cast<float>(H) * static_cast<float>(L_v)), accumulate);
  }
}

template <int D>
void cross_f32(const float* q_a, const float* k_v, const float* q_v,
               const float* k_a, int B, int H, int L_v, int L_a, float scale,
               int block, float* sal_v_tok, float* sal_v_blk, float* sal_a_tok,
               int accumulate, char* ws, hipStream_t s) {
  const CrossWs lay = cross_ws_layout(B, H, L_v, L_a);
  const float c = scale * kLog2e;
  const int P = B * H;
  float* lse_a = reinterpret_cast<float*>(ws + lay.lse_a);
  float* colmass = reinterpret_cast<float*>(ws + lay.colmass);
  const size_t na = static_cast<size_t>(P) * L_a;
  hipLaunchKernelGGL(row_lse2_f32_kernel<D>, dim3((na + 127) / 128), dim3(128), 0, s,
                     q_a, k_v, lse_a, P, L_a, L_v, c);
  const size_t nv = static_cast<size_t>(B) * L_v;
  hipLaunchKernelGGL(colmass_f32_kernel<D>, dim3((nv + 127) / 128), dim3(128), 0, s,
                     q_a, k_v, lse_a, colmass, B, H, L_a, L_v, c);
  const int n_b = ceil_div(L_v, block);
  hipLaunchKernelGGL(a2v_finalize_kernel, dim3(n_b, B), dim3(block), 0, s, colmass,
                     sal_v_tok, sal_v_blk, L_v, 1,
                     1.0f / (static_cast<float>(H) * static_cast<float>(L_a)), accumulate);
  if (q_v != nullptr) {
    float* lse_v = reinterpret_cast<float*>(ws + lay.lse_v);
    float* v2a = reinterpret_cast<float*>(ws + lay.v2a_part);
    const size_t nvq = static_cast<size_t>(P) * L_v;
    hipLaunchKernelGGL(row_lse2_f32_kernel<D>, dim3((nvq + 127) / 128), dim3(128), 0, s,
                       q_v, k_a, lse_v, P, L_v, L_a, c);
    const size_t nak = static_cast<size_t>(B) * L_a;
    hipLaunchKernelGGL(colmass_f32_kernel<D>, dim3((nak + 127) / 128), dim3(128), 0, s,
                       q_v, k_a, lse_v, v2a, B, H, L_v, L_a, c);
    hipLaunchKernelGGL(v2a_finalize_kernel, dim3((nak + 255) / 256), dim3(256), 0, s,
                       v2a, sal_a_tok, B, 1, L_a,
                       1.0f / (static_cast<float>(H) * static_cast<float>(L_v)), accumulate);
  }
}

}  // namespace

void launch_cross_scores_bf16(const uint16_t* q_a, const uint16_t* k_v,
                              const uint16_t* q_v, const uint16_t* k_a, int B,
                              int H, int L_v, int L_a, int d, float scale,
                              int block, float* sal_v_tok, float* sal_v_blk,
                              float* sal_a_tok, int accumulate, char* ws,
                              hipStream_t s) {
  if (d == 128)
    cross_bf16<128>(q_a, k_v, q_v, k_a, B, H, L_v, L_a, scale, block, sal_v_tok,
                    sal_v_blk, sal_a_tok, accumulate, ws, s);
  else
    cross_bf16<64>(q_a, k_v, q_v, k_a, B, H, L_v, L_a, scale, block, sal_v_tok,
                   sal_v_blk, sal_a_tok, accumulate, ws, s);
}

void launch_cross_scores_f32(const float* q_a, const float* k_v,
                             const float* q_v, const float* k_a, int B, int H,
                             int L_v, int L_a, int d, float scale, int block,
                             float* sal_v_tok, float* sal_v_blk,
                             float* sal_a_tok, int accumulate, char* ws,
                             hipStream_t s) {
  if (d == 128)
    cross_f32<128>(q_a, k_v, q_v, k_a, B, H, L_v, L_a, scale, block, sal_v_tok,
                   sal_v_blk, sal_a_tok, accumulate, ws, s);
  else
    cross_f32<64>(q_a, k_v, q_v, k_a, B, H, L_v, L_a, scale, block, sal_v_tok,
                  sal_v_blk, sal_a_tok, accumulate, ws, s);
}

}  // namespace sa
