// Protected block-sparse flash attention (Sec. 4.2, Eq. (10) in the row
// form of Eq. (11); Eq. (5) when a list holds every key block).
//
// bf16 path (MFMA, gfx950)
// ------------------------
// One workgroup per query block (BLOCK rows, BLOCK/32 waves of 32 query rows
// each).  The workgroup walks its compacted key-block list; every key block
// is streamed as 64-key tiles through double-buffered LDS (K as [key][d],
// V as V^T [d][key], both XOR-swizzled so the MFMA operand reads are free of
// bank conflicts).  Each wave computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16, so a lane owns one query column: the row max and
// row sum of the online softmax are lane-local, plus one exchange with the
// lane holding the other 16 keys of the same query.  P^T is packed to bf16 in
// registers and feeds O^T += V^T P^T directly as the B operand.  The scale is
// folded into exp2.  Keys past L are -inf, rows past L are never written.
//
// V^T comes from a transposing copy into the workspace (zero-filled past L);
// query blocks are launched heaviest list first (protected rows hold the
// full list), rank-major over (batch, head) pairs, so that when the pair
// count is a multiple of 8 every pair stays on one XCD and its K/V tiles are
// shared through that XCD's L2.
//
// f32 path: a plain per-row online softmax with K/V tiles in LDS (used by the
// small fp32 workloads; fp32 MFMA would not change its role).
#include "sa_device.h"
#include "sa_internal.h"

namespace sa {
namespace {

constexpr int kTile = 64;  // keys per LDS tile

// Query blocks of every (b,h) pair ordered by kv_cnt descending, then by
// block index ascending.
__global__ void __launch_bounds__(256)
order_rows_kernel(const int32_t* __restrict__ kv_cnt, int32_t* __restrict__ order,
                  int n_b) {
  __shared__ int cnt[kMaxBlocks];
  const size_t base = static_cast<size_t>(blockIdx.x) * n_b;
  for (int r = threadIdx.x; r < n_b; r += blockDim.x) {
    int c = kv_cnt[base + r];
    cnt[r] = c < 0 ? 0 : (c > n_b ? n_b : c);
  }
  __syncthreads();
  for (int r = threadIdx.x; r < n_b; r += blockDim.x) {
    const int mine = cnt[r];
    int rank = 0;
    for (int j = 0; j < n_b; ++j) {
      const int o = cnt[j];
      rank += (o > mine) || (o == mine && j < r);
    }
    order[base + rank] = r;
  }
}

// V [pair][L][D] -> V^T [pair][D][Lp], zero for keys >= L.  Grid (Lp/64, P).
template <int D>
__global__ void __launch_bounds__(256)
transpose_v_kernel(const uint16_t* __restrict__ v, uint16_t* __restrict__ vt,
                   int L, int Lp) {
  constexpr int ROW32 = D / 2 + 1;  // padded row, in 32-bit words
  __shared__ uint32_t tile[kTile * ROW32];
  const size_t pair = blockIdx.y;
  const int key0 = blockIdx.x * kTile;
  const uint16_t* src = v + pair * L * D;
  for (int q = threadIdx.x; q < kTile * D / 8; q += 256) {
    const int row = q / (D / 8), cc = q % (D / 8);
    u32x4 val = {0u, 0u, 0u, 0u};
    if (key0 + row < L) val = ldg16(src + static_cast<size_t>(key0 + row) * D + cc * 8);
    uint32_t* dst = tile + row * ROW32 + cc * 4;
    dst[0] = val.x; dst[1] = val.y; dst[2] = val.z; dst[3] = val.w;
  }
  __syncthreads();
  const uint16_t* t16 = reinterpret_cast<const uint16_t*>(tile);
  uint16_t* dst = vt + pair * D * Lp;
  for (int q = threadIdx.x; q < D * (kTile / 8); q += 256) {
    const int d = q / (kTile / 8), c = q % (kTile / 8);
    u32x4 out;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t lo = t16[(8 * c + 2 * j) * (2 * ROW32) + d];
      const uint32_t hi = t16[(8 * c + 2 * j + 1) * (2 * ROW32) + d];
      out[j] = lo | (hi << 16);
    }
    stg16(dst + static_cast<size_t>(d) * Lp + key0 + 8 * c, out);
  }
}

template <int D, int BLOCK>
__global__ void __launch_bounds__(BLOCK * 2)
sparse_attn_bf16_kernel(const uint16_t* __restrict__ q,
                        const uint16_t* __restrict__ k,
                        const uint16_t* __restrict__ vt,
                        uint16_t* __restrict__ o, float* __restrict__ lse,
                        const int32_t* __restrict__ kv_idx,
                        const int32_t* __restrict__ kv_cnt,
                        const int32_t* __restrict__ order, int P, int L,
                        int Lp, int n_b, float c) {
  constexpr int NT = BLOCK * 2;              // threads per workgroup
  constexpr int CPR = D / 8;                 // 16-byte chunks per K row
  constexpr int KCH = kTile * CPR / NT;      // K chunks per thread per tile
  constexpr int VCH = D * (kTile / 8) / NT;  // V^T chunks per thread per tile
  constexpr int TPB = BLOCK / kTile;         // tiles per key block
  constexpr int KC = D / 16;                 // k-steps of Q K^T
  constexpr int DT = D / 32;                 // 32-row d tiles of O^T
  static_assert(KCH >= 1 && VCH >= 1, "tile too small for the workgroup");

  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][kTile * D];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2][D * kTile];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, n = lane & 31;

  const int pair = blockIdx.x % P;
  const int rank = blockIdx.x / P;
  const size_t row_base = static_cast<size_t>(pair) * n_b;
  const int r = order[row_base + rank];
  int cnt = kv_cnt[row_base + r];
  cnt = cnt < 0 ? 0 : (cnt > n_b ? n_b : cnt);
  const int32_t* idx = kv_idx + (row_base + r) * n_b;

  const uint16_t* qh = q + static_cast<size_t>(pair) * L * D;
  const uint16_t* kh = k + static_cast<size_t>(pair) * L * D;
  const uint16_t* vth = vt + static_cast<size_t>(pair) * D * Lp;

  const int qrow = r * BLOCK + wave * 32 + n;
  u32x4 qf[KC];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    qf[kc] = qrow < L ? ldg16(qh + static_cast<size_t>(qrow) * D + 16 * kc + 8 * g)
                      : u32x4{0u, 0u, 0u, 0u};
  }

  f32x16 acc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) acc[dt] = zero16();
  float m = -INFINITY;
  float lsum = 0.f;

  const int T = cnt * TPB;
  u32x4 kr[KCH], vr[VCH];

  auto tile_key0 = [&](int t, bool& ok) {
    const int kb = idx[t / TPB];
    const int key0 = kb * BLOCK + kTile * (t % TPB);
    ok = kb >= 0 && kb < n_b && key0 < L;
    return key0;
  };
  auto load_tile = [&](int t) {
    bool ok;
    const int key0 = tile_key0(t, ok);
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int qq = tid + NT * i;
      const int row = qq / CPR, cc = qq % CPR;
      kr[i] = (ok && key0 + row < L)
                  ? ldg16(kh + static_cast<size_t>(key0 + row) * D + cc * 8)
                  : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int qq = tid + NT * i;
      const int d = qq / (kTile / 8), cc = qq % (kTile / 8);
      vr[i] = ok ? ldg16(vth + static_cast<size_t>(d) * Lp + key0 + cc * 8)
                 : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int qq = tid + NT * i;
      const int row = qq / CPR, cc = qq % CPR;
      stg16(&Ks[buf][row * D + ((cc ^ (row & (CPR - 1))) * 8)], kr[i]);
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int qq = tid + NT * i;
      const int d = qq / (kTile / 8), cc = qq % (kTile / 8);
      const int s = d & 15;
      const int unit = (2 * cc) ^ (s & 14);  // 8-byte units, pairs stay aligned
      u32x4 val = vr[i];
      if (s & 1) val = u32x4{val.z, val.w, val.x, val.y};
      stg16(&Vs[buf][d * kTile + unit * 4], val);
    }
  };

  if (T > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  for (int t = 0; t < T; ++t) {
    const int buf = t & 1;
    if (t + 1 < T) load_tile(t + 1);
    bool ok;
    const int key0 = tile_key0(t, ok);
    if (ok) {
      const uint16_t* Kb = Ks[buf];
      const uint16_t* Vb = Vs[buf];
      f32x16 s0 = zero16(), s1 = zero16();
#pragma unroll
      for (int kc = 0; kc < KC; ++kc) {
        const int ch = 2 * kc + g;
        const u32x4 a0 = *reinterpret_cast<const u32x4*>(
            Kb + n * D + ((ch ^ (n & (CPR - 1))) * 8));
        const u32x4 a1 = *reinterpret_cast<const u32x4*>(
            Kb + (32 + n) * D + ((ch ^ ((32 + n) & (CPR - 1))) * 8));
        s0 = mfma32x32x16(a0, qf[kc], s0);
        s1 = mfma32x32x16(a1, qf[kc], s1);
      }
      if (key0 + kTile > L) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          if (key0 + crow(i, g) >= L) s0[i] = -INFINITY;
          if (key0 + 32 + crow(i, g) >= L) s1[i] = -INFINITY;
        }
      }
      float mx = s0[0];
#pragma unroll
      for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s0[i]);
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s1[i]);
      mx = fmaxf(mx, swap_halves(mx));
      const float m_new = fmaxf(m, mx * c);
      const float alpha = fast_exp2(m - m_new);
      m = m_new;
      float rs = 0.f;
      uint32_t pb0[8], pb1[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float p0 = fast_exp2(fmaf(s0[2 * i], c, -m_new));
        const float p1 = fast_exp2(fmaf(s0[2 * i + 1], c, -m_new));
        const float p2 = fast_exp2(fmaf(s1[2 * i], c, -m_new));
        const float p3 = fast_exp2(fmaf(s1[2 * i + 1], c, -m_new));
        rs += (p0 + p1) + (p2 + p3);
        pb0[i] = pack_bf16x2(p0, p1);
        pb1[i] = pack_bf16x2(p2, p3);
      }
      lsum = fmaf(lsum, alpha, rs);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[dt][i] *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int drow = 32 * dt + n;
        const int sw = drow & 15;
        const uint16_t* vrow = Vb + drow * kTile;
#pragma unroll
        for (int mm = 0; mm < 4; ++mm) {
          const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow + (((4 * mm + g) ^ sw) * 4));
          const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + (((4 * mm + 2 + g) ^ sw) * 4));
          const uint32_t* pb = (mm < 2) ? pb0 : pb1;
          const int h = (mm & 1) * 4;
          const u32x4 a = {lo.x, lo.y, hi.x, hi.y};
          const u32x4 b = {pb[h], pb[h + 1], pb[h + 2], pb[h + 3]};
          acc[dt] = mfma32x32x16(a, b, acc[dt]);
        }
      }
    }
    if (t + 1 < T) store_tile(buf ^ 1);
    __syncthreads();
  }

  const float ltot = lsum + swap_halves(lsum);
  const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
  if (qrow < L) {
    uint16_t* orow = o + (static_cast<size_t>(pair) * L + qrow) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int d0 = 32 * dt + 8 * rg + 4 * g;
        u32x2 val = {pack_bf16x2(acc[dt][4 * rg] * inv, acc[dt][4 * rg + 1] * inv),
                     pack_bf16x2(acc[dt][4 * rg + 2] * inv, acc[dt][4 * rg + 3] * inv)};
        *reinterpret_cast<u32x2*>(orow + d0) = val;
      }
    }
    if (lse != nullptr && g == 0)
      lse[static_cast<size_t>(pair) * L + qrow] =
          ltot > 0.f ? (m + __log2f(ltot)) * kLn2 : -INFINITY;
  }
}

// ---- fp32 path ------------------------------------------------------------
constexpr int kF32Keys = 32;

template <int D>
__global__ void __launch_bounds__(128)
sparse_attn_f32_kernel(const float* __restrict__ q, const float* __restrict__ k,
                       const float* __restrict__ v, float* __restrict__ o,
                       float* __restrict__ lse,
                       const int32_t* __restrict__ kv_idx,
                       const int32_t* __restrict__ kv_cnt, int L, int n_b,
                       int block, float scale) {
  __shared__ float Kt[kF32Keys][D + 1];
  __shared__ float Vt[kF32Keys][D];
  const int pair = blockIdx.y;
  const int r = blockIdx.x;
  const size_t row_base = static_cast<size_t>(pair) * n_b + r;
  int cnt = kv_cnt[row_base];
  cnt = cnt < 0 ? 0 : (cnt > n_b ? n_b : cnt);
  const int32_t* idx = kv_idx + row_base * n_b;
  const float* qh = q + static_cast<size_t>(pair) * L * D;
  const float* kh = k + static_cast<size_t>(pair) * L * D;
  const float* vh = v + static_cast<size_t>(pair) * L * D;
  const int tid = threadIdx.x;
  const int qrow = r * block + tid;
  const bool active = tid < block && qrow < L;

  float qv[D], acc[D];
#pragma unroll
  for (int e = 0; e < D; ++e) {
    qv[e] = active ? qh[static_cast<size_t>(qrow) * D + e] : 0.f;
    acc[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;

  for (int i = 0; i < cnt; ++i) {
    const int kb = idx[i];
    if (kb < 0 || kb >= n_b) continue;
    const int kend = min((kb + 1) * block, L);
    for (int key0 = kb * block; key0 < kend; key0 += kF32Keys) {
      const int nk = min(kF32Keys, kend - key0);
      __syncthreads();
      for (int e = tid; e < nk * D; e += blockDim.x) {
        const int j = e / D, dd = e % D;
        Kt[j][dd] = kh[static_cast<size_t>(key0 + j) * D + dd];
        Vt[j][dd] = vh[static_cast<size_t>(key0 + j) * D + dd];
      }
      __syncthreads();
      if (active) {
        for (int j = 0; j < nk; ++j) {
          float s = 0.f;
#pragma unroll
          for (int e = 0; e < D; ++e) s = fmaf(qv[e], Kt[j][e], s);
          s *= scale;
          const float m_new = fmaxf(m, s);
          const float alpha = expf(m - m_new);
          const float p = expf(s - m_new);
          l = l * alpha + p;
#pragma unroll
          for (int e = 0; e < D; ++e) acc[e] = fmaf(acc[e], alpha, p * Vt[j][e]);
          m = m_new;
        }
      }
    }
  }
  if (active) {
    const float inv = l > 0.f ? 1.f / l : 0.f;
    float* orow = o + (static_cast<size_t>(pair) * L + qrow) * D;
#pragma unroll
    for (int e = 0; e < D; ++e) orow[e] = acc[e] * inv;
    if (lse != nullptr)
      lse[static_cast<size_t>(pair) * L + qrow] = l > 0.f ? m + logf(l) : -INFINITY;
  }
}

}  // namespace

void launch_sparse_attention_bf16(const uint16_t* q, const uint16_t* k,
                                  const uint16_t* v, uint16_t* o, float* lse,
                                  int B, int H, int L, int d, float scale,
                                  int block, const int32_t* kv_idx,
                                  const int32_t* kv_cnt, char* ws,
                                  hipStream_t s) {
  const int n_b = ceil_div(L, block);
  const int P = B * H;
  const int Lp = n_b * block;
  const AttnWs lay = attn_ws_layout(B, H, n_b, d, block);
  uint16_t* vt = reinterpret_cast<uint16_t*>(ws + lay.vt);
  int32_t* order = reinterpret_cast<int32_t*>(ws + lay.order);
  const float c = scale * kLog2e;
  const dim3 tgrid(Lp / kTile, P);
  if (d == 128)
    hipLaunchKernelGGL(transpose_v_kernel<128>, tgrid, dim3(256), 0, s, v, vt, L, Lp);
  else
    hipLaunchKernelGGL(transpose_v_kernel<64>, tgrid, dim3(256), 0, s, v, vt, L, Lp);
  hipLaunchKernelGGL(order_rows_kernel, dim3(P), dim3(256), 0, s, kv_cnt, order, n_b);
  const dim3 grid(P * n_b);
  if (d == 128 && block == 128)
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<128, 128>), grid, dim3(256), 0, s,
                       q, k, vt, o, lse, kv_idx, kv_cnt, order, P, L, Lp, n_b, c);
  else if (d == 128 && block == 64)
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<128, 64>), grid, dim3(128), 0, s,
                       q, k, vt, o, lse, kv_idx, kv_cnt, order, P, L, Lp, n_b, c);
  else if (d == 64 && block == 128)
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<64, 128>), grid, dim3(256), 0, s,
                       q, k, vt, o, lse, kv_idx, kv_cnt, order, P, L, Lp, n_b, c);
  else
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<64, 64>), grid, dim3(128), 0, s,
                       q, k, vt, o, lse, kv_idx, kv_cnt, order, P, L, Lp, n_b, c);
}

void launch_sparse_attention_f32(const float* q, const float* k,
                                 const float* v, float* o, float* lse, int B,
                                 int H, int L, int d, float scale, int block,
                                 const int32_t* kv_idx, const int32_t* kv_cnt,
                                 char* /*ws*/, hipStream_t s) {
  const int n_b = ceil_div(L, block);
  const dim3 grid(n_b, B * H);
  if (d == 128)
    hipLaunchKernelGGL(sparse_attn_f32_kernel<128>, grid, dim3(128), 0, s, q, k, v,
                       o, lse, kv_idx, kv_cnt, L, n_b, block, scale);
  else
    hipLaunchKernelGGL(sparse_attn_f32_kernel<64>, grid, dim3(128), 0, s, q, k, v,
                       o, lse, kv_idx, kv_cnt, L, n_b, block, scale);
}

}  // namespace sa
