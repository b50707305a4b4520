// Cross-modal saliency (Sec. 4.1, Eq. (1)-(2) and the reverse v->a
// direction).
//
// a->v: s^v_i = 1/(H*L_a) * sum_h sum_j softmax_i(scale * q^a_j . k^v_i).
//   K1 a2v_lse_partial : per (1024-key chunk, 512-query slab, b*h) one 8-wave
//                        workgroup holding the slab's audio queries (64 per
//                        wave) streams the chunk's video keys with
//                        S^T = K^v Q^a^T, so a lane owns an audio query and
//                        keeps a lane-local (max, sum); partials go to
//                        workspace.
//   K1b lse_combine    : fixed-order merge of the chunk partials (log2 units).
//   K2 a2v_colmass     : per (1024-key chunk, h, b) the workgroup streams the
//                        chunk's video keys once per audio slab with
//                        S = Q^a K^v^T, so a lane owns a video key column and
//                        sums exp2(S*c - lse) over its query rows; the 16
//                        lane partials of a key are added in a fixed order.
//   K2b a2v_finalize   : sum over heads, divide by H*L_a, block sums.
// v->a: s^a_j = 1/(H*L_v) * sum_h sum_i softmax_j(scale * q^v_i . k^a_j).
//   K3 v2a_colmass     : per (512 video queries, b*h); pass 1 streams every
//                        audio key with S^T for each video query's
//                        log-sum-exp, pass 2 streams them again, 512 at a
//                        time, with S and sums the column mass of each key.
//   K3b v2a_chunk_sum  : fixed-order sum over video chunks per head, then
//       v2a_finalize   : fixed-order sum over heads, / (H*L_v).
// From the forwards: with the row LSEs of the a->v and v->a cross-attention
// forwards (natural log, as the attention kernels write them), K1/K1b and
// pass 1 of K3 are skipped: lse_to_log2 converts lse_a for K2, and K3 reads
// lse_v.
// All bf16 kernels share one key-stream engine (below).  No atomics: every
// output element has one writer, so results are reproducible.
// fp32 inputs use plain per-thread kernels with the same outputs.
#include "sa_device.h"
#include "sa_internal.h"

namespace sa {
namespace {

template <int D>
__device__ __forceinline__ void load_qfrag(const uint16_t* base, int row, int nrows,
                                           int g, u32x4* qf) {
#pragma unroll
  for (int kc = 0; kc < D / 16; ++kc)
    qf[kc] = row < nrows ? ldg16(base + static_cast<size_t>(row) * D + 16 * kc + 8 * g)
                         : u32x4{0u, 0u, 0u, 0u};
}

// sum_{i < n} p[i * stride], added in index order; the loads are issued in
// batches of 8 so that they are in flight together.
__device__ __forceinline__ float sum_strided(const float* __restrict__ p, size_t stride,
                                             int n) {
  float acc = 0.f;
  int i = 0;
  for (; i + 8 <= n; i += 8) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = p[static_cast<size_t>(i + k) * stride];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc += v[k];
  }
  for (; i < n; ++i) acc += p[static_cast<size_t>(i) * stride];
  return acc;
}

// ---- bf16 key-stream engine (K1, K2, K3) -------------------------------------
// A workgroup of 8 waves holds 512 query rows in registers, 64 per wave as two
// 32-row MFMA blocks, and streams 64-key tiles of one key matrix through an
// LDS ring (plane layout of sa_device.h) in groups of two tiles: the copy of
// the next group is in flight while the current one is read.  A wave works in units of 32 keys
// (one half of a tile): the D/8 MFMAs of unit u+1 are interleaved with the
// exponentials of unit u, so that the matrix cores and the vector ALU of a
// SIMD work at the same time.
constexpr int kXW = 8;                 // waves per workgroup
constexpr int kXNT = kXW * 64;         // threads per workgroup
constexpr int kGroup = 2;              // tiles per barrier interval
constexpr int kRing = 2 * kGroup;      // stages of the LDS key ring
static_assert(kXW * 64 == kQSlab && kXW * 64 == kV2aChunk,
              "one workgroup holds one slab of 512 query rows");
constexpr int kColKeys = 1024;         // video keys per K2 workgroup
constexpr int kAWin = 512;             // audio keys per K3 column-mass window
// A log-sum-exp unit whose sum against the running max reaches 2^64 is
// redone against its own max (the running max is only raised then).
constexpr float kSumGuard = 18446744073709551616.0f;

template <int D>
struct KeyRing {
  static constexpr int TB = 128 * D;            // bytes per 64-key tile
  static constexpr int CPT = TB / (16 * kXNT);  // 16-byte copies per thread per tile
  static_assert(CPT >= 1 && CPT * 16 * kXNT == TB, "tile copy split");
  uint32_t lds;         // LDS byte address of stage 0
  uint32_t span[CPT];   // byte offset of this wave's 1 KB spans in a stage
  int row[CPT];         // tile row copied by this lane
  uint32_t col[CPT];    // byte offset of the lane's source slot within the row
  int rd[2];            // lane offsets of the operand reads (k-step even / odd)

  __device__ __forceinline__ void init(char* ring, int wave, int lane) {
    lds = (uint32_t)(size_t)(lds_void_t*)ring;
    const int n = lane & 31, g = lane >> 5;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int sp = wave + kXW * i;  // span sp = plane sp/4, rows 16*(sp%4) ..
      span[i] = sp * 1024;
      row[i] = 16 * (sp & 3) + (lane >> 2);
      col[i] = static_cast<uint32_t>((sp >> 2) * 64 + 16 * ((lane & 3) ^ plane_swz(row[i])));
    }
    // operand row n (+32 for the second unit of a tile), slot 2*(kc&1) + g
    rd[0] = n * 64 + 16 * (g ^ plane_swz(n));
    rd[1] = n * 64 + 16 * ((2 + g) ^ plane_swz(n));
  }
  // Copy keys [key0, key0 + 64) of the [L][D] matrix at src into stage st;
  // rows past L repeat row L - 1.
  __device__ __forceinline__ void issue(const char* src, int key0, int L, int st) const {
    const char* base = src + static_cast<size_t>(key0) * (2 * D);
    const int limit = min(63, L - 1 - key0);
#pragma unroll
    for (int i = 0; i < CPT; ++i)
      lds_dma16(base, static_cast<uint32_t>(min(row[i], limit) * (2 * D)) + col[i],
                __builtin_amdgcn_readfirstlane(lds + st * TB + span[i]));
  }
};

// MFMAs of one unit: keys 32*kb .. 32*kb+31 of the tile at `tile` against both
// query blocks, into acc.  KEYS_A: acc[h] = K Q_h^T (a lane owns a query
// column, its 16 elements are keys crow(i, g)); otherwise acc[h] = Q_h K^T (a
// lane owns a key column, its elements are query rows 32h + crow(i, g)).
// work(s), s = 0 .. D/8-1, runs on the vector ALU before the s-th MFMA.
template <int D, bool KEYS_A, class W>
__device__ __forceinline__ void unit_mfma(const char* tile, const int (&rd)[2], int kb,
                                          const u32x4 (&qf)[2][D / 16], f32x16 (&acc)[2],
                                          W&& work) {
  constexpr int KC = D / 16;
  auto rdk = [&](int kc) {
    return *reinterpret_cast<const u32x4*>(tile + (kc >> 1) * 4096 + kb * 2048 + rd[kc & 1]);
  };
  u32x4 kf[KC];
  kf[0] = rdk(0);
  kf[1] = rdk(1);
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    if (kc + 2 < KC) kf[kc + 2] = rdk(kc + 2);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      work(2 * kc + h);
      const f32x16 c0 = kc == 0 ? zero16() : acc[h];
      acc[h] = KEYS_A ? mfma32x32x16(kf[kc], qf[h][kc], c0) : mfma32x32x16(qf[h][kc], kf[kc], c0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Wait until at most n (0 <= n <= N, wave-uniform) vector-memory operations
// of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm_le(int n) {
  if constexpr (N > 0) {
    if (n >= N) {
      wait_vm<N>();
      return;
    }
    wait_vm_le<N - 1>(n);
  } else {
    wait_vm<0>();
  }
}

// Streams tiles t = 0 .. T-1 (T >= 1) of keys key_begin + 64t of the [L][D]
// matrix at src; unit u = 2t + kb.  Tiles go through the ring in groups of
// kGroup (stage t % kRing): the copies of group j+1 are issued right after
// the barrier that opens group j, whose stages held group j-1, and are
// awaited at the barrier that opens group j+1, so one barrier serves
// 2*kGroup units of every wave.  acc.first(x) sees unit 0 once,
// acc.slot(x, s, u, last) is the share of the work on a finished unit placed
// beside the s-th MFMA of the next one, acc.fin(x, u, last) closes the unit;
// `last` marks the units of tile T-1.  Ends with a barrier (ring free).
template <int D, bool KEYS_A, class Acc>
__device__ __forceinline__ void stream_keys(const KeyRing<D>& ring, const char* ring_lds,
                                            const char* src, int key_begin, int L, int T,
                                            const u32x4 (&qf)[2][D / 16], Acc& acc) {
  constexpr int TB = KeyRing<D>::TB, CPT = KeyRing<D>::CPT, NS = D / 8;
  auto issue_group = [&](int grp) {
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const int t = grp * kGroup + i;
      if (t < T) ring.issue(src, key_begin + 64 * t, L, t % kRing);
    }
  };
  issue_group(0);
  issue_group(1);
  // group 0 has landed once at most the copies of group 1 are outstanding
  wait_vm_le<kGroup * CPT>(CPT * min(kGroup, max(0, T - kGroup)));
  __syncthreads();
  f32x16 a[2], b[2];
  unit_mfma<D, KEYS_A>(ring_lds, ring.rd, 0, qf, a, [](int) {});
  acc.first(a);
  for (int t = 0; t + 1 < T; ++t) {
    unit_mfma<D, KEYS_A>(ring_lds + (t % kRing) * TB, ring.rd, 1, qf, b,
                         [&](int s) { acc.slot(a, s, 2 * t, false); });
    acc.fin(a, 2 * t, false);
    if ((t + 1) % kGroup == 0) {
      wait_vm<0>();  // this wave's copies of the group that opens here
      __syncthreads();
      issue_group((t + 1) / kGroup + 1);
    }
    unit_mfma<D, KEYS_A>(ring_lds + ((t + 1) % kRing) * TB, ring.rd, 0, qf, a,
                         [&](int s) { acc.slot(b, s, 2 * t + 1, false); });
    acc.fin(b, 2 * t + 1, false);
  }
  unit_mfma<D, KEYS_A>(ring_lds + ((T - 1) % kRing) * TB, ring.rd, 1, qf, b,
                       [&](int s) { acc.slot(a, s, 2 * T - 2, true); });
  acc.fin(a, 2 * T - 2, true);
#pragma unroll
  for (int s = 0; s < NS; ++s) acc.slot(b, s, 2 * T - 1, true);
  acc.fin(b, 2 * T - 1, true);
  __syncthreads();
}

// Lane-local online log2-sum-exp over the keys of KEYS_A units, for the two
// query columns of the lane.  The running max m starts at the max of unit 0
// and is raised only when a unit's sum against it reaches kSumGuard, so the
// per-score work is one FMA, one exp2 and one add.  Keys >= key_end (tail of
// the last tile) are masked to -inf.
template <int D>
struct LseAcc {
  static constexpr int VPS = 32 / (D / 8);  // scores per lane per slot
  float m[2], l[2], rs[2];
  float c;
  int key_begin, key_end, g;

  __device__ __forceinline__ float val(const f32x16 (&x)[2], int h, int i, int u,
                                       bool last) const {
    const float v = x[h][i];
    return (last && key_begin + 32 * u + crow(i, g) >= key_end) ? -INFINITY : v;
  }
  __device__ __forceinline__ void first(const f32x16 (&x)[2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float mx = x[h][0];
#pragma unroll
      for (int i = 1; i < 16; ++i) mx = fmaxf(mx, x[h][i]);
      m[h] = mx * c;
      l[h] = 0.f;
    }
  }
  __device__ __forceinline__ void slot(const f32x16 (&x)[2], int s, int u, bool last) {
#pragma unroll
    for (int j = 0; j < VPS; ++j) {
      const int v = s * VPS + j, h = v >> 4, i = v & 15;
      const float p = fast_exp2(fmaf(val(x, h, i, u, last), c, -m[h]));
      rs[h] = i == 0 ? p : rs[h] + p;
    }
    // keep this slot's share beside its MFMA (the compiler would otherwise
    // sink it towards the first use of the sum)
    asm volatile("" : "+v"(rs[(s * VPS) >> 4]));
  }
  __device__ __forceinline__ void fin(const f32x16 (&x)[2], int u, bool last) {
    if (!(rs[0] < kSumGuard) || !(rs[1] < kSumGuard)) redo(x, u, last);
    l[0] += rs[0];
    l[1] += rs[1];
  }
  // Rare path: raise the running max to the unit's max and redo its sum.
  __device__ __forceinline__ void redo(const f32x16 (&x)[2], int u, bool last) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (!(rs[h] < kSumGuard)) {
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, val(x, h, i, u, last));
        const float mn = fmaxf(m[h], mx * c);
        float r = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) r += fast_exp2(fmaf(val(x, h, i, u, last), c, -mn));
        l[h] *= fast_exp2(m[h] - mn);
        m[h] = mn;
        rs[h] = r;
      }
    }
  }
  // (max, sum) of query column h over the keys of both lane halves.
  __device__ __forceinline__ float2 merged(int h) const {
    const float m2 = swap_halves(m[h]), l2 = swap_halves(l[h]);
    const float mm = fmaxf(m[h], m2);
    float lt = 0.f;
    if (mm > -INFINITY) lt = l[h] * fast_exp2(m[h] - mm) + l2 * fast_exp2(m2 - mm);
    return make_float2(mm, lt);
  }
};

// Column mass of !KEYS_A units: the lane sums 2^(S*c - lse_row) over its 32
// query rows and adds it to its own LDS slot of the unit's key (one writer
// per slot, fixed order).  Rows without a query carry lse = +inf.
template <int D>
struct ColAcc {
  static constexpr int VPS = 32 / (D / 8);
  float lr[2][16];
  float cs;
  float c;
  float* red;  // this lane's slot row, offset by its key column n

  __device__ __forceinline__ void first(const f32x16 (&)[2]) {}
  __device__ __forceinline__ void slot(const f32x16 (&x)[2], int s, int, bool) {
#pragma unroll
    for (int j = 0; j < VPS; ++j) {
      const int v = s * VPS + j, h = v >> 4, i = v & 15;
      const float p = fast_exp2(fmaf(x[h][i], c, -lr[h][i]));
      cs = v == 0 ? p : cs + p;
    }
    asm volatile("" : "+v"(cs));
  }
  __device__ __forceinline__ void fin(const f32x16 (&)[2], int u, bool) { red[32 * u] += cs; }
};

// ---- block means fused into the streams (Sec. 4.2, Eq. (6)) ------------------
// The mean of Q^v and of K^v over each block of `block` tokens (the last block
// over its true length), written as [d][n_pad] per (b,h) like the mask call's
// own pooling.  A sum of at most 128 bf16 values (8 significant bits each) is
// exact in fp64 whenever their magnitudes lie within 2^44 of each other, so
// the means equal that pooling bit for bit whatever the order of the
// additions, and are divided once.

// 8 bf16 of a 16-byte chunk added to acc in fp64.
__device__ __forceinline__ void add_bf16x8(u32x4 v, double (&acc)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc[2 * i] += static_cast<double>(__uint_as_float(v[i] << 16));
    acc[2 * i + 1] += static_cast<double>(__uint_as_float(v[i] & 0xffff0000u));
  }
}

// x summed over the 16 lanes of its DPP row, the same total in every lane:
// lane pairs (quad_perm 1,0,3,2), then quads (2,3,0,1), then the two halves
// of each 8 lanes (half-row mirror) and of the row (row mirror).  Each step
// moves the two dwords of x with DPP and adds in fp64.
__device__ __forceinline__ double dpp_row_sum(double x) {
  auto step = [](double v, int ctrl) {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    const int lo = static_cast<int>(u & 0xffffffffu), hi = static_cast<int>(u >> 32);
    int plo, phi;
    switch (ctrl) {  // the DPP control must be a constant
      case 0:
        plo = __builtin_amdgcn_mov_dpp(lo, 0xB1, 0xF, 0xF, false);
        phi = __builtin_amdgcn_mov_dpp(hi, 0xB1, 0xF, 0xF, false);
        break;
      case 1:
        plo = __builtin_amdgcn_mov_dpp(lo, 0x4E, 0xF, 0xF, false);
        phi = __builtin_amdgcn_mov_dpp(hi, 0x4E, 0xF, 0xF, false);
        break;
      case 2:
        plo = __builtin_amdgcn_mov_dpp(lo, 0x141, 0xF, 0xF, false);
        phi = __builtin_amdgcn_mov_dpp(hi, 0x141, 0xF, 0xF, false);
        break;
      default:
        plo = __builtin_amdgcn_mov_dpp(lo, 0x140, 0xF, 0xF, false);
        phi = __builtin_amdgcn_mov_dpp(hi, 0x140, 0xF, 0xF, false);
        break;
    }
    const uint64_t w = (static_cast<uint64_t>(static_cast<uint32_t>(phi)) << 32) |
                       static_cast<uint32_t>(plo);
    return v + __longlong_as_double(static_cast<long long>(w));
  };
  x = step(x, 0);
  x = step(x, 1);
  x = step(x, 2);
  return step(x, 3);
}

// Keys of a column-mass stream (K2), pooled from the LDS ring.  Lane l of
// wave w takes d quarter q = 4w + l/16 (d = 4q .. 4q+3) of key rows l % 16 and
// l % 16 + 16 of every 32-key unit, read while the unit's MFMAs run; at the
// end of a block the 16 lanes that share q (one DPP row) add their sums
// (dpp_row_sum), and the lane of row 0 writes the 4 means.  Waves from D/16
// on (at d = 64) take no part.
template <int D>
struct KeyPool {
  static constexpr int TB = KeyRing<D>::TB;
  double acc[4];
  u32x2 raw[2];
  const char* ring;    // LDS ring, stage 0
  int off;             // lane offset of its quarter of row l % 16 in a unit
  int key_begin, L, block, nunits, n_pad;
  bool on;             // wave-uniform: this wave pools
  double* dst;         // kbar + pair * D * n_pad

  __device__ __forceinline__ void init(const char* ring_lds, int wave, int lane, int key_begin_,
                                       int L_, int block_, int T, int n_pad_, double* dst_) {
    const int r = lane & 15;
    const int q = 4 * wave + (lane >> 4);  // = threadIdx.x / 16
    on = 4 * wave < D / 4;
    const int cc = q >> 1;  // 16-byte chunk; the plane swizzle of rows r, r + 16 and
                            // 32*kb + r is that of row r
    off = (cc >> 2) * 4096 + r * 64 + 16 * ((cc & 3) ^ plane_swz(r)) + 8 * (q & 1);
    ring = ring_lds;
    key_begin = key_begin_;
    L = L_;
    block = block_;
    nunits = 2 * T;
    n_pad = n_pad_;
    dst = dst_;
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = 0.0;
  }
  // unit p = keys key_begin + 32p ..; tile p/2 sits in stage (p/2) % kRing
  __device__ __forceinline__ void load(int p) {
    if (on && p < nunits) {
      const char* base = ring + ((p >> 1) % kRing) * TB + (p & 1) * 2048 + off;
      raw[0] = *reinterpret_cast<const u32x2*>(base);
      raw[1] = *reinterpret_cast<const u32x2*>(base + 16 * 64);
    }
  }
  // Dword part (0..3) of the unit's two rows: 2 elements.
  __device__ __forceinline__ void add(int p, int part) {
    if (on && p < nunits) {
      const int j = part >> 1, i = part & 1;
      uint32_t v = raw[j][i];
      // rows past L repeat row L-1 in the ring: they add nothing
      if (key_begin + 32 * p + 32 > L && key_begin + 32 * p + (threadIdx.x & 15) + 16 * j >= L)
        v = 0u;
      acc[2 * i] += static_cast<double>(__uint_as_float(v << 16));
      acc[2 * i + 1] += static_cast<double>(__uint_as_float(v & 0xffff0000u));
    }
  }
  // After unit p: at the end of a block, sum over the 32 rows and write.
  __device__ __forceinline__ void close(int p) {
    const int upb = block >> 5;  // units per block
    if (!on || p >= nunits || (p % upb != upb - 1 && p != nunits - 1)) return;
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = dpp_row_sum(acc[e]);
    const int c = (key_begin + 32 * p) / block;
    const int len = min(block, L - c * block);
    if ((threadIdx.x & 15) == 0) {
      const int q = threadIdx.x >> 4;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        dst[static_cast<size_t>(4 * q + e) * n_pad + c] = acc[e] / static_cast<double>(len);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = 0.0;
  }
};

// ColAcc with the keys' block means: unit p = u + 1 (whose MFMAs run beside
// the slots of unit u) is read a few slots in and added two elements at a
// time beside four of the later MFMAs; unit 0 is pooled in first().
template <int D>
struct ColPoolAcc : ColAcc<D> {
  KeyPool<D> pool;
  static constexpr int NS = D / 8;
  __device__ __forceinline__ void first(const f32x16 (&)[2]) {
    pool.load(0);
#pragma unroll
    for (int part = 0; part < 4; ++part) pool.add(0, part);
    pool.close(0);
  }
  __device__ __forceinline__ void slot(const f32x16 (&x)[2], int s, int u, bool last) {
    constexpr int GAP = NS / 8;  // slots between two parts
    if (s == NS / 4 - GAP) pool.load(u + 1);
    // the four dword parts beside four of the later MFMAs
    if (s >= NS / 4 && s < NS / 4 + 4 * GAP && (s - NS / 4) % GAP == 0)
      pool.add(u + 1, (s - NS / 4) / GAP);
    ColAcc<D>::slot(x, s, u, last);
  }
  __device__ __forceinline__ void fin(const f32x16 (&x)[2], int u, bool last) {
    ColAcc<D>::fin(x, u, last);
    pool.close(u + 1);
  }
};

// Query rows of a v->a workgroup (K3), pooled from a second load of the rows
// it has just loaded for its MFMAs (L2 hits).  Thread t takes block
// t / block of the kV2aChunk rows from row0, 16-byte chunk cc and every
// (block / CPR)-th row of that block (CPR rows); the partial sums go through
// `part` (32 KB of LDS, [thread][element]) and are added in a fixed order.
// Ends with a barrier, after which `part` may be reused.
template <int D>
__device__ __forceinline__ void pool_query_chunk(const uint16_t* __restrict__ src, int row0,
                                                 int L, int block, int n_pad,
                                                 double* __restrict__ dst, double* part) {
  constexpr int CPR = D / 8;
  const int t = threadIdx.x;
  const int bl = t / block, w = t % block;
  const int cc = w % CPR, rg = w / CPR;
  const int RG = block / CPR;  // row groups of a block
  const int rb = row0 + bl * block;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll
  for (int i0 = 0; i0 < CPR; i0 += 8) {
    u32x4 raw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = rb + rg + RG * (i0 + i);
      raw[i] = r < L ? ldg16(src + static_cast<size_t>(r) * D + 8 * cc)
                     : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) add_bf16x8(raw[i], acc);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[8 * t + e] = acc[e];
  __syncthreads();
  const int nbl = kV2aChunk / block;
  for (int o = t; o < nbl * D; o += kXNT) {
    const int b2 = o / D, dd = o % D;
    const int rs = row0 + b2 * block;
    if (rs >= L) continue;
    const int len = min(block, L - rs);
    const int base = b2 * block + dd / 8;  // thread of row group 0, chunk dd / 8
    double sum = 0.0;
    for (int g = 0; g < RG; ++g) sum += part[8 * (base + g * CPR) + (dd & 7)];
    dst[static_cast<size_t>(dd) * n_pad + rs / block] = sum / static_cast<double>(len);
  }
  __syncthreads();
}

// ---- K1 ---------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kXNT) __attribute__((amdgpu_waves_per_eu(2, 2)))
a2v_lse_partial_kernel(const uint16_t* __restrict__ q_a,
                       const uint16_t* __restrict__ k_v,
                       float2* __restrict__ part, int L_v, int L_a, int nchunk,
                       float c) {
  __shared__ __attribute__((aligned(1024))) char ring_lds[kRing * KeyRing<D>::TB];
  const int chunk = blockIdx.x, slab = blockIdx.y, pair = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 5, n = lane & 31;
  const int j0 = slab * kQSlab + wave * 64;  // first audio query row of the wave
  const int key_begin = chunk * kLseChunk;
  const int key_end = min(key_begin + kLseChunk, L_v);

  u32x4 qf[2][D / 16];
  const uint16_t* qh = q_a + static_cast<size_t>(pair) * L_a * D;
  load_qfrag<D>(qh, j0 + n, L_a, g, qf[0]);
  load_qfrag<D>(qh, j0 + 32 + n, L_a, g, qf[1]);
  KeyRing<D> ring;
  ring.init(ring_lds, wave, lane);
  LseAcc<D> acc;
  acc.c = c;
  acc.key_begin = key_begin;
  acc.key_end = key_end;
  acc.g = g;
  stream_keys<D, true>(ring, ring_lds,
                       reinterpret_cast<const char*>(k_v + static_cast<size_t>(pair) * L_v * D),
                       key_begin, L_v, ceil_div(key_end - key_begin, 64), qf, acc);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const float2 ml = acc.merged(h);
    const int j = j0 + 32 * h + n;
    if (g == 0 && j < L_a)
      part[(static_cast<size_t>(pair) * nchunk + chunk) * L_a + j] = ml;
  }
}

// lse2[pair][j] = log2(sum over chunks of l * 2^m), merged in chunk order
// (max first, then the sum); one thread per (pair, j), loads in batches of 8.
__global__ void __launch_bounds__(64)
lse_combine_kernel(const float2* __restrict__ part, float* __restrict__ lse2, int P,
                   int L_a, int nchunk) {
  const size_t t = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<size_t>(P) * L_a) return;
  const size_t pair = t / L_a, j = t % L_a;
  const float2* p = part + pair * nchunk * L_a + j;
  float M = -INFINITY;
  for (int c0 = 0; c0 < nchunk; c0 += 8) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      v[k] = c0 + k < nchunk ? p[static_cast<size_t>(c0 + k) * L_a].x : -INFINITY;
#pragma unroll
    for (int k = 0; k < 8; ++k) M = fmaxf(M, v[k]);
  }
  float S = 0.f;
  for (int c0 = 0; c0 < nchunk; c0 += 8) {
    float2 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      v[k] = c0 + k < nchunk ? p[static_cast<size_t>(c0 + k) * L_a] : make_float2(0.f, 0.f);
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (v[k].y > 0.f) S += v[k].y * fast_exp2(v[k].x - M);
  }
  lse2[t] = M + __log2f(S);
}

// ---- K2 ---------------------------------------------------------------------
// a->v column mass: grid (ceil(L_v/1024), H, B); the workgroup streams its
// 1024 video keys once per slab of 512 audio queries (S = Q^a K^v^T, a lane
// owns a key column) and adds exp2(S*c - lse) into per-lane LDS slots; the 16
// slots of a key (8 waves x 2 lane halves) are then summed in a fixed order.
// Keys past L_v only reach their own columns, which are not written.
// POOL: the stream of the first slab also writes the block means of K^v
// (KeyPool) to kbar ([B,H,d,n_pad]).
template <int D, bool POOL>
__global__ void __launch_bounds__(kXNT) __attribute__((amdgpu_waves_per_eu(2, 2)))
a2v_colmass_kernel(const uint16_t* __restrict__ q_a,
                   const uint16_t* __restrict__ k_v,
                   const float* __restrict__ lse2, float* __restrict__ colmass,
                   int H, int L_v, int L_a, float c, double* __restrict__ kbar, int block,
                   int n_pad) {
  constexpr int RS = kColKeys + 32;  // slot row stride (the two lane halves use different banks)
  __shared__ __attribute__((aligned(1024))) char ring_lds[kRing * KeyRing<D>::TB];
  __shared__ float red[2 * kXW][RS];
  const int chunk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 5, n = lane & 31;
  const int key_begin = chunk * kColKeys;
  const int key_end = min(key_begin + kColKeys, L_v);
  const size_t pair = static_cast<size_t>(b) * H + h;
  const uint16_t* qh = q_a + pair * L_a * D;
  const float* lh = lse2 + pair * L_a;
  const char* kh = reinterpret_cast<const char*>(k_v + pair * L_v * D);
  const int T = ceil_div(key_end - key_begin, 64);

  KeyRing<D> ring;
  ring.init(ring_lds, wave, lane);
  ColAcc<D> acc;
  acc.c = c;
  acc.red = &red[2 * wave + g][n];
  for (int k = 0; k < kColKeys; k += 32) acc.red[k] = 0.f;  // the lane's own slots

  for (int slab = 0; slab * kQSlab < L_a; ++slab) {
    const int j0 = slab * kQSlab + wave * 64;
    u32x4 qf[2][D / 16];
    load_qfrag<D>(qh, j0 + n, L_a, g, qf[0]);
    load_qfrag<D>(qh, j0 + 32 + n, L_a, g, qf[1]);
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int jj = j0 + 32 * hh + crow(i, g);
        acc.lr[hh][i] = jj < L_a ? lh[jj] : INFINITY;
      }
    if (POOL && slab == 0) {
      ColPoolAcc<D> pacc;
      static_cast<ColAcc<D>&>(pacc) = acc;
      pacc.pool.init(ring_lds, wave, lane, key_begin, L_v, block, T, n_pad,
                     kbar + pair * D * n_pad);
      stream_keys<D, false>(ring, ring_lds, kh, key_begin, L_v, T, qf, pacc);
    } else {
      stream_keys<D, false>(ring, ring_lds, kh, key_begin, L_v, T, qf, acc);
    }
  }
  for (int k = threadIdx.x; k < kColKeys; k += kXNT) {
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < 2 * kXW; ++w) sum += red[w][k];
    if (key_begin + k < L_v) colmass[pair * L_v + key_begin + k] = sum;
  }
}

// ---- K3 ---------------------------------------------------------------------
// v->a column mass: grid (ceil(L_v/512), 1, P).  The workgroup holds 512
// video queries; pass 1 streams every audio key with S^T = K^a Q^v^T (a lane
// owns a video query) for its log2-sum-exp, pass 2 streams the audio keys
// again, one window of 512 at a time, with S = Q^v K^a^T and sums the column
// mass of each key over the 512 queries (per-lane LDS slots, fixed order).
// FROM_LSE: pass 1 is replaced by the natural-log LSE of each video query
// that a v->a cross-attention forward produced (lse_v [P][L_v]).
// qbar != NULL: the workgroup first writes the block means of its 512 video
// queries (pool_query_chunk) to qbar ([B,H,d,n_pad]).
template <int D, bool FROM_LSE>
__global__ void __launch_bounds__(kXNT) __attribute__((amdgpu_waves_per_eu(2, 2)))
v2a_colmass_kernel(const uint16_t* __restrict__ q_v,
                   const uint16_t* __restrict__ k_a, float* __restrict__ part,
                   int L_v, int L_a, int nchunk, float c, const float* __restrict__ lse_v,
                   double* __restrict__ qbar, int block, int n_pad) {
  constexpr int RS = kAWin + 32;
  __shared__ __attribute__((aligned(1024))) char ring_lds[kRing * KeyRing<D>::TB];
  __shared__ float red[2 * kXW][RS];
  __shared__ float lse_w[kXW][64];
  const int chunk = blockIdx.x, pair = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 5, n = lane & 31;
  const int i0 = chunk * kV2aChunk + wave * 64;  // first video query row of the wave
  const char* kah = reinterpret_cast<const char*>(k_a + static_cast<size_t>(pair) * L_a * D);

  u32x4 qf[2][D / 16];
  const uint16_t* qh = q_v + static_cast<size_t>(pair) * L_v * D;
  load_qfrag<D>(qh, i0 + n, L_v, g, qf[0]);
  load_qfrag<D>(qh, i0 + 32 + n, L_v, g, qf[1]);
  KeyRing<D> ring;
  ring.init(ring_lds, wave, lane);
  if (qbar != nullptr)  // the ring is free until the first stream
    pool_query_chunk<D>(qh, chunk * kV2aChunk, L_v, block, n_pad,
                        qbar + static_cast<size_t>(pair) * D * n_pad,
                        reinterpret_cast<double*>(ring_lds));

  if constexpr (FROM_LSE) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int row = i0 + 32 * h + n;
      if (g == 0)
        lse_w[wave][32 * h + n] =
            row < L_v ? lse_v[static_cast<size_t>(pair) * L_v + row] * kLog2e : INFINITY;
    }
  } else {
    // pass 1: log2-sum-exp of every video query over all audio keys
    LseAcc<D> acc;
    acc.c = c;
    acc.key_begin = 0;
    acc.key_end = L_a;
    acc.g = g;
    stream_keys<D, true>(ring, ring_lds, kah, 0, L_a, ceil_div(L_a, 64), qf, acc);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float2 ml = acc.merged(h);
      // rows past L_v get +inf: their probabilities are exactly 0
      if (g == 0) lse_w[wave][32 * h + n] = (i0 + 32 * h + n < L_v) ? ml.x + __log2f(ml.y) : INFINITY;
    }
  }
  __syncthreads();

  // pass 2: column mass of the audio keys, one window of 512 keys at a time
  ColAcc<D> acc;
  acc.c = c;
  acc.red = &red[2 * wave + g][n];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc.lr[h][i] = lse_w[wave][32 * h + crow(i, g)];
  for (int key_begin = 0; key_begin < L_a; key_begin += kAWin) {
    const int key_end = min(key_begin + kAWin, L_a);
    if (key_begin > 0) __syncthreads();  // the previous window's slots have been read
    for (int k = 0; k < kAWin; k += 32) acc.red[k] = 0.f;
    // ends with a barrier: every wave's slots are complete below
    stream_keys<D, false>(ring, ring_lds, kah, key_begin, L_a,
                          ceil_div(key_end - key_begin, 64), qf, acc);
    for (int k = threadIdx.x; k < key_end - key_begin; k += kXNT) {
      float sum = 0.f;
#pragma unroll
      for (int w = 0; w < 2 * kXW; ++w) sum += red[w][k];
      part[(static_cast<size_t>(pair) * nchunk + chunk) * L_a + key_begin + k] = sum;
    }
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
    v = sum_strided(colmass + static_cast<size_t>(b) * nsum * L_v + i, L_v, nsum);
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
  if (j < L_a && ph < nchunk)
    v = sum_strided(part + (pair * nchunk + ph) * L_a + j, 4 * static_cast<size_t>(L_a),
                    (nchunk - ph + 3) / 4);
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
  float v = sum_strided(part + b * nparts * L_a + j, L_a, nparts);
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

// K2, with the block means of K^v written to kbar when it is not NULL.
template <int D>
void launch_a2v_colmass(const uint16_t* q_a, const uint16_t* k_v, const float* lse2,
                        float* colmass, int B, int H, int L_v, int L_a, float c, double* kbar,
                        int block, hipStream_t s) {
  const dim3 grid(ceil_div(L_v, kColKeys), H, B);
  const int n_pad = mask_n_pad(ceil_div(L_v, block));
  if (kbar != nullptr)
    hipLaunchKernelGGL((a2v_colmass_kernel<D, true>), grid, dim3(kXNT), 0, s, q_a, k_v, lse2,
                       colmass, H, L_v, L_a, c, kbar, block, n_pad);
  else
    hipLaunchKernelGGL((a2v_colmass_kernel<D, false>), grid, dim3(kXNT), 0, s, q_a, k_v, lse2,
                       colmass, H, L_v, L_a, c, kbar, block, n_pad);
}

template <int D>
void cross_bf16(const uint16_t* q_a, const uint16_t* k_v, const uint16_t* q_v,
                const uint16_t* k_a, int B, int H, int L_v, int L_a, float scale,
                int block, float* sal_v_tok, float* sal_v_blk, float* sal_a_tok,
                int accumulate, double* qbar, double* kbar, char* ws, hipStream_t s) {
  const CrossWs lay = cross_ws_layout(B, H, L_v, L_a);
  const float c = scale * kLog2e;
  const int P = B * H;
  const int nchunk = ceil_div(L_v, kLseChunk);
  const int nslab = ceil_div(L_a, kQSlab);
  float2* lse_part = reinterpret_cast<float2*>(ws + lay.lse_part);
  float* lse_a = reinterpret_cast<float*>(ws + lay.lse_a);
  float* colmass = reinterpret_cast<float*>(ws + lay.colmass);
  hipLaunchKernelGGL(a2v_lse_partial_kernel<D>, dim3(nchunk, nslab, P), dim3(kXNT), 0, s,
                     q_a, k_v, lse_part, L_v, L_a, nchunk, c);
  const size_t nlse = static_cast<size_t>(P) * L_a;
  hipLaunchKernelGGL(lse_combine_kernel, dim3((nlse + 63) / 64), dim3(64), 0, s,
                     lse_part, lse_a, P, L_a, nchunk);
  launch_a2v_colmass<D>(q_a, k_v, lse_a, colmass, B, H, L_v, L_a, c, kbar, block, s);
  const int n_b = ceil_div(L_v, block);
  hipLaunchKernelGGL(a2v_finalize_kernel, dim3(n_b, B), dim3(block), 0, s, colmass,
                     sal_v_tok, sal_v_blk, L_v, H,
                     1.0f / (static_cast<float>(H) * static_cast<float>(L_a)), accumulate);
  if (q_v != nullptr) {
    float* v2a_part = reinterpret_cast<float*>(ws + lay.v2a_part);
    const int nchunk3 = ceil_div(L_v, kV2aChunk);
    float* v2a_head = reinterpret_cast<float*>(ws + lay.v2a_head);
    hipLaunchKernelGGL((v2a_colmass_kernel<D, false>), dim3(nchunk3, 1, P),
                       dim3(kXNT), 0, s, q_v, k_a, v2a_part, L_v, L_a, nchunk3, c, nullptr,
                       qbar, block, mask_n_pad(ceil_div(L_v, block)));
    hipLaunchKernelGGL(v2a_chunk_sum_kernel, dim3(ceil_div(L_a, 64), P), dim3(256), 0, s,
                       v2a_part, v2a_head, L_a, nchunk3);
    const size_t na = static_cast<size_t>(B) * L_a;
    hipLaunchKernelGGL(v2a_finalize_kernel, dim3((na + 255) / 256), dim3(256), 0, s,
                       v2a_head, sal_a_tok, B, H, L_a,
                       1.0f / (static_cast<float>(H) * static_cast<float>(L_v)), accumulate);
  }
}

// lse2 = lse * log2(e): natural-log LSE of the scaled scores to the log2
// units of the key-stream kernels.
__global__ void __launch_bounds__(256)
lse_to_log2_kernel(const float* __restrict__ lse, float* __restrict__ lse2, size_t n) {
  for (size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<size_t>(gridDim.x) * 256)
    lse2[i] = lse[i] * kLog2e;
}

// The saliency of both directions from the row LSEs of the two cross-
// attention forwards: K2 and K3's column-mass pass only.
template <int D>
void cross_bf16_from_lse(const uint16_t* q_a, const uint16_t* k_v, const uint16_t* q_v,
                         const uint16_t* k_a, const float* lse_a, const float* lse_v, int B,
                         int H, int L_v, int L_a, float scale, int block, float* sal_v_tok,
                         float* sal_v_blk, float* sal_a_tok, int accumulate, double* qbar,
                         double* kbar, char* ws, hipStream_t s) {
  const CrossWs lay = cross_ws_layout(B, H, L_v, L_a);
  const float c = scale * kLog2e;
  const int P = B * H;
  float* lse2 = reinterpret_cast<float*>(ws + lay.lse_a);
  float* colmass = reinterpret_cast<float*>(ws + lay.colmass);
  const size_t nlse = static_cast<size_t>(P) * L_a;
  const size_t cblocks = (nlse + 255) / 256;
  hipLaunchKernelGGL(lse_to_log2_kernel, dim3(static_cast<unsigned>(cblocks < 1024 ? cblocks : 1024)),
                     dim3(256), 0, s, lse_a, lse2, nlse);
  launch_a2v_colmass<D>(q_a, k_v, lse2, colmass, B, H, L_v, L_a, c, kbar, block, s);
  const int n_b = ceil_div(L_v, block);
  hipLaunchKernelGGL(a2v_finalize_kernel, dim3(n_b, B), dim3(block), 0, s, colmass,
                     sal_v_tok, sal_v_blk, L_v, H,
                     1.0f / (static_cast<float>(H) * static_cast<float>(L_a)), accumulate);
  if (q_v != nullptr) {
    float* v2a_part = reinterpret_cast<float*>(ws + lay.v2a_part);
    const int nchunk3 = ceil_div(L_v, kV2aChunk);
    float* v2a_head = reinterpret_cast<float*>(ws + lay.v2a_head);
    hipLaunchKernelGGL((v2a_colmass_kernel<D, true>), dim3(nchunk3, 1, P),
                       dim3(kXNT), 0, s, q_v, k_a, v2a_part, L_v, L_a, nchunk3, c, lse_v,
                       qbar, block, mask_n_pad(ceil_div(L_v, block)));
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
                              float* sal_a_tok, int accumulate, double* qbar,
                              double* kbar, char* ws, hipStream_t s) {
  if (d == 128)
    cross_bf16<128>(q_a, k_v, q_v, k_a, B, H, L_v, L_a, scale, block, sal_v_tok,
                    sal_v_blk, sal_a_tok, accumulate, qbar, kbar, ws, s);
  else
    cross_bf16<64>(q_a, k_v, q_v, k_a, B, H, L_v, L_a, scale, block, sal_v_tok,
                   sal_v_blk, sal_a_tok, accumulate, qbar, kbar, ws, s);
}

void launch_cross_scores_from_lse_bf16(const uint16_t* q_a, const uint16_t* k_v,
                                       const uint16_t* q_v, const uint16_t* k_a,
                                       const float* lse_a, const float* lse_v, int B, int H,
                                       int L_v, int L_a, int d, float scale, int block,
                                       float* sal_v_tok, float* sal_v_blk, float* sal_a_tok,
                                       int accumulate, double* qbar, double* kbar,
                                       char* ws, hipStream_t s) {
  if (d == 128)
    cross_bf16_from_lse<128>(q_a, k_v, q_v, k_a, lse_a, lse_v, B, H, L_v, L_a, scale, block,
                             sal_v_tok, sal_v_blk, sal_a_tok, accumulate, qbar, kbar, ws, s);
  else
    cross_bf16_from_lse<64>(q_a, k_v, q_v, k_a, lse_a, lse_v, B, H, L_v, L_a, scale, block,
                            sal_v_tok, sal_v_blk, sal_a_tok, accumulate, qbar, kbar, ws, s);
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
