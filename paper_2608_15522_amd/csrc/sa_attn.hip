// Protected block-sparse flash attention (Sec. 4.2, Eq. (10) in the row
// form of Eq. (11); Eq. (5) when a list holds every key block).
//
// bf16 path (MFMA, gfx950)
// ------------------------
// One workgroup per query block (BLOCK rows, BLOCK/32 waves of 32 query rows
// each).  The workgroup walks its compacted key-block list; every key block
// is streamed as 64-key tiles of K and V into double-buffered LDS by
// global_load_lds_dwordx4 (planes of 32 d per key, 16-byte slots swizzled by
// row), so the copy of tile t+1 runs under the math of tile t without
// staging registers.  Each wave computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16,
// so a lane owns one query column: the row max and row sum of the online
// softmax are lane-local, plus one exchange with the lane holding the other
// 16 keys of the same query.  P^T is packed to bf16 in registers and feeds
// O^T += V^T P^T directly as the B operand; the V^T operand is read from the
// key-major tile with ds_read_b64_tr_b16 (a transposing LDS read).  The row
// sum is taken on the same bf16 probabilities with v_dot2_f32_bf16 (the
// gather form adds the fp32 probabilities instead, for an lse exact to fp32
// rounding).  The scale is folded into exp2; the running output is rescaled
// only when a lane's max grows by more than 2^8.  Keys past L are -inf, rows
// past L are never written.
//
// Query blocks of a (batch, head) pair are launched heaviest list first
// (protected rows hold the full list).  With a pair count that is a multiple
// of 8, each XCD takes every 8th pair: first the full rows of all its pairs,
// then the other rows one pair at a time, so that a pair's K/V blocks are
// shared through one XCD's L2 and the long full rows do not run alone at the
// end of the launch; otherwise the launch is rank-major over pairs.
//
// Gather form: dense rows gathered by index (protected tokens) or all rows
// of a query tensor of another length (cross-modal attention), every key
// kept; the keys of a row block may be split into runs whose partial rows
// token_combine_kernel merges.
//
// f32 path: a plain per-row online softmax with K/V tiles in LDS (used by the
// small fp32 workloads; fp32 MFMA would not change its role).
#include <algorithm>

#include "sa_device.h"
#include "sa_internal.h"

namespace sa {
namespace {

constexpr int kTile = 64;       // keys per LDS tile
constexpr int kCusPerXcd = 32;  // MI355X: 8 XCDs of 32 CUs

// Query blocks of every (b,h) pair ordered by kv_cnt descending, then by
// block index ascending.  Each block gets the key (n_b - cnt) * 4096 + index,
// unique and in that order, and its rank is the number of smaller keys.
// Grid (pairs, ceil(n_b / kOrderRows)): every workgroup loads the pair's keys
// into LDS and ranks kOrderRows of its blocks, reading the keys four at a time
// (entries past n_b hold INT_MAX and never count).
constexpr int kOrderRows = 256;
__global__ void __launch_bounds__(kOrderRows)
order_rows_kernel(const int32_t* __restrict__ kv_cnt, int32_t* __restrict__ order,
                  int n_b) {
  __shared__ __attribute__((aligned(16))) int key[kMaxBlocks];
  const size_t base = static_cast<size_t>(blockIdx.x) * n_b;
  const int n4 = ceil_div(n_b, 4);
  for (int r = threadIdx.x; r < 4 * n4; r += blockDim.x) {
    int k = 0x7fffffff;
    if (r < n_b) {
      int c = kv_cnt[base + r];
      c = c < 0 ? 0 : (c > n_b ? n_b : c);
      k = (n_b - c) * 4096 + r;
    }
    key[r] = k;
  }
  __syncthreads();
  const int r = blockIdx.y * kOrderRows + threadIdx.x;
  if (r >= n_b) return;
  const int mine = key[r];
  const int4* k4 = reinterpret_cast<const int4*>(key);
  int rk[4] = {0, 0, 0, 0};
#pragma unroll 4
  for (int j4 = 0; j4 < n4; ++j4) {
    const int4 o = k4[j4];
    rk[0] += o.x < mine;
    rk[1] += o.y < mine;
    rk[2] += o.z < mine;
    rk[3] += o.w < mine;
  }
  order[base + (rk[0] + rk[1]) + (rk[2] + rk[3])] = r;
}

// Launch schedule when the pair count is a multiple of 8.  Workgroup w runs
// on XCD w % 8, which owns the pairs x, x+8, x+16, ...; entry i of XCD x's
// list (pair << 11 | query block) is the work of its workgroup 8*i + x.  The
// list holds first the full rows (lists of all n_b key blocks: the protected
// query blocks) of every pair the XCD owns, pair by pair, then the other rows
// pair by pair, each pair's rows in launch order (heaviest list first).  A
// full row takes n_b / k_keep times as long as the others; started first, the
// full rows of the XCD's last pairs no longer run alone at the end of the
// launch, while the other rows still go through one pair at a time, so that
// their K/V blocks are shared through the XCD's L2.
__global__ void __launch_bounds__(1024)
schedule_rows_kernel(const int32_t* __restrict__ kv_cnt, const int32_t* __restrict__ order,
                     int32_t* __restrict__ sched, int* __restrict__ claim, int P, int n_b) {
  __shared__ int nfull[kMaxPairs / 8 + 1];
  __shared__ int total_full;
  const int x = blockIdx.x, np = P >> 3, tid = threadIdx.x;
  if (tid == 0) claim[64 * x] = 0;  // the attention kernel's row counter of XCD x
  for (int j = 0; j < np; ++j) {
    const size_t base = static_cast<size_t>(x + 8 * j) * n_b;
    int nf = 0;
    for (int r0 = 0; r0 < n_b; r0 += blockDim.x) {
      const int r = r0 + tid;
      nf += __syncthreads_count(r < n_b && kv_cnt[base + r] >= n_b);
    }
    if (tid == 0) nfull[j] = nf;
  }
  __syncthreads();
  if (tid == 0) {  // exclusive prefix over the pairs, in pair order
    int acc = 0;
    for (int j = 0; j < np; ++j) {
      const int nf = nfull[j];
      nfull[j] = acc;
      acc += nf;
    }
    nfull[np] = acc;
    total_full = acc;
  }
  __syncthreads();
  int32_t* out = sched + static_cast<size_t>(x) * np * n_b;
  const int F = total_full;
  for (int j = 0; j < np; ++j) {
    const int pair = x + 8 * j;
    const size_t base = static_cast<size_t>(pair) * n_b;
    const int fpre = nfull[j], nf = nfull[j + 1] - fpre;
    const int rest_pre = j * n_b - fpre;  // other rows of the earlier pairs
    for (int rank = tid; rank < n_b; rank += blockDim.x) {
      const int pos = rank < nf ? fpre + rank : F + rest_pre + (rank - nf);
      out[pos] = (pair << 11) | order[base + rank];
    }
  }
}

typedef __attribute__((address_space(3))) uint16_t lds_u16_t;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

// Rescale the running output only when some lane's max has grown by more
// than 2^8: the stale max keeps every probability below 256, exact after the
// final division by the row sum taken against the same max.
constexpr float kRescaleSlack = 8.0f;

template <bool B>
struct CopyFlag {
  static constexpr bool value = B;
};

// Max of x over the two lanes n and n+32 (robust to which half each output
// of the swap carries).
__device__ __forceinline__ float max_halves(float x) {
  const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                   false, false);
  return fmaxf(x, fmaxf(__uint_as_float(pr[0]), __uint_as_float(pr[1])));
}

// GATHER (dense rows): queries and outputs have Lq rows per pair, keys and
// values L.  Workgroup row j of pair (b,h) is query rows[b*n_rows + j], or j
// itself when rows is NULL (rows >= n_rows, or a query outside [0, Lq), are
// skipped); kv_idx, kv_cnt and order are not read.  This serves the dense
// rows of protected tokens (Eq. (11) first case, Lq == L) and cross-modal
// attention (Lq != L).  The key blocks are cut into n_split equal runs, one
// per workgroup: with n_split == 1 the workgroup keeps every key and writes
// O and lse to the query's own row; otherwise it writes its unnormalised O,
// running max m (log2 units) and row sum to `part` for token_combine_kernel.
template <int D, int BLOCK, bool GATHER>
__global__ void __launch_bounds__(BLOCK * 2) __attribute__((amdgpu_waves_per_eu(2, 2)))
sparse_attn_bf16_kernel(const uint16_t* __restrict__ q,
                        const uint16_t* __restrict__ k,
                        const uint16_t* __restrict__ v,
                        uint16_t* __restrict__ o, float* __restrict__ lse,
                        const int32_t* __restrict__ kv_idx,
                        const int32_t* __restrict__ kv_cnt,
                        const int32_t* __restrict__ order,
                        const int32_t* __restrict__ sched, int* __restrict__ claim, int P,
                        int L, int n_b, float c, const int32_t* __restrict__ rows,
                        int n_rows, int H, int n_split, float* __restrict__ part, int Lq) {
  constexpr int NW = BLOCK / 32;             // waves per workgroup
  constexpr int TPB = BLOCK / kTile;         // tiles per key block
  constexpr int KC = D / 16;                 // k-steps of Q K^T
  constexpr int DT = D / 32;                 // 32-row d tiles of O^T (= planes)
  constexpr int SPANS = kTile * D * 2 / 1024;
  constexpr int NI = SPANS / NW;             // DMA instructions per wave per matrix
  constexpr int TILE_ELEMS = kTile * D;
  static_assert(SPANS % NW == 0, "tile spans must split over waves");

  __shared__ __attribute__((aligned(1024))) uint16_t Ks[2][TILE_ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t Vs[2][TILE_ELEMS];
  __shared__ uint16_t tiles[kMaxBlocks * TPB];  // valid tiles, as key0 / 64
  __shared__ int ntiles_sh, nfull_sh, item_sh;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave_u = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, n = lane & 31;

  // Workgroup w runs on XCD w % 8.  Block lists with a pair count that is a
  // multiple of 8: the workgroups are persistent, and those of XCD x take
  // rows from x's launch list (its pairs' full rows, then its pairs one at a
  // time, so that a pair's K/V blocks are shared through one L2) by an atomic
  // counter per XCD; once that list is used up they take rows from the other
  // XCDs' lists, which evens out XCDs that run at different speeds.  Each row
  // is computed the same way whichever workgroup takes it.  Otherwise there
  // is one workgroup per row (dense rows: XCD-major over pairs).
  const bool persistent = !GATHER && (P & 7) == 0;
  const int per_xcd = (P >> 3) * n_b;  // rows in each XCD's list (persistent form)
  const int xcd = blockIdx.x & 7;
  int exhausted = 0;                   // lists found empty (thread 0)
  for (int item_iter = 0;; ++item_iter) {
  const int n_qr = GATHER ? ceil_div(n_rows, BLOCK) : n_b;  // query blocks per pair
  const int n_q = GATHER ? n_qr * n_split : n_b;              // workgroups per pair
  int pair, rank = 0, r = 0;
  if (persistent) {
    if (tid == 0) {
      int item = -1;
      for (int k = 0; k < 8 && item < 0; ++k) {
        const int xq = (xcd + k) & 7;
        if (exhausted & (1 << xq)) continue;
        const int i = atomicAdd(claim + 64 * xq, 1);
        if (i < per_xcd)
          item = xq * per_xcd + i;
        else
          exhausted |= 1 << xq;
      }
      item_sh = item;
    }
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(item_sh);  // uniform: scalar addressing
    if (item < 0) break;
    const int e = __builtin_amdgcn_readfirstlane(sched[item]);
    pair = e >> 11;
    r = e & 2047;
  } else {
    if (item_iter > 0) break;
    if (GATHER && (P & 7) == 0) {
      const int i = blockIdx.x >> 3;
      pair = (blockIdx.x & 7) + 8 * (i / n_q);
      rank = i % n_q;
    } else {
      pair = blockIdx.x % P;
      rank = blockIdx.x / P;
    }
  }
  const size_t row_base = static_cast<size_t>(pair) * n_b;
  int cnt, kb0 = 0, split = 0;
  const int32_t* idx = nullptr;
  if constexpr (GATHER) {
    // consecutive ranks share a key run and so its K/V tiles in L2
    split = rank / n_qr;
    r = rank - split * n_qr;
    kb0 = n_b * split / n_split;
    cnt = n_b * (split + 1) / n_split - kb0;
  } else {
    if (!persistent) r = order[row_base + rank];
    cnt = kv_cnt[row_base + r];
    cnt = cnt < 0 ? 0 : (cnt > n_b ? n_b : cnt);
    idx = kv_idx + (row_base + r) * n_b;
  }

  // Compact the list into 64-key tiles (wave 0): entries outside [0, n_b)
  // are dropped, and so is the second half of a last block of <= 64 keys.
  // Full tiles keep the list order; the tile that reaches past L (at most
  // one per list entry of block n_b-1) is placed after all of them, so that
  // only the last iterations mask keys.
  if (tid < 64) {
    int nfull = 0, npart = 0;
    const uint64_t below = (1ull << lane) - 1ull;
    for (int i0 = 0; i0 < cnt; i0 += 64) {
      const int i = i0 + lane;
      const int kb = i < cnt ? (GATHER ? kb0 + i : idx[i]) : -1;
      const bool v0 = kb >= 0 && kb < n_b;
      const bool v1 = TPB == 2 && v0 && kb * BLOCK + kTile < L;
      const bool f0 = v0 && kb * BLOCK + kTile <= L;
      const bool f1 = v1 && kb * BLOCK + 2 * kTile <= L;  // implies f0
      const uint64_t b0 = __ballot(f0), b1 = __ballot(f1);
      const int pos = nfull + __popcll(b0 & below) + __popcll(b1 & below);
      if (f0) tiles[pos] = static_cast<uint16_t>(kb * TPB);
      if (f1) tiles[pos + 1] = static_cast<uint16_t>(kb * TPB + 1);
      nfull += __popcll(b0) + __popcll(b1);
      npart += __popcll(__ballot(v0 && !f0)) + __popcll(__ballot(v1 && !f1));
    }
    for (int j = lane; j < npart; j += 64)
      tiles[nfull + j] = static_cast<uint16_t>((L - 1) / kTile);
    if (lane == 0) {
      ntiles_sh = nfull + npart;
      nfull_sh = nfull;
    }
  }

  const int LQ = GATHER ? Lq : L;  // query and output rows per pair
  const uint16_t* qh = q + static_cast<size_t>(pair) * LQ * D;
  const char* kh = reinterpret_cast<const char*>(k + static_cast<size_t>(pair) * L * D);
  const char* vh = reinterpret_cast<const char*>(v + static_cast<size_t>(pair) * L * D);

  int qrow = r * BLOCK + (tid >> 6) * 32 + n;
  if constexpr (GATHER) {
    if (qrow >= n_rows)
      qrow = -1;
    else if (rows != nullptr)
      qrow = rows[static_cast<size_t>(pair / H) * n_rows + qrow];
    if (qrow >= LQ) qrow = -1;
  }
  const bool qvalid = GATHER ? qrow >= 0 : qrow < L;
  u32x4 qf[KC];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc) {
    qf[kc] = qvalid ? ldg16(qh + static_cast<size_t>(qrow) * D + 16 * kc + 8 * g)
                    : u32x4{0u, 0u, 0u, 0u};
  }

  // DMA instruction i of wave w fills span w + NW*i of a tile: its lanes
  // cover key row 16*(span%4) + lane/4 of plane span/4, and lane l's source is
  // the logical 16-byte slot that the swizzle stores at physical slot l%4.
  int dma_row[NI];
  uint32_t dma_col[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int span = wave_u + NW * i;
    dma_row[i] = 16 * (span & 3) + (lane >> 2);
    dma_col[i] = static_cast<uint32_t>((span >> 2) * 64 +
                                       16 * ((lane & 3) ^ plane_swz(dma_row[i])));
  }

  // Lane-constant LDS byte offsets of the operand reads.
  //  K (A operand of S^T = K Q^T): row 32*st + n, slot 2*(kc&1) + g of plane kc/2.
  const int k_off0 = n * 64 + 16 * ((0 + g) ^ plane_swz(n));
  const int k_off1 = n * 64 + 16 * ((2 + g) ^ plane_swz(n));
  //  V (ds_read_b64_tr_b16): within each 16-lane group, source lane i points
  //  at V[kb + i/4][db + 4*(i%4) .. +3] so that lane i receives
  //  V[kb + 0..3][db + i]; rows 16*mm + 8*h + tr_key, d = 32*dt + tr_d.
  const int grp = lane >> 4, gi = lane & 15;
  const int tr_key = 4 * (grp >> 1) + (gi >> 2);
  const int tr_byte = 32 * (grp & 1) + 8 * (gi & 3);
  const int v_off0 = tr_key * 64 + 16 * ((tr_byte >> 4) ^ plane_swz(tr_key)) + (tr_byte & 15);
  const int v_off1 = (8 + tr_key) * 64 + 16 * ((tr_byte >> 4) ^ plane_swz(8 + tr_key)) +
                     (tr_byte & 15);

  __syncthreads();  // the tile list is visible
  const int T = ntiles_sh;
  const int T_full = nfull_sh;
  auto tile_key0 = [&](int t) {
    return __builtin_amdgcn_readfirstlane(static_cast<int>(tiles[t]) * kTile);
  };
  // Source offsets of tile t's copy; rows past L (tail tile only) repeat
  // row L-1, whose values the -inf mask discards.
  auto prep = [&](const char* src, int t, uint32_t* off) {
    const int key0 = tile_key0(t);
    const int limit = min(kTile - 1, L - 1 - key0);
#pragma unroll
    for (int i = 0; i < NI; ++i)
      off[i] = static_cast<uint32_t>(min(dma_row[i], limit) * (D * 2)) + dma_col[i];
    return src + static_cast<size_t>(key0) * D * 2;
  };
  auto dma = [&](const char* base, const uint32_t* off, uint16_t* lds, int i) {
    const uint32_t lds_base = (uint32_t)(size_t)(lds_void_t*)lds;  // LDS byte address
    lds_dma16(base, off[i], __builtin_amdgcn_readfirstlane(lds_base + (wave_u + NW * i) * 1024));
  };
  auto issue = [&](const char* src, int t, uint16_t* lds) {
    uint32_t off[NI];
    const char* base = prep(src, t, off);
#pragma unroll
    for (int i = 0; i < NI; ++i) dma(base, off, lds, i);
  };
  // S^T of one tile: rows 0..31 in s0, 32..63 in s1.
  // The NI copy instructions of the next K tile are spread over the k-steps
  // (one every NW/2 steps) so that no wave stalls on a full memory queue in
  // front of its matrix instructions.
  auto qk = [&](auto with_copy, const uint16_t* Kt, f32x16& s0, f32x16& s1,
                const char* dbase, const uint32_t* doff, uint16_t* dlds) {
    const char* Kb = reinterpret_cast<const char*>(Kt);
    s0 = zero16();
    s1 = zero16();
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      const int off = (kc & 1) ? k_off1 : k_off0;
      const u32x4 a0 = *reinterpret_cast<const u32x4*>(Kb + (kc >> 1) * 4096 + off);
      const u32x4 a1 = *reinterpret_cast<const u32x4*>(Kb + (kc >> 1) * 4096 + 2048 + off);
      s0 = mfma32x32x16(a0, qf[kc], s0);
      s1 = mfma32x32x16(a1, qf[kc], s1);
      if constexpr (decltype(with_copy)::value) {
        if (kc % (KC / NI) == KC / NI - 1) dma(dbase, doff, dlds, kc / (KC / NI));
      }
    }
  };
  // Lane-local row max over the 64 keys of a tile.  Rows past L were copied
  // from row L-1 of the same tile, so they repeat a valid logit and leave
  // the max unchanged; their probabilities are zeroed when P is formed.
  auto tile_max = [&](const f32x16& s0, const f32x16& s1) {
    float mx = s0[0];
#pragma unroll
    for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s0[i]);
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s1[i]);
    return mx;
  };

  f32x16 acc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) acc[dt] = zero16();
  float m = -INFINITY;
  float lsum = 0.f;
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};

  // Pipeline: K runs one tile ahead of V.  On entry to iteration t, K(t+1)
  // and V(t) are in LDS and S(t) is in registers.
  f32x16 sc0 = zero16(), sc1 = zero16(), sn_0, sn_1;
  float mx_cur = -INFINITY;
  if (T > 0) {
    issue(kh, 0, Ks[0]);
    issue(vh, 0, Vs[0]);
  }
  if (T > 1) issue(kh, 1, Ks[1]);
  wait_dma();
  __syncthreads();
  if (T > 0) {
    qk(CopyFlag<false>{}, Ks[0], sc0, sc1, nullptr, nullptr, nullptr);
    mx_cur = tile_max(sc0, sc1);
  }
  __syncthreads();  // every wave has read K(0) before iteration 0 refills its buffer
  // One iteration: the copies of K(t+2) and V(t+1) run under S(t+1) = QK^T
  // on the matrix cores, P(t) on the VALUs, and PV(t).  Past the end of the
  // list the last tile is copied again into the free buffer, which keeps the
  // iteration free of branches around the copies.  `tail` marks iterations
  // whose tile t reaches past L: only they zero P for rows past L.
  auto iteration = [&](int t, auto tail) {
    uint32_t koff[NI], voff[NI];
    const char* kbase = prep(kh, min(t + 2, T - 1), koff);
    const char* vbase = prep(vh, min(t + 1, T - 1), voff);
    const float mx = max_halves(mx_cur) * c;
    if (__any(mx > m + kRescaleSlack)) {
      const float m_new = fmaxf(m, mx);
      const float alpha = fast_exp2(m - m_new);
      m = m_new;
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[dt][i] *= alpha;
    }
    // S(t+1) on the matrix cores (computed on stale data in the last
    // iteration and discarded) while the VALUs form P(t).
    f32x16 sn0, sn1;
    qk(CopyFlag<true>{}, Ks[(t + 1) & 1], sn0, sn1, kbase, koff, Ks[t & 1]);
    uint32_t pb0[8], pb1[8];
    if constexpr (decltype(tail)::value) {
      const int kv = L - tile_key0(t);  // valid rows of this tile
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float p0 = crow(2 * i, g) < kv ? fast_exp2(fmaf(sc0[2 * i], c, -m)) : 0.f;
        const float p1 = crow(2 * i + 1, g) < kv ? fast_exp2(fmaf(sc0[2 * i + 1], c, -m)) : 0.f;
        const float p2 = 32 + crow(2 * i, g) < kv ? fast_exp2(fmaf(sc1[2 * i], c, -m)) : 0.f;
        const float p3 =
            32 + crow(2 * i + 1, g) < kv ? fast_exp2(fmaf(sc1[2 * i + 1], c, -m)) : 0.f;
        pb0[i] = pack_bf16x2(p0, p1);
        pb1[i] = pack_bf16x2(p2, p3);
        if constexpr (GATHER) lsum += (p0 + p1) + (p2 + p3);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float p0 = fast_exp2(fmaf(sc0[2 * i], c, -m));
        const float p1 = fast_exp2(fmaf(sc0[2 * i + 1], c, -m));
        const float p2 = fast_exp2(fmaf(sc1[2 * i], c, -m));
        const float p3 = fast_exp2(fmaf(sc1[2 * i + 1], c, -m));
        pb0[i] = pack_bf16x2(p0, p1);
        pb1[i] = pack_bf16x2(p2, p3);
        if constexpr (GATHER) lsum += (p0 + p1) + (p2 + p3);
      }
    }
    // row sum: of the bf16 probabilities that the PV product uses, or (GATHER)
    // of the fp32 probabilities, so that lse is exact to fp32 rounding
    if constexpr (!GATHER) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pb0[i]), ones,
                                               lsum, false);
        lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pb1[i]), ones,
                                               lsum, false);
      }
    }
    // O^T += V(t)^T P(t)^T while the row max of S(t+1) is taken.
    const lds_u16_t* Vb = (const lds_u16_t*)Vs[t & 1];
#pragma unroll
    for (int mm = 0; mm < 4; ++mm) {
      const uint32_t* pb = (mm < 2) ? pb0 : pb1;
      const int h = (mm & 1) * 4;
      const u32x4 b = {pb[h], pb[h + 1], pb[h + 2], pb[h + 3]};
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const lds_u16_t* base = Vb + (dt * 4096 + mm * 1024) / 2;
        const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4_t*)(base + v_off0 / 2)));
        const u32x2 hi = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4_t*)(base + v_off1 / 2)));
        const u32x4 a = {lo.x, lo.y, hi.x, hi.y};
        acc[dt] = mfma32x32x16(a, b, acc[dt]);
        const int j = mm * DT + dt;
        if (j % NW == NW - 1) dma(vbase, voff, Vs[(t + 1) & 1], j / NW);
      }
    }
    // max of S(t+1); in the last iteration it is not used
    mx_cur = tile_max(sn0, sn1);
    sc0 = sn0;
    sc1 = sn1;
    wait_dma();
    __syncthreads();
  };
  // Steady-state iteration: tiles t, t+1 and t+2 hold 64 keys each, with the
  // copy indices t+1 and t+2 clamped to the last tile (a list without a tail
  // tile runs every iteration here; past its end the last tile is copied
  // again into the free buffer, and S(t+1) of the last iteration is
  // discarded).  The issue order is fixed by scheduling barriers so that
  // every MFMA is followed by a share of the VALU work: in the QK^T phase
  // (S(t+1) into n0/n1) one bf16 pair of P(t) per MFMA; in the PV phase the
  // row sums of P(t), then the row max of S(t+1).  Operand reads run two
  // MFMAs ahead, and the NI copies of each matrix are spread over its phase.
  uint32_t dma_full[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) dma_full[i] = static_cast<uint32_t>(dma_row[i] * (D * 2)) + dma_col[i];
  auto main_iter = [&](int t, f32x16& c0, f32x16& c1, f32x16& n0, f32x16& n1) {
    const char* kbase = kh + static_cast<size_t>(tile_key0(min(t + 2, T - 1))) * D * 2;
    const char* vbase = vh + static_cast<size_t>(tile_key0(min(t + 1, T - 1))) * D * 2;
    const float mx = max_halves(mx_cur) * c;
    if (__any(mx > m + kRescaleSlack)) {
      const float m_new = fmaxf(m, mx);
      const float alpha = fast_exp2(m - m_new);
      m = m_new;
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[dt][i] *= alpha;
    }
    const char* Kb = reinterpret_cast<const char*>(Ks[(t + 1) & 1]);
    const lds_u16_t* Vb = (const lds_u16_t*)Vs[t & 1];
    uint16_t* kdst = Ks[t & 1];
    uint16_t* vdst = Vs[(t + 1) & 1];
    auto kread = [&](int kc, u32x4* dst) {
      const int off = (kc & 1) ? k_off1 : k_off0;
      dst[0] = *reinterpret_cast<const u32x4*>(Kb + (kc >> 1) * 4096 + off);
      dst[1] = *reinterpret_cast<const u32x4*>(Kb + (kc >> 1) * 4096 + 2048 + off);
    };
    auto vread = [&](int j, u32x4& dst) {
      const lds_u16_t* base = Vb + ((j % DT) * 4096 + (j / DT) * 1024) / 2;
      const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_s16x4_t*)(base + v_off0 / 2)));
      const u32x2 hi = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_s16x4_t*)(base + v_off1 / 2)));
      dst = u32x4{lo.x, lo.y, hi.x, hi.y};
    };
    // ---- QK^T phase: S(t+1) on the matrix cores, P(t) on the VALUs.  The
    // wave issues at raised priority here, where most of its VALU work lies,
    // and at normal priority in the PV phase.
    __builtin_amdgcn_s_setprio(1);
    constexpr int NA = 2 * KC;          // MFMAs
    constexpr int PPA = 16 / NA;        // bf16 pairs of P per MFMA
    u32x4 ka[3][2];
    uint32_t pb[16];
    kread(0, ka[0]);
    kread(1, ka[1]);
    n0 = zero16();
    n1 = zero16();
    // P(t) is formed in three stages a step apart, so that no instruction
    // waits on the one just before it: in step st the FMAs of pair group
    // st+1, the exponentials of group st, and the bf16 packing of group st-1
    // (a group is the PPA pairs of one step; pair pk holds elements 2pk and
    // 2pk+1 of S(t), from c0 for pk < 8, else from c1).
    float fx[2][PPA][2], ex[2][PPA][2];
    auto stage_fma = [&](int grp) {
#pragma unroll
      for (int u = 0; u < PPA; ++u) {
        const int pk = grp * PPA + u;
        const f32x16& src = pk < 8 ? c0 : c1;
        const int e = 2 * (pk & 7);
        fx[grp & 1][u][0] = fmaf(src[e], c, -m);
        fx[grp & 1][u][1] = fmaf(src[e + 1], c, -m);
      }
    };
    auto stage_exp = [&](int grp) {
#pragma unroll
      for (int u = 0; u < PPA; ++u) {
        ex[grp & 1][u][0] = fast_exp2(fx[grp & 1][u][0]);
        ex[grp & 1][u][1] = fast_exp2(fx[grp & 1][u][1]);
        if constexpr (GATHER) lsum += ex[grp & 1][u][0] + ex[grp & 1][u][1];  // fp32 row sum
      }
    };
    auto stage_pack = [&](int grp) {
#pragma unroll
      for (int u = 0; u < PPA; ++u)
        pb[grp * PPA + u] = pack_bf16x2(ex[grp & 1][u][0], ex[grp & 1][u][1]);
    };
    stage_fma(0);
#pragma unroll
    for (int st = 0; st < NA; ++st) {
      const int kc = st >> 1;
      if ((st & 1) == 0 && kc + 2 < KC) kread(kc + 2, ka[(kc + 2) % 3]);
      if (st & 1)
        n1 = mfma32x32x16(ka[kc % 3][1], qf[kc], n1);
      else
        n0 = mfma32x32x16(ka[kc % 3][0], qf[kc], n0);
      if (st > 0) stage_pack(st - 1);
      stage_exp(st);
      if (st + 1 < NA) stage_fma(st + 1);
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        if (i * NA / NI == st) {
          const uint32_t la = (uint32_t)(size_t)(lds_void_t*)kdst;
          lds_dma16(kbase, dma_full[i],
                    __builtin_amdgcn_readfirstlane(la + (wave_u + NW * i) * 1024));
        }
        if (i * NA / NI + NA / (2 * NI) == st) {
          const uint32_t la = (uint32_t)(size_t)(lds_void_t*)vdst;
          lds_dma16(vbase, dma_full[i],
                    __builtin_amdgcn_readfirstlane(la + (wave_u + NW * i) * 1024));
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    stage_pack(NA - 1);
    // ---- PV phase: O^T += V(t)^T P(t)^T; row sums of P(t), row max of S(t+1)
    __builtin_amdgcn_s_setprio(0);
    constexpr int NB = 4 * DT;          // MFMAs
    constexpr int VB = 32 / NB;         // VALU ops per MFMA
    u32x4 va[3];
    vread(0, va[0]);
    vread(1, va[1]);
    float mxn = -INFINITY;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (j + 2 < NB) vread(j + 2, va[(j + 2) % 3]);
      const int mm = j / DT, dt = j % DT;
      const int h = (mm & 1) * 4 + (mm < 2 ? 0 : 8);
      const u32x4 b = {pb[h], pb[h + 1], pb[h + 2], pb[h + 3]};
      acc[dt] = mfma32x32x16(va[j % 3], b, acc[dt]);
#pragma unroll
      for (int u = 0; u < VB; ++u) {
        const int w = j * VB + u;  // 0..15: row sums, 16..31: max pairs
        if (w < 16) {
          if constexpr (!GATHER)
            lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pb[w]), ones,
                                                   lsum, false);
        } else {
          const int e = w - 16;  // pair e: elements 2e, 2e+1 of n0 (e < 8) or n1
          const f32x16& src = e < 8 ? n0 : n1;
          mxn = fmaxf(mxn, src[2 * (e & 7)]);
          mxn = fmaxf(mxn, src[2 * (e & 7) + 1]);
          asm volatile("" : "+v"(mxn));  // keeps this share of the max in its slot
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    mx_cur = mxn;
    __builtin_amdgcn_s_setprio(0);
    wait_dma();
    __syncthreads();
  };

  // With a tail tile (T_full < T), its copies (row clamp) and its masked P
  // take the generic iterations, from the one that first copies it.
  const int T_main = T_full == T ? T : (T_full > 2 ? T_full - 2 : 0);
  int t = 0;
  for (; t + 1 < T_main; t += 2) {
    main_iter(t, sc0, sc1, sn_0, sn_1);
    main_iter(t + 1, sn_0, sn_1, sc0, sc1);
  }
  if (t < T_main) {
    main_iter(t, sc0, sc1, sn_0, sn_1);
    sc0 = sn_0;
    sc1 = sn_1;
    ++t;
  }
  for (; t < T; ++t) iteration(t, CopyFlag<true>{});

  const float ltot = lsum + swap_halves(lsum);
  if constexpr (GATHER) {
    if (part != nullptr) {
      if (qvalid) {
        const size_t prow = static_cast<size_t>(split * P + pair) * n_rows +
                            (r * BLOCK + (tid >> 6) * 32 + n);
        float* orow = part + prow * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int rg = 0; rg < 4; ++rg) {
            const f32x4 val = {acc[dt][4 * rg], acc[dt][4 * rg + 1], acc[dt][4 * rg + 2],
                               acc[dt][4 * rg + 3]};
            *reinterpret_cast<f32x4*>(orow + 32 * dt + 8 * rg + 4 * g) = val;
          }
        if (g == 0) {
          float2* ml = reinterpret_cast<float2*>(
              part + static_cast<size_t>(n_split) * P * n_rows * D);
          ml[prow] = make_float2(m, ltot);
        }
      }
      return;
    }
  }
  const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
  if (qvalid) {
    uint16_t* orow = o + (static_cast<size_t>(pair) * LQ + qrow) * D;
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
      lse[static_cast<size_t>(pair) * LQ + qrow] =
          ltot > 0.f ? (m + __log2f(ltot)) * kLn2 : -INFINITY;
  }
  }  // next row
}

// Merges the n_split partial rows of each gathered query (rows[b*n_rows + j],
// or j when rows is NULL; Lq output rows per pair): with M the largest
// running max, O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s and
// lse = (M + log2 of the denominator) ln 2, the splits added in index order.
// One thread per 4 channels of a row.
template <int D>
__global__ void __launch_bounds__(256)
token_combine_kernel(const float* __restrict__ part, int n_split, int P, int Lq, int H,
                     const int32_t* __restrict__ rows, int n_rows, uint16_t* __restrict__ o,
                     float* __restrict__ lse) {
  constexpr int TPR = D / 4;
  const size_t gid = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  const size_t pr = gid / TPR;  // pair * n_rows + j
  if (pr >= static_cast<size_t>(P) * n_rows) return;
  const int d4 = static_cast<int>(gid % TPR) * 4;
  const int pair = static_cast<int>(pr / n_rows), j = static_cast<int>(pr % n_rows);
  const int t = rows != nullptr ? rows[static_cast<size_t>(pair / H) * n_rows + j] : j;
  if (t < 0 || t >= Lq) return;
  const size_t stride = static_cast<size_t>(P) * n_rows;  // rows per split
  const float2* ml = reinterpret_cast<const float2*>(part + n_split * stride * D);
  float M = -INFINITY;
  for (int s = 0; s < n_split; ++s) {
    const float2 v = ml[s * stride + pr];
    if (v.y > 0.f) M = fmaxf(M, v.x);
  }
  float den = 0.f;
  f32x4 num = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < n_split; ++s) {
    const float2 v = ml[s * stride + pr];
    const float w = v.y > 0.f ? exp2f(v.x - M) : 0.f;
    const f32x4 x = *reinterpret_cast<const f32x4*>(part + (s * stride + pr) * D + d4);
    den = fmaf(w, v.y, den);
#pragma unroll
    for (int e = 0; e < 4; ++e) num[e] = fmaf(w, x[e], num[e]);
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
  const u32x2 val = {pack_bf16x2(num[0] * inv, num[1] * inv),
                     pack_bf16x2(num[2] * inv, num[3] * inv)};
  *reinterpret_cast<u32x2*>(o + (static_cast<size_t>(pair) * Lq + t) * D + d4) = val;
  if (lse != nullptr && d4 == 0)
    lse[static_cast<size_t>(pair) * Lq + t] = den > 0.f ? (M + __log2f(den)) * kLn2 : -INFINITY;
}

// ---- fp32 path ------------------------------------------------------------
constexpr int kF32Keys = 32;

// GATHER: as in the bf16 kernel, row j of pair (b,h) is token
// rows[b*n_rows + j] and every key block is kept.
template <int D, bool GATHER>
__global__ void __launch_bounds__(128)
sparse_attn_f32_kernel(const float* __restrict__ q, const float* __restrict__ k,
                       const float* __restrict__ v, float* __restrict__ o,
                       float* __restrict__ lse,
                       const int32_t* __restrict__ kv_idx,
                       const int32_t* __restrict__ kv_cnt, int L, int n_b,
                       int block, float scale, const int32_t* __restrict__ rows,
                       int n_rows, int H) {
  __shared__ float Kt[kF32Keys][D + 1];
  __shared__ float Vt[kF32Keys][D];
  const int pair = blockIdx.y;
  const int r = blockIdx.x;
  const size_t row_base = static_cast<size_t>(pair) * n_b + r;
  int cnt = n_b;
  const int32_t* idx = nullptr;
  if constexpr (!GATHER) {
    cnt = kv_cnt[row_base];
    cnt = cnt < 0 ? 0 : (cnt > n_b ? n_b : cnt);
    idx = kv_idx + row_base * n_b;
  }
  const float* qh = q + static_cast<size_t>(pair) * L * D;
  const float* kh = k + static_cast<size_t>(pair) * L * D;
  const float* vh = v + static_cast<size_t>(pair) * L * D;
  const int tid = threadIdx.x;
  int qrow = r * block + tid;
  bool active = tid < block && qrow < L;
  if constexpr (GATHER) {
    active = tid < block && qrow < n_rows;
    qrow = active ? rows[static_cast<size_t>(pair / H) * n_rows + qrow] : -1;
    active = active && qrow >= 0 && qrow < L;
  }

  float qv[D], acc[D];
#pragma unroll
  for (int e = 0; e < D; ++e) {
    qv[e] = active ? qh[static_cast<size_t>(qrow) * D + e] : 0.f;
    acc[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;

  for (int i = 0; i < cnt; ++i) {
    const int kb = GATHER ? i : idx[i];
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
  const AttnWs lay = attn_ws_layout(B, H, n_b, d, block);
  int32_t* order = reinterpret_cast<int32_t*>(ws + lay.order);
  int32_t* sched = reinterpret_cast<int32_t*>(ws + lay.sched);
  int* claim = reinterpret_cast<int*>(ws + lay.claim);
  const float c = scale * kLog2e;
  hipLaunchKernelGGL(order_rows_kernel, dim3(P, ceil_div(n_b, kOrderRows)), dim3(kOrderRows), 0,
                     s, kv_cnt, order, n_b);
  // pair count a multiple of 8: persistent workgroups, as many as the chip
  // holds at once (2 per CU, 32 CUs per XCD) and no more than the rows
  dim3 grid(P * n_b);
  if ((P & 7) == 0) {
    hipLaunchKernelGGL(schedule_rows_kernel, dim3(8), dim3(1024), 0, s, kv_cnt, order, sched,
                       claim, P, n_b);
    grid = dim3(8 * std::min((P >> 3) * n_b, 2 * kCusPerXcd));
  }
  if (d == 128 && block == 128)
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<128, 128, false>), grid, dim3(256), 0, s,
                       q, k, v, o, lse, kv_idx, kv_cnt, order, sched, claim, P, L, n_b, c, nullptr, 0, H, 1,
                       nullptr, L);
  else if (d == 128 && block == 64)
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<128, 64, false>), grid, dim3(128), 0, s,
                       q, k, v, o, lse, kv_idx, kv_cnt, order, sched, claim, P, L, n_b, c, nullptr, 0, H, 1,
                       nullptr, L);
  else if (d == 64 && block == 128)
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<64, 128, false>), grid, dim3(256), 0, s,
                       q, k, v, o, lse, kv_idx, kv_cnt, order, sched, claim, P, L, n_b, c, nullptr, 0, H, 1,
                       nullptr, L);
  else
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<64, 64, false>), grid, dim3(128), 0, s,
                       q, k, v, o, lse, kv_idx, kv_cnt, order, sched, claim, P, L, n_b, c, nullptr, 0, H, 1,
                       nullptr, L);
}

void launch_sparse_attention_f32(const float* q, const float* k,
                                 const float* v, float* o, float* lse, int B,
                                 int H, int L, int d, float scale, int block,
                                 const int32_t* kv_idx, const int32_t* kv_cnt,
                                 char* /*ws*/, hipStream_t s) {
  const int n_b = ceil_div(L, block);
  const dim3 grid(n_b, B * H);
  if (d == 128)
    hipLaunchKernelGGL((sparse_attn_f32_kernel<128, false>), grid, dim3(128), 0, s, q, k, v,
                       o, lse, kv_idx, kv_cnt, L, n_b, block, scale, nullptr, 0, H);
  else
    hipLaunchKernelGGL((sparse_attn_f32_kernel<64, false>), grid, dim3(128), 0, s, q, k, v,
                       o, lse, kv_idx, kv_cnt, L, n_b, block, scale, nullptr, 0, H);
}

// Dense rows gathered from Q ([B,H,Lq,d]; rows[b*n_rows + j], or j when rows
// is NULL) against every key of K/V ([B,H,Lk,d]), in blocks of 128 rows;
// with more than one key split the partials go to ws and
// token_combine_kernel writes O/lse.
void launch_gather_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                  uint16_t* o, float* lse, int B, int H, int Lq, int Lk,
                                  int d, float scale, const int32_t* rows, int n_rows,
                                  char* ws, hipStream_t s) {
  const int n_b = ceil_div(Lk, kTokRowBlock);
  const int P = B * H;
  const float c = scale * kLog2e;
  const int ns = token_attn_splits(P, n_rows, n_b);
  float* part = ns > 1 ? reinterpret_cast<float*>(ws) : nullptr;
  const dim3 grid(P * ceil_div(n_rows, kTokRowBlock) * ns);
  if (d == 128)
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<128, kTokRowBlock, true>), grid, dim3(256), 0,
                       s, q, k, v, o, lse, nullptr, nullptr, nullptr, nullptr, nullptr, P, Lk, n_b, c, rows,
                       n_rows, H, ns, part, Lq);
  else
    hipLaunchKernelGGL((sparse_attn_bf16_kernel<64, kTokRowBlock, true>), grid, dim3(256), 0,
                       s, q, k, v, o, lse, nullptr, nullptr, nullptr, nullptr, nullptr, P, Lk, n_b, c, rows,
                       n_rows, H, ns, part, Lq);
  if (ns > 1) {
    const size_t threads = static_cast<size_t>(P) * n_rows * (d / 4);
    const dim3 cgrid(static_cast<unsigned>((threads + 255) / 256));
    if (d == 128)
      hipLaunchKernelGGL(token_combine_kernel<128>, cgrid, dim3(256), 0, s, part, ns, P, Lq, H,
                         rows, n_rows, o, lse);
    else
      hipLaunchKernelGGL(token_combine_kernel<64>, cgrid, dim3(256), 0, s, part, ns, P, Lq, H,
                         rows, n_rows, o, lse);
  }
}

// Dense rows of the protected tokens (Eq. (11) first case), written over O
// and lse.
void launch_protected_token_attention_bf16(const uint16_t* q, const uint16_t* k,
                                           const uint16_t* v, uint16_t* o, float* lse,
                                           int B, int H, int L, int d, float scale,
                                           const int32_t* tok_idx, int k_tok, char* ws,
                                           hipStream_t s) {
  launch_gather_attention_bf16(q, k, v, o, lse, B, H, L, L, d, scale, tok_idx, k_tok, ws, s);
}

// Cross-modal attention: every query of Q [B,H,Lq,d] against K/V [B,H,Lk,d].
void launch_cross_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                 uint16_t* o, float* lse, int B, int H, int Lq, int Lk, int d,
                                 float scale, char* ws, hipStream_t s) {
  launch_gather_attention_bf16(q, k, v, o, lse, B, H, Lq, Lk, d, scale, nullptr, Lq, ws, s);
}

void launch_protected_token_attention_f32(const float* q, const float* k, const float* v,
                                          float* o, float* lse, int B, int H, int L, int d,
                                          float scale, const int32_t* tok_idx, int k_tok,
                                          hipStream_t s) {
  constexpr int kRowBlock = kTokRowBlock;
  const int n_b = ceil_div(L, kRowBlock);
  const dim3 grid(ceil_div(k_tok, kRowBlock), B * H);
  if (d == 128)
    hipLaunchKernelGGL((sparse_attn_f32_kernel<128, true>), grid, dim3(128), 0, s, q, k, v,
                       o, lse, nullptr, nullptr, L, n_b, kRowBlock, scale, tok_idx, k_tok, H);
  else
    hipLaunchKernelGGL((sparse_attn_f32_kernel<64, true>), grid, dim3(128), 0, s, q, k, v,
                       o, lse, nullptr, nullptr, L, n_b, kRowBlock, scale, tok_idx, k_tok, H);
}

}  // namespace sa
