// Device helpers shared by the gfx950 kernels of libsa.so.
//
// MFMA operand layout used throughout (v_mfma_f32_32x32x16_bf16, wave64):
//   A operand (32 x 16): lane l holds row (l % 32), 8 consecutive k values
//                        starting at 8 * (l / 32);
//   B operand (16 x 32): lane l holds column (l % 32), the same 8 k values;
//   C/D (32 x 32, 16 floats per lane): element r of lane l sits at
//       row crow(r, l / 32) = 8 * (r / 4) + 4 * (l / 32) + r % 4,
//       column l % 32.
// A and B are always filled symmetrically (the same k index for the same
// lane half and element), so a contraction is correct whatever order the
// hardware gives the k values inside a lane.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

__device__ __forceinline__ constexpr int crow(int r, int g) {
  return 8 * (r >> 2) + 4 * g + (r & 3);
}

__device__ __forceinline__ f32x16 mfma32x32x16(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(
      __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// bf16 <-> f32.  The conversion to bf16 rounds to nearest even.
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Value held by the lane 32 positions away (the other half of the wave).
__device__ __forceinline__ float swap_halves(float x) {
  return __shfl_xor(x, 32, 64);
}

__device__ __forceinline__ float fast_exp2(float x) {
  return __builtin_amdgcn_exp2f(x);
}

typedef __attribute__((address_space(3))) void lds_void_t;

// LDS tile layout: D/32 "planes" of [64 keys][32 d] bf16 (64 bytes per key
// row, 4 KB per plane); 16-byte slot s of row r is stored at slot
// s ^ plane_swz(r).  With this swizzle both the K operand reads
// (ds_read_b128: 16 consecutive rows, one slot) and the transposing V reads
// (ds_read_b64_tr_b16: 4 consecutive rows, two slots) are free of bank
// conflicts, and every read address is a lane constant plus an immediate.
__device__ __forceinline__ constexpr int plane_swz(int r) {
  return ((r >> 2) & 1) | ((((r >> 1) ^ (r >> 3)) & 1) << 1);
}

// Copy of 16 bytes per lane, global -> LDS (global_load_lds_dwordx4): lane l
// writes LDS bytes [lds_addr + 16*l, +16) with the 16 bytes at sbase + voff.
// A 64-key tile of a [L][D] bf16 matrix is 4*D such chunks, i.e. 4*D/64 spans
// of 1 KB; chunk i of the tile is LDS byte 16*i = plane i/256, row (i%256)/4,
// physical slot i%4, holding logical slot (i%4) ^ plane_swz(row).
//
// The copy is issued with inline assembly on purpose: the compiler cannot
// tell that an in-flight copy into one buffer does not alias the operand
// reads of the other, and would otherwise wait for every copy (vmcnt(0))
// before the first LDS read that follows it, serialising the pipeline.  The
// kernel orders the buffers itself: s_waitcnt vmcnt(0) and a barrier end
// every iteration, before any copied tile is read or a buffer is refilled.
__device__ __forceinline__ void lds_dma16(const char* sbase, uint32_t voff, uint32_t lds_addr) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1"
      :
      : "v"(voff), "s"(sbase), "s"(lds_addr)
      : "memory", "m0");
}

__device__ __forceinline__ void wait_dma() {
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
}
// Wait until at most n (< 16) vector-memory operations of this wave are
// outstanding; they complete in issue order.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

__device__ __forceinline__ u32x4 ldg16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
// The same load with the nontemporal cache policy (`nt`), for data that a
// pass reads exactly once.  On gfx950 the block pooling's reads of Q^v and
// K^v ran at about 6.1 TB/s with it against 5.0-5.4 TB/s without (same
// kernel and box).
__device__ __forceinline__ u32x4 ldg16_nt(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void stg16(void* p, u32x4 v) {
  *reinterpret_cast<u32x4*>(p) = v;
}

// Monotone map of a float to an unsigned integer (larger float -> larger
// integer); -0.0 is folded into +0.0 so equal values compare equal.
__device__ __forceinline__ uint32_t float_order_key(float v) {
  uint32_t u = __float_as_uint(v);
  if ((u & 0x7fffffffu) == 0u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Sort key for "value descending, index ascending" as one ascending u64.
__device__ __forceinline__ uint64_t desc_value_asc_index_key(float v,
                                                            uint32_t idx) {
  return (static_cast<uint64_t>(~float_order_key(v)) << 32) | idx;
}

// Sort key for "value descending, index ascending" from a double: the low 12
// bits of the order-preserving image are replaced by the index (idx < 4096),
// so values within 2^-40 relative of each other rank as ties (lower index
// first).
__device__ __forceinline__ uint64_t desc_double_asc_index_key(double v,
                                                             uint32_t idx) {
  uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
  if ((u & 0x7fffffffffffffffull) == 0ull) u = 0ull;
  const uint64_t ord = (u >> 63) ? ~u : (u | 0x8000000000000000ull);
  return (~ord & ~0xfffull) | idx;
}

// In-place ascending bitonic sort of n (a power of two) keys in LDS by the
// whole workgroup.  Ends with a barrier.
__device__ __forceinline__ void bitonic_sort_lds(uint64_t* keys, int n) {
  const int tid = threadIdx.x;
  const int nt = blockDim.x;
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      for (int t = tid; t < (n >> 1); t += nt) {
        const int lo = 2 * t - (t & (stride - 1));
        const int hi = lo + stride;
        const bool up = (lo & size) == 0;
        const uint64_t a = keys[lo];
        const uint64_t b = keys[hi];
        if ((a > b) == up) {
          keys[lo] = b;
          keys[hi] = a;
        }
      }
    }
  }
  __syncthreads();
}

__host__ __device__ constexpr int ceil_div(int a, int b) {
  return (a + b - 1) / b;
}

__host__ __device__ constexpr size_t align_to_8(size_t x) {
  return (x + 7) & ~static_cast<size_t>(7);
}

__host__ __device__ constexpr int next_pow2(int n) {
  int p = 1;
  while (p < n) p <<= 1;
  return p;
}

}  // namespace sa
