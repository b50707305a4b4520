// Sustained bf16 MFMA throughput probe (declared in sa_bench.h).
#include <hip/hip_runtime.h>
#include <cstdint>

#include "sa_bench.h"

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlocks = 1024;   // 4 workgroups of 4 waves per CU on 256 CUs
constexpr int kThreads = 256;

template <bool RANDOM>
__global__ void __launch_bounds__(kThreads)
mfma_probe_kernel(int iters, float* __restrict__ sink, unsigned long long* __restrict__ clk) {
  const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
  uint32_t x = 0x9e3779b9u ^ (tid * 2654435761u);
  auto next = [&]() {
    x ^= x << 13;
    x ^= x >> 17;
    x ^= x << 5;
    return x;
  };
  // bf16 0x3f80 | (sign, mantissa bits): magnitudes in [1, 2)
  auto val = [&]() { return RANDOM ? (0x3f80u | (next() & 0x807fu)) : 0u; };
  u32x4 a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      a[i][j] = val() | (val() << 16);
      b[i][j] = val() | (val() << 16);
    }
  f32x16 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x16{};
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, a[(c + s) & 3]),
            __builtin_bit_cast(bf16x8, b[(c + 2 * s) & 3]), acc[c], 0, 0, 0);
    if (RANDOM) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i][it & 3] ^= 0x00550055u;  // mantissa bits only
        b[i][(it + 1) & 3] ^= 0x002a002au;
      }
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 16; ++j) s += acc[i][j];
  sink[tid] = s;
  if (threadIdx.x == 0) {
    clk[2 * blockIdx.x] = t1 - t0;
    clk[2 * blockIdx.x + 1] = r1 - r0;
  }
}

}  // namespace

extern "C" int sa_bench_mfma_peak(int random_operands, int iters, int reps, float* tflops,
                                  float* ghz) {
  if (iters < 1 || reps < 1 || tflops == nullptr || ghz == nullptr) return -1;
  float* sink = nullptr;
  unsigned long long* clk = nullptr;
  if (hipMalloc(&sink, sizeof(float) * kBlocks * kThreads) != hipSuccess) return -1;
  if (hipMalloc(&clk, sizeof(unsigned long long) * 2 * kBlocks) != hipSuccess) {
    (void)hipFree(sink);
    return -1;
  }
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = 0;
  float best = 0.f, best_ghz = 0.f;
  static unsigned long long host[2 * kBlocks];
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) rc = -1;
  for (int r = 0; r < reps && rc == 0; ++r) {
    (void)hipEventRecord(e0, nullptr);
    if (random_operands)
      hipLaunchKernelGGL(mfma_probe_kernel<true>, dim3(kBlocks), dim3(kThreads), 0, nullptr,
                         iters, sink, clk);
    else
      hipLaunchKernelGGL(mfma_probe_kernel<false>, dim3(kBlocks), dim3(kThreads), 0, nullptr,
                         iters, sink, clk);
    if (hipGetLastError() != hipSuccess || hipEventRecord(e1, nullptr) != hipSuccess ||
        hipEventSynchronize(e1) != hipSuccess) {
      rc = -1;
      break;
    }
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess ||
        hipMemcpy(host, clk, sizeof(host), hipMemcpyDeviceToHost) != hipSuccess) {
      rc = -1;
      break;
    }
    double c = 0.0, t = 0.0;
    for (int i = 0; i < kBlocks; ++i) {
      c += static_cast<double>(host[2 * i]);
      t += static_cast<double>(host[2 * i + 1]);
    }
    const double flops = static_cast<double>(kBlocks) * 4.0 * iters * 16.0 * 32768.0;
    const float tf = static_cast<float>(flops / (ms * 1e-3) / 1e12);
    if (tf > best) {
      best = tf;
      best_ghz = t > 0.0 ? static_cast<float>(c / t * 0.1) : 0.f;  // realtime is 100 MHz
    }
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipFree(sink);
  (void)hipFree(clk);
  *tflops = best;
  *ghz = best_ghz;
  return rc;
}
