// Synchronization-aware cache-reuse indicator (Sec. 4.3, Eq. (12)-(15)).
//
// K10 cache_partial: one pass over the block outputs.  Workgroups
//     [0, wg_v) share the video rows (B*L_v rows of C channels) and the
//     matching entries of the two saliency maps, [wg_v, wg_v + wg_a) the
//     audio rows.  Each thread adds |Y - Y_hat| and |Y| (and the same on rows of
//     protected tokens) in fp32 over its 16-byte chunks; the workgroup sums
//     are formed in a fixed order and written as 9 partials per
//     workgroup ([9][workgroups]): video diff/mag, protected diff/mag, audio
//     diff/mag, <s_bar, s_hat>, ||s_bar||^2, ||s_hat||^2.
// K11 cache_finish: one workgroup (a wave per partial) adds the partials in
//     fp64 in a fixed order and writes {dv, da, dp, ds, sync, reuse}
//     (Eq. (12)-(15)).
#include "sa_device.h"
#include "sa_internal.h"

namespace sa {
namespace {

constexpr int kCacheThreads = 256;
constexpr int kCacheParts = 9;

template <typename T> struct Chunk;
template <> struct Chunk<uint16_t> {
  static constexpr int kElems = 8;
  __device__ static void unpack(u32x4 v, float* out) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out[2 * i] = __uint_as_float(v[i] << 16);
      out[2 * i + 1] = __uint_as_float(v[i] & 0xffff0000u);
    }
  }
};
template <> struct Chunk<float> {
  static constexpr int kElems = 4;
  __device__ static void unpack(u32x4 v, float* out) {
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = __uint_as_float(v[i]);
  }
};

// Workgroup sums of the kCacheParts values of every thread (wave shuffles,
// then the 4 wave sums in wave order); valid in thread 0.
template <typename A>
__device__ __forceinline__ void block_sums(A (&acc)[kCacheParts], A (*red)[kCacheParts]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < kCacheParts; ++j) {
    A v = acc[j];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) red[wave][j] = v;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int j = 0; j < kCacheParts; ++j) {
      A v = red[0][j];
      for (int w = 1; w < kCacheThreads / 64; ++w) v += red[w][j];
      acc[j] = v;
    }
  }
}

// |y - y_hat| and |y| over rows [r0, r1) of [rows][C] (C a multiple of the
// chunk width); rows with flag[row] != 0 also count into the second pair.
// The rows are one contiguous span of 16-byte chunks, dealt out to the
// threads in steps of U chunks each (2*U loads in flight per thread); the
// host keeps (r1 - r0) * C / chunk below 2^32.
template <typename T>
__device__ __forceinline__ void rows_l1(const T* y, const T* yh, const uint8_t* flag,
                                        size_t r0, size_t r1, int C, float* acc) {
  constexpr int EPC = Chunk<T>::kElems;
  constexpr int U = 8;
  const uint32_t cpr = static_cast<uint32_t>(C / EPC);
  const uint32_t n = static_cast<uint32_t>((r1 - r0) * cpr);
  const T* ya = y + r0 * C;
  const T* yb = yh + r0 * C;
  for (uint32_t j0 = threadIdx.x; j0 < n; j0 += U * kCacheThreads) {
    u32x4 va[U], vb[U];
    bool pr[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t j = j0 + u * kCacheThreads;
      const bool ok = j < n;
      va[u] = ok ? ldg16_nt(ya + static_cast<size_t>(j) * EPC) : u32x4{0u, 0u, 0u, 0u};
      vb[u] = ok ? ldg16_nt(yb + static_cast<size_t>(j) * EPC) : u32x4{0u, 0u, 0u, 0u};
      pr[u] = flag != nullptr && ok && flag[r0 + j / cpr] != 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float a[EPC], b[EPC];
      Chunk<T>::unpack(va[u], a);
      Chunk<T>::unpack(vb[u], b);
      float d = 0.f, m = 0.f;
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        d += fabsf(a[e] - b[e]);
        m += fabsf(a[e]);
      }
      acc[0] += d;
      acc[1] += m;
      if (pr[u]) {
        acc[2] += d;
        acc[3] += m;
      }
    }
  }
}

// Video workgroup wg owns rows [r0, r1) of the B*L_v video rows and the same
// entries of the two [B, L_v] saliency maps; audio workgroups own audio rows.
template <typename T>
__global__ void __launch_bounds__(kCacheThreads)
cache_partial_kernel(const T* __restrict__ yv, const T* __restrict__ yvh,
                     const uint8_t* __restrict__ pflag, size_t rows_v, int C,
                     const T* __restrict__ ya, const T* __restrict__ yah, size_t rows_a,
                     const float* __restrict__ sb, const float* __restrict__ sh, int wg_v,
                     int wg_a, float* __restrict__ part) {
  __shared__ float red[kCacheThreads / 64][kCacheParts];
  const int wg = blockIdx.x;
  float acc[kCacheParts];
#pragma unroll
  for (int j = 0; j < kCacheParts; ++j) acc[j] = 0.f;
  if (wg < wg_v) {
    const size_t r0 = rows_v * wg / wg_v, r1 = rows_v * (wg + 1) / wg_v;
    if (sb != nullptr) {
      for (size_t i = r0 + threadIdx.x; i < r1; i += kCacheThreads) {
        const float x = sb[i], z = sh[i];
        acc[6] = fmaf(x, z, acc[6]);
        acc[7] = fmaf(x, x, acc[7]);
        acc[8] = fmaf(z, z, acc[8]);
      }
    }
    rows_l1(yv, yvh, pflag, r0, r1, C, acc);
  } else {
    const int a = wg - wg_v;
    const size_t r0 = rows_a * a / wg_a, r1 = rows_a * (a + 1) / wg_a;
    float tmp[4] = {0.f, 0.f, 0.f, 0.f};
    rows_l1<T>(ya, yah, nullptr, r0, r1, C, tmp);
    acc[4] = tmp[0];
    acc[5] = tmp[1];
  }
  block_sums(acc, red);
  if (threadIdx.x == 0) {
#pragma unroll
    for (int j = 0; j < kCacheParts; ++j) part[static_cast<size_t>(j) * gridDim.x + wg] = acc[j];
  }
}

// One wave per partial sum: lane l adds workgroups l, l+64, ... in order in
// fp64, the lanes are summed by shuffles, wave 0 forms the outputs.
constexpr int kFinishThreads = kCacheParts * 64;

__global__ void __launch_bounds__(kFinishThreads)
cache_finish_kernel(const float* __restrict__ part, int nwg, int has_prot, int has_audio,
                    int has_sal, float lambda_p, float lambda_s, float tau, float eps,
                    float* __restrict__ out) {
  __shared__ double tot[kCacheParts];
  const int lane = threadIdx.x & 63, j = threadIdx.x >> 6;
  const float* p = part + static_cast<size_t>(j) * nwg;
  double s = 0.0;
  for (int w0 = lane; w0 < nwg; w0 += 8 * 64) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = w0 + 64 * u < nwg ? p[w0 + 64 * u] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) s += static_cast<double>(v[u]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) tot[j] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double e = eps;
    const double dv = tot[0] / (tot[1] + e);
    const double dp = has_prot ? tot[2] / (tot[3] + e) : 0.0;
    const double da = has_audio ? tot[4] / (tot[5] + e) : 0.0;
    const double ds = has_sal ? 1.0 - tot[6] / (sqrt(tot[7]) * sqrt(tot[8]) + e) : 0.0;
    const double sync = fmax(fmax(dv, da), fmax(lambda_p * dp, lambda_s * ds));
    const float sync_f = static_cast<float>(sync);
    out[0] = static_cast<float>(dv);
    out[1] = static_cast<float>(da);
    out[2] = static_cast<float>(dp);
    out[3] = static_cast<float>(ds);
    out[4] = sync_f;
    out[5] = sync_f < tau ? 1.f : 0.f;  // decided on the reported fp32 value
  }
}

}  // namespace

void launch_cache_indicator(const void* y_v, const void* y_v_hat, const uint8_t* prot_flag,
                            const void* y_a, const void* y_a_hat, const float* s_bar,
                            const float* s_hat, int B, int L_v, int L_a, int C, int dtype,
                            float lambda_p, float lambda_s, float tau, float eps,
                            float* out, char* ws, hipStream_t s) {
  const size_t rows_v = static_cast<size_t>(B) * L_v;
  const size_t rows_a = y_a != nullptr ? static_cast<size_t>(B) * L_a : 0;
  const int wg_v = cache_workgroups_video(rows_v);
  const int wg_a = cache_workgroups_audio(rows_a);
  const int nwg = wg_v + wg_a;
  float* part = reinterpret_cast<float*>(ws);
  if (dtype == 0)
    hipLaunchKernelGGL(cache_partial_kernel<uint16_t>, dim3(nwg), dim3(kCacheThreads), 0, s,
                       static_cast<const uint16_t*>(y_v), static_cast<const uint16_t*>(y_v_hat),
                       prot_flag, rows_v, C, static_cast<const uint16_t*>(y_a),
                       static_cast<const uint16_t*>(y_a_hat), rows_a, s_bar, s_hat, wg_v,
                       wg_a, part);
  else
    hipLaunchKernelGGL(cache_partial_kernel<float>, dim3(nwg), dim3(kCacheThreads), 0, s,
                       static_cast<const float*>(y_v), static_cast<const float*>(y_v_hat),
                       prot_flag, rows_v, C, static_cast<const float*>(y_a),
                       static_cast<const float*>(y_a_hat), rows_a, s_bar, s_hat, wg_v,
                       wg_a, part);
  hipLaunchKernelGGL(cache_finish_kernel, dim3(1), dim3(kFinishThreads), 0, s, part, nwg,
                     prot_flag != nullptr, y_a != nullptr, s_bar != nullptr, lambda_p,
                     lambda_s, tau, eps, out);
}

}  // namespace sa
