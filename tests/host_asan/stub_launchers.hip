// Stand-ins for the kernel launchers of libsa.so, for the host-only build of
// the C ABI that runs under AddressSanitizer and UndefinedBehaviorSanitizer.
// Each records that it was reached instead of enqueuing kernels, so the
// checks can tell that a rejected call launched nothing.
#include "../../paper_2608_15522_amd/csrc/sa_device.h"
#include "../../paper_2608_15522_amd/csrc/sa_internal.h"

extern "C" int sa_host_stub_launches = 0;

namespace sa {

#define SA_STUB(...) { (void)sizeof(#__VA_ARGS__); ++sa_host_stub_launches; }

void launch_cache_indicator(const void*, const void*, const uint8_t*, const void*, const void*,
                            const float*, const float*, int, int, int, int, int, float, float,
                            float, float, float*, char*, hipStream_t) SA_STUB()
void launch_saliency_ema(float*, const float*, size_t, float, hipStream_t) SA_STUB()
void launch_select_protected_tokens(const float*, int, int, int, int32_t*, uint8_t*,
                                    hipStream_t) SA_STUB()
void launch_protected_token_attention_bf16(const uint16_t*, const uint16_t*, const uint16_t*,
                                           uint16_t*, float*, int, int, int, int, float,
                                           const int32_t*, int, char*, hipStream_t) SA_STUB()
void launch_cross_attention_bf16(const uint16_t*, const uint16_t*, const uint16_t*, uint16_t*,
                                 float*, int, int, int, int, int, float, char*,
                                 hipStream_t) SA_STUB()
void launch_protected_token_attention_f32(const float*, const float*, const float*, float*,
                                          float*, int, int, int, int, float, const int32_t*,
                                          int, hipStream_t) SA_STUB()
void launch_cross_scores_bf16(const uint16_t*, const uint16_t*, const uint16_t*,
                              const uint16_t*, int, int, int, int, int, float, int, float*,
                              float*, float*, int, double*, double*, char*, hipStream_t) SA_STUB()
void launch_cross_scores_from_lse_bf16(const uint16_t*, const uint16_t*, const uint16_t*,
                                       const uint16_t*, const float*, const float*, int, int,
                                       int, int, int, float, int, float*, float*, float*, int,
                                       double*, double*, char*, hipStream_t) SA_STUB()
void launch_cross_scores_f32(const float*, const float*, const float*, const float*, int, int,
                             int, int, int, float, int, float*, float*, float*, int, char*,
                             hipStream_t) SA_STUB()
void launch_select_protected(const float*, int, int, int, int32_t*, uint8_t*,
                             hipStream_t) SA_STUB()
void launch_build_block_mask(const void*, const void*, int, int, int, int, int, float, int, int,
                             const uint8_t*, int32_t*, int32_t*, uint8_t*, float*, char*,
                             hipStream_t) SA_STUB()
void launch_block_pool(const void*, const void*, int, int, int, int, int, int, double*, double*,
                       hipStream_t) SA_STUB()
void launch_mask_from_means(const double*, const double*, int, int, int, int, float, int, int,
                            const uint8_t*, int32_t*, int32_t*, uint8_t*, float*,
                            hipStream_t) SA_STUB()
void launch_sparse_attention_bf16(const uint16_t*, const uint16_t*, const uint16_t*, uint16_t*,
                                  float*, int, int, int, int, float, int, const int32_t*,
                                  const int32_t*, char*, hipStream_t) SA_STUB()
void launch_sparse_attention_f32(const float*, const float*, const float*, float*, float*, int,
                                 int, int, int, float, int, const int32_t*, const int32_t*,
                                 char*, hipStream_t) SA_STUB()

}  // namespace sa
