// Prefill path (MFMA grouped GEMM): placeholder until the kernels land.
#include "moe_internal.h"

namespace moe {

hipError_t launch_prefill_up(const ExpertEntry*, const WorkList*, const int32_t*,
                             const f16*, f16*, f16*, int, int, int, int, int, hipStream_t) {
  return hipErrorNotSupported;
}

hipError_t launch_prefill_down(const ExpertEntry*, const WorkList*, const f16*, float*,
                               int, int, int, int, int, hipStream_t) {
  return hipErrorNotSupported;
}

hipError_t launch_combine_prefill(const float*, const int32_t*, const float*,
                                  const int8_t*, int, int, int, float*, float*, f16*,
                                  float, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace moe
