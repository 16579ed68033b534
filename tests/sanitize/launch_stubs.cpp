// Stand-ins for the kernel launchers, for a host-only build of the C ABI layer
// (api.hip) under AddressSanitizer and UndefinedBehaviorSanitizer.  No GPU is
// involved: every launcher reports a failed launch, so an entry point that
// passes validation returns PHSA_ERR_HIP without touching the pointers.
#include "../../paper_2601_02819_amd/csrc/launch.h"

namespace phsa {

hipError_t launch_punct_mask(const int32_t *, int64_t, const int32_t *, int, uint8_t *, hipStream_t) {
  return hipErrorLaunchFailure;
}
hipError_t launch_compress(const Geom &, const void *, const uint8_t *, float *, hipStream_t) {
  return hipErrorLaunchFailure;
}
hipError_t launch_select(const Geom &, const void *, const float *, int32_t *, void *, hipStream_t) {
  return hipErrorLaunchFailure;
}
hipError_t launch_attn_fwd(const Geom &, const void *, const void *, const void *, const int32_t *, void *, float *,
                           const IndexWs &, void *, float2 *, hipStream_t) {
  return hipErrorLaunchFailure;
}
hipError_t launch_attn_bwd(const Geom &, const void *, const void *, const void *, const void *, const void *,
                           const float *, const int32_t *, void *, void *, void *, const IndexWs &, float *, void *,
                           float *, float *, bool, hipStream_t) {
  return hipErrorLaunchFailure;
}
hipError_t launch_attn_fwd_fp32(const Geom &, const float *, const float *, const float *, const int32_t *, float *,
                                float *, hipStream_t) {
  return hipErrorLaunchFailure;
}
hipError_t launch_attn_bwd_fp32(const Geom &, const float *, const float *, const float *, const float *,
                                const float *, const float *, const int32_t *, float *, float *, float *, float *,
                                hipStream_t) {
  return hipErrorLaunchFailure;
}
hipError_t launch_decode(const Geom &, const void *, const void *, const void *, const float *, const int32_t *,
                         int32_t *, void *, float *, hipStream_t) {
  return hipErrorLaunchFailure;
}
hipError_t launch_cache_append(const Geom &, const void *, const void *, const uint8_t *, void *, void *, uint8_t *,
                               int32_t *, float *, hipStream_t) {
  return hipErrorLaunchFailure;
}

}  // namespace phsa
