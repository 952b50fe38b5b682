// attn_bf16.hip -- fast_bf16 contract kernels (not yet built; launchers refuse).
#include "launch.h"

namespace mg {
hipError_t launch_fwd_bf16(const AttnProblem &, const uint16_t *, const uint16_t *,
                           const uint16_t *, uint16_t *, float *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_bwd_rowdot_bf16(const AttnProblem &, const uint16_t *, const uint16_t *,
                                  float *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_bwd_dkdv_bf16(const AttnProblem &, const uint16_t *, const uint16_t *,
                                const uint16_t *, const uint16_t *, const float *,
                                const float *, uint16_t *, uint16_t *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_bwd_dq_bf16(const AttnProblem &, const uint16_t *, const uint16_t *,
                              const uint16_t *, const uint16_t *, const float *, const float *,
                              uint16_t *, hipStream_t) {
    return hipErrorNotSupported;
}
}  // namespace mg
