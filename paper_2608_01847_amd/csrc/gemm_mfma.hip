// bf16 MFMA reconstruction GEMMs for gfx950 (not yet enabled: every shape takes the VALU path).
#include "gemm_common.h"

namespace focus {

bool mfma_fwd_supported(int64_t, int64_t, int64_t) { return false; }
bool mfma_bwd_supported(int64_t, int64_t, int64_t) { return false; }

hipError_t launch_fwd_mfma(const void *, const void *, int64_t, int64_t, int64_t, const void *, void *, float,
                           double *, hipStream_t) {
    return hipErrorInvalidValue;
}

hipError_t launch_bwd_mfma(int, int, const void *, const void *, int64_t, int64_t, int64_t, int64_t, int64_t,
                           const void *, const float *, const float *, int, const float *, int, float *, float *,
                           uint32_t *, hipStream_t) {
    return hipErrorInvalidValue;
}

}  // namespace focus
