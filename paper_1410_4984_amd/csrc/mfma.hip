// Matrix-core (MFMA) path for F32.  Placeholder until the kernels land.
#include "internal.h"

namespace gpps {

bool mfma_supports(const Shape &) { return false; }
size_t mfma_workspace_bytes(const Shape &) { return 0; }

hipError_t mfma_psi_stats(const Shape &, const float *, const float *, const float *,
                          const Hyp<float> &, float *, float *, float *, int, void *,
                          hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t mfma_psi_grads(const Shape &, const float *, const float *, const float *,
                          const Hyp<float> &, float, const float *, const float *, float *,
                          float *, float *, float *, float *, int, void *, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace gpps
