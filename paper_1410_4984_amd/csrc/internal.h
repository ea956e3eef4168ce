// Internal declarations of the gpps HIP library (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/gpps.h"

namespace gpps {

// Host-side hyper-parameters, passed to kernels by value (kernel arguments land
// in scalar registers, so every lane sees them without a memory access).
template <typename T>
struct Hyp {
    T l[GPPS_MAX_Q];       // lengthscales l_q
    T l2[GPPS_MAX_Q];      // l_q^2
    T sf2;                 // sigma_f^2
    T log_sf2;             // log sigma_f^2
};

// Shape of one call plus the derived launch decomposition shared by the
// workspace query and the launchers (so both always agree).
struct Shape {
    int64_t N, M, Q;
    int64_t P;             // M (M + 1) / 2 unique pairs
};

inline Shape make_shape(int64_t N, int64_t M, int64_t Q) {
    return Shape{N, M, Q, M * (M + 1) / 2};
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Brackets one kernel launch with HIP events on `st` while timing is enabled
// (gpps_timing_enable); a no-op otherwise.
class TimedScope {
  public:
    TimedScope(hipStream_t st, const char *name);
    ~TimedScope();
    TimedScope(const TimedScope &) = delete;
    TimedScope &operator=(const TimedScope &) = delete;

  private:
    hipStream_t st_;
    const char *name_;
    hipEvent_t start_{}, stop_{};
    bool active_ = false;
};

// ---------------------------------------------------------------- generic path
// Vector-ALU kernels templated on the element type; they serve F64 and any F32
// shape the matrix-core path does not take.
size_t generic_workspace_bytes(const Shape &s, size_t elem);

template <typename T>
hipError_t generic_psi_stats(const Shape &s, const T *mu, const T *S, const T *Z,
                             const Hyp<T> &h, T *psi0, T *Psi1, T *Psi2, int accumulate,
                             void *ws, hipStream_t st);

template <typename T>
hipError_t generic_psi_grads(const Shape &s, const T *mu, const T *S, const T *Z,
                             const Hyp<T> &h, T dL_dpsi0, const T *G1, const T *G2, T *dmu,
                             T *dS, T *dZ, T *dsf2, T *dl, int accumulate, void *ws,
                             hipStream_t st);

// ---------------------------------------------------------------- matrix-core path
// F32 only: per-datapoint Gram blocks and W * D products on MFMA, exp on VALU.
bool mfma_supports(const Shape &s);
size_t mfma_workspace_bytes(const Shape &s);

hipError_t mfma_psi_stats(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float *psi0, float *Psi1, float *Psi2,
                          int accumulate, void *ws, hipStream_t st);

hipError_t mfma_psi_grads(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float dL_dpsi0, const float *G1,
                          const float *G2, float *dmu, float *dS, float *dZ, float *dsf2,
                          float *dl, int accumulate, void *ws, hipStream_t st);

}  // namespace gpps
