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
// Vector-ALU kernels templated on the element type; they serve F64, any F32
// shape the matrix-core path does not take, and F32 calls whose operands the
// matrix-core range guard rejects.  gate: NULL, or a device word; the kernels
// then do their work only where it is nonzero (the matrix-core route word).
size_t generic_workspace_bytes(const Shape &s, size_t elem);

template <typename T>
hipError_t generic_psi_stats(const Shape &s, const T *mu, const T *S, const T *Z,
                             const Hyp<T> &h, T *psi0, T *Psi1, T *Psi2, int accumulate,
                             void *ws, const int *gate, hipStream_t st);

template <typename T>
hipError_t generic_psi_grads(const Shape &s, const T *mu, const T *S, const T *Z,
                             const Hyp<T> &h, T dL_dpsi0, const T *G1, const T *G2, T *dmu,
                             T *dS, T *dZ, T *dsf2, T *dl, int accumulate, void *ws,
                             const int *gate, hipStream_t st);

// ---------------------------------------------------------------- matrix-core path
// F32 only: per-datapoint Gram blocks and W * D products on MFMA, exp on VALU.
// route: a device word outside the workspace regions of both paths; the call
// writes 0 there when its operands fit the fp16 range (and computes the
// result), 1 otherwise (and its remaining kernels return at once).
bool mfma_supports(const Shape &s);
size_t mfma_workspace_bytes(const Shape &s);

hipError_t mfma_psi_stats(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float *psi0, float *Psi1, float *Psi2,
                          int accumulate, int *route, void *ws, hipStream_t st);

hipError_t mfma_psi_grads(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float dL_dpsi0, const float *G1,
                          const float *G2, float *dmu, float *dS, float *dZ, float *dsf2,
                          float *dl, int accumulate, int *route, void *ws, hipStream_t st);

// ---------------------------------------------------------------- known inputs (S = 0)
// Psi1 = Kfu, Psi2 = Kfu^T Kfu on the matrix cores (fp32 and fp64); X holds the
// inputs (the mu argument of the ABI).
size_t known_workspace_bytes(const Shape &s, size_t elem);

template <typename T>
hipError_t known_psi_stats(const Shape &s, const T *X, const T *Z, const Hyp<T> &h, T *psi0,
                           T *Psi1, T *Psi2, int accumulate, void *ws, hipStream_t st);

template <typename T>
hipError_t known_psi_grads(const Shape &s, const T *X, const T *Z, const Hyp<T> &h, T dL_dpsi0,
                           const T *G1, const T *G2, T *dX, T *dZ, T *dsf2, T *dl, int accumulate,
                           void *ws, hipStream_t st);

// ---------------------------------------------------------------- entry points, split
// The checks of gpps_psi_stats / gpps_psi_grads (no HIP call; *path gets the
// path that will serve the call) and their launches, for entry points that
// validate several calls before enqueueing any (the multi-view ones).
gpps_status check_stats(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, const void *mu,
                        const void *S, const void *Z, double sigma_f2, const double *l,
                        void *psi0, void *Psi1, void *Psi2, int flags, void *workspace,
                        size_t workspace_bytes, int *path);
hipError_t launch_stats(gpps_dtype dt, int path, int64_t N, int64_t M, int64_t Q, const void *mu,
                        const void *S, const void *Z, double sigma_f2, const double *l, void *psi0,
                        void *Psi1, void *Psi2, int flags, void *workspace, hipStream_t st);
gpps_status check_grads(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, const void *mu,
                        const void *S, const void *Z, double sigma_f2, const double *l,
                        double dL_dpsi0, const void *dL_dPsi1, const void *dL_dPsi2, void *dmu,
                        void *dS, void *dZ, void *dsigma_f2, void *dl, int flags, void *workspace,
                        size_t workspace_bytes, int *path);
hipError_t launch_grads(gpps_dtype dt, int path, int64_t N, int64_t M, int64_t Q, const void *mu,
                        const void *S, const void *Z, double sigma_f2, const double *l,
                        double dL_dpsi0, const void *dL_dPsi1, const void *dL_dPsi2, void *dmu,
                        void *dS, void *dZ, void *dsigma_f2, void *dl, int flags, void *workspace,
                        hipStream_t st);

// ---------------------------------------------------------------- Bayesian GP-LVM bound
// Byte offsets of the psi-statistic buffers inside the bound's workspace (after
// the first psi_ws bytes, which serve the psi-statistic kernels).
struct BoundBufs {
    size_t psi0, psi1, psi2, g2;
};
size_t bound_workspace_bytes(const Shape &s, int64_t D, size_t elem, size_t psi_ws);
BoundBufs bound_buffers(const Shape &s, int64_t D, size_t elem, size_t psi_ws);

// After the psi-statistics: Kmm, A, their inverses and log determinants, Psi1^T Y,
// the bound L and dL/dbeta, and dL/dPsi1 (over Psi1) and dL/dPsi2 in the workspace.
// S = nullptr: known inputs, no KL term.
template <typename T>
hipError_t bound_middle(const Shape &s, int64_t D, const T *mu, const T *S, const T *Z, const T *Y,
                        const Hyp<T> &h, double beta, double jitter, T *L, T *dbeta, void *ws,
                        size_t psi_ws, hipStream_t st);

// After the psi-statistic gradients: the chain rule through Kmm (added to dZ,
// dsigma_f2, dl) and the KL term (added to dmu, dS; skipped when S = nullptr).
template <typename T>
hipError_t bound_tail(const Shape &s, int64_t D, const T *mu, const T *S, const T *Z, const Hyp<T> &h,
                      T *dmu, T *dS, T *dZ, T *dsf2, T *dl, void *ws, size_t psi_ws, hipStream_t st);

}  // namespace gpps
