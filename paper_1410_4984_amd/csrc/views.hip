// Several views of the data sharing one q(X): the multi-output compositions the
// method serves beside the Bayesian GP-LVM (section 1: MRD, where each view has
// its own GP mapping from the shared latent points).  View v has its own
// inducing inputs Z_v (M_v x Q), variance sigma_f2[v] and lengthscales
// l[v Q .. v Q + Q - 1]; every view's statistics are those of gpps_psi_stats on
// the shared mu and S, and since the bound is a sum over views (plus one KL term
// of q(X)), the gradient w.r.t. the shared mu and S is the sum of the views'
// gradients, taken here in view order.
//
// Each view runs on the single-view kernels (and path choice) in turn on the
// caller's stream; every view is validated before the first launch, so a
// rejected call enqueues nothing.  The per-view dmu, dS of views 1 .. V-1 go to a
// workspace buffer placed after the largest single-view workspace and are added
// to dmu, dS by a fixed-order kernel.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace {

constexpr int64_t kMaxViews = 64;

template <typename T>
__global__ __launch_bounds__(256) void add_kernel(int64_t n, const T *__restrict__ src,
                                                  T *__restrict__ dst) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        dst[i] += src[i];
}

hipError_t add(gpps_dtype dt, int64_t n, const void *src, void *dst, hipStream_t st) {
    const unsigned blocks = (unsigned)std::min<int64_t>((n + 255) / 256, 2048);
    gpps::TimedScope ts(st, "views_add");
    if (dt == GPPS_F32)
        add_kernel<float><<<blocks, 256, 0, st>>>(n, (const float *)src, (float *)dst);
    else
        add_kernel<double><<<blocks, 256, 0, st>>>(n, (const double *)src, (double *)dst);
    return hipGetLastError();
}

size_t largest_view_ws(gpps_dtype dt, int64_t V, int64_t N, const int64_t *M, int64_t Q) {
    size_t b = 0;
    for (int64_t v = 0; v < V; ++v) {
        const size_t w = gpps_workspace_bytes(dt, N, M[v], Q);
        if (w == 0) return 0;
        b = std::max(b, w);
    }
    return gpps::align_up(b, 256);
}

}  // namespace

extern "C" {

size_t gpps_views_workspace_bytes(gpps_dtype dt, int64_t V, int64_t N, const int64_t *M, int64_t Q) {
    if (V < 1 || V > kMaxViews || !M) return 0;
    const size_t b = largest_view_ws(dt, V, N, M, Q);
    if (b == 0) return 0;
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    return b + gpps::align_up(2 * elem * (size_t)N * (size_t)Q, 256);
}

gpps_status gpps_psi_stats_views(gpps_dtype dt, int64_t V, int64_t N, const int64_t *M, int64_t Q,
                                 const void *mu, const void *S, const void *const *Z,
                                 const double *sigma_f2, const double *l, void *const *psi0,
                                 void *const *Psi1, void *const *Psi2, int flags, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    if (V < 1 || V > kMaxViews) return GPPS_ERR_SHAPE;
    if (!M || !Z || !sigma_f2 || !l || !psi0 || !Psi2) return GPPS_ERR_NULL;
    const size_t need = gpps_views_workspace_bytes(dt, V, N, M, Q);
    if (need == 0)
        return (dt == GPPS_F32 || dt == GPPS_F64) ? GPPS_ERR_SHAPE : GPPS_ERR_DTYPE;
    if (workspace && workspace_bytes < need) return GPPS_ERR_WORKSPACE;
    int path[kMaxViews];
    for (int64_t v = 0; v < V; ++v)
        if (gpps_status r = gpps::check_stats(dt, N, M[v], Q, mu, S, Z[v], sigma_f2[v], l + v * Q,
                                              psi0[v], Psi1 ? Psi1[v] : nullptr, Psi2[v], flags,
                                              workspace, workspace_bytes, &path[v]))
            return r;
    hipStream_t st = static_cast<hipStream_t>(stream);
    for (int64_t v = 0; v < V; ++v) {
        const hipError_t e = gpps::launch_stats(dt, path[v], N, M[v], Q, mu, S, Z[v], sigma_f2[v],
                                                l + v * Q, psi0[v], Psi1 ? Psi1[v] : nullptr,
                                                Psi2[v], flags, workspace, st);
        if (e != hipSuccess) return GPPS_ERR_HIP;
    }
    return GPPS_OK;
}

gpps_status gpps_psi_grads_views(gpps_dtype dt, int64_t V, int64_t N, const int64_t *M, int64_t Q,
                                 const void *mu, const void *S, const void *const *Z,
                                 const double *sigma_f2, const double *l, const double *dL_dpsi0,
                                 const void *const *dL_dPsi1, const void *const *dL_dPsi2,
                                 void *dmu, void *dS, void *const *dZ, void *const *dsigma_f2,
                                 void *const *dl, int flags, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    if (V < 1 || V > kMaxViews) return GPPS_ERR_SHAPE;
    if (!M || !Z || !sigma_f2 || !l || !dL_dpsi0 || !dZ || !dsigma_f2 || !dl)
        return GPPS_ERR_NULL;
    const size_t need = gpps_views_workspace_bytes(dt, V, N, M, Q);
    if (need == 0)
        return (dt == GPPS_F32 || dt == GPPS_F64) ? GPPS_ERR_SHAPE : GPPS_ERR_DTYPE;
    if (workspace && workspace_bytes < need) return GPPS_ERR_WORKSPACE;
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    char *tmp = workspace ? static_cast<char *>(workspace) + largest_view_ws(dt, V, N, M, Q)
                          : nullptr;
    void *tmp_mu = tmp, *tmp_S = tmp ? tmp + elem * (size_t)N * (size_t)Q : nullptr;
    int path[kMaxViews];
    for (int64_t v = 0; v < V; ++v) {
        // view 0 writes dmu, dS; the others write the workspace buffers
        if (gpps_status r = gpps::check_grads(
                dt, N, M[v], Q, mu, S, Z[v], sigma_f2[v], l + v * Q, dL_dpsi0[v],
                dL_dPsi1 ? dL_dPsi1[v] : nullptr, dL_dPsi2 ? dL_dPsi2[v] : nullptr,
                v == 0 ? dmu : tmp_mu, v == 0 ? dS : (S ? tmp_S : nullptr), dZ[v], dsigma_f2[v],
                dl[v], flags, workspace, workspace_bytes, &path[v]))
            return r;
    }
    hipStream_t st = static_cast<hipStream_t>(stream);
    for (int64_t v = 0; v < V; ++v) {
        void *vmu = v == 0 ? dmu : tmp_mu, *vS = v == 0 ? dS : (S ? tmp_S : nullptr);
        hipError_t e = gpps::launch_grads(
            dt, path[v], N, M[v], Q, mu, S, Z[v], sigma_f2[v], l + v * Q, dL_dpsi0[v],
            dL_dPsi1 ? dL_dPsi1[v] : nullptr, dL_dPsi2 ? dL_dPsi2[v] : nullptr, vmu, vS, dZ[v],
            dsigma_f2[v], dl[v], flags, workspace, st);
        if (e == hipSuccess && v > 0) {
            e = add(dt, N * Q, tmp_mu, dmu, st);
            if (e == hipSuccess && S) e = add(dt, N * Q, tmp_S, dS, st);
        }
        if (e != hipSuccess) return GPPS_ERR_HIP;
    }
    return GPPS_OK;
}

}  // extern "C"
