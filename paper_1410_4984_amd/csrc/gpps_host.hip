// C ABI of the gpps library: argument validation, workspace sizing and path
// dispatch.  Every check runs before the first HIP call, so a rejected call
// enqueues nothing and writes nothing.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>

#include "internal.h"

namespace {

std::atomic<int> g_path{GPPS_PATH_AUTO};

bool valid_dtype(gpps_dtype dt) { return dt == GPPS_F32 || dt == GPPS_F64; }

bool valid_shape(int64_t N, int64_t M, int64_t Q) {
    return N >= 1 && M >= 1 && Q >= 1 && Q <= GPPS_MAX_Q && M <= GPPS_MAX_M &&
           N <= (int64_t(1) << 40) / M;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

gpps_status check_hypers(double sigma_f2, const double *l, int64_t Q) {
    if (!l) return GPPS_ERR_NULL;
    if (!(sigma_f2 > 0.0) || !std::isfinite(sigma_f2)) return GPPS_ERR_HYPER;
    for (int64_t q = 0; q < Q; ++q)
        if (!(l[q] > 0.0) || !std::isfinite(l[q])) return GPPS_ERR_HYPER;
    return GPPS_OK;
}

template <typename T>
gpps::Hyp<T> make_hyp(double sigma_f2, const double *l, int64_t Q) {
    gpps::Hyp<T> h{};
    for (int64_t q = 0; q < Q; ++q) {
        h.l[q] = T(l[q]);
        h.l2[q] = h.l[q] * h.l[q];
    }
    h.sf2 = T(sigma_f2);
    h.log_sf2 = T(std::log(double(h.sf2)));
    return h;
}

// Which path serves this call (or -1 if the requested one cannot).
int choose_path(gpps_dtype dt, const gpps::Shape &s) {
    int p = g_path.load();
    bool mfma_ok = dt == GPPS_F32 && gpps::mfma_supports(s);
    if (p == GPPS_PATH_AUTO) return mfma_ok ? GPPS_PATH_MFMA : GPPS_PATH_GENERIC;
    if (p == GPPS_PATH_MFMA) return mfma_ok ? GPPS_PATH_MFMA : -1;
    return GPPS_PATH_GENERIC;
}

gpps_status check_workspace(gpps_dtype dt, const gpps::Shape &s, void *ws, size_t ws_bytes) {
    if (!ws) return GPPS_ERR_NULL;
    if (!aligned(ws, 256)) return GPPS_ERR_ALIGN;
    if (ws_bytes < gpps_workspace_bytes(dt, s.N, s.M, s.Q)) return GPPS_ERR_WORKSPACE;
    return GPPS_OK;
}

}  // namespace

extern "C" {

size_t gpps_workspace_bytes(gpps_dtype dt, int64_t N, int64_t M, int64_t Q) {
    if (!valid_dtype(dt) || !valid_shape(N, M, Q)) return 0;
    const gpps::Shape s = gpps::make_shape(N, M, Q);
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    size_t b = gpps::generic_workspace_bytes(s, elem);
    if (dt == GPPS_F32 && gpps::mfma_supports(s)) b = std::max(b, gpps::mfma_workspace_bytes(s));
    return b;
}

gpps_status gpps_psi_stats(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, const void *mu,
                           const void *S, const void *Z, double sigma_f2, const double *l,
                           void *psi0, void *Psi1, void *Psi2, int accumulate, void *workspace,
                           size_t workspace_bytes, void *stream) {
    if (!valid_dtype(dt)) return GPPS_ERR_DTYPE;
    if (!valid_shape(N, M, Q)) return GPPS_ERR_SHAPE;
    if (!mu || !S || !Z || !psi0 || !Psi2) return GPPS_ERR_NULL;
    if (gpps_status r = check_hypers(sigma_f2, l, Q)) return r;
    const gpps::Shape s = gpps::make_shape(N, M, Q);
    if (gpps_status r = check_workspace(dt, s, workspace, workspace_bytes)) return r;
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    for (const void *p : {mu, S, Z, (const void *)psi0, (const void *)Psi1, (const void *)Psi2})
        if (p && !aligned(p, elem)) return GPPS_ERR_ALIGN;
    const int path = choose_path(dt, s);
    if (path < 0) return GPPS_ERR_PATH;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (dt == GPPS_F32) {
        const auto h = make_hyp<float>(sigma_f2, l, Q);
        if (path == GPPS_PATH_MFMA)
            e = gpps::mfma_psi_stats(s, (const float *)mu, (const float *)S, (const float *)Z, h,
                                     (float *)psi0, (float *)Psi1, (float *)Psi2, accumulate != 0,
                                     workspace, st);
        else
            e = gpps::generic_psi_stats<float>(s, (const float *)mu, (const float *)S,
                                               (const float *)Z, h, (float *)psi0, (float *)Psi1,
                                               (float *)Psi2, accumulate != 0, workspace, st);
    } else {
        const auto h = make_hyp<double>(sigma_f2, l, Q);
        e = gpps::generic_psi_stats<double>(s, (const double *)mu, (const double *)S,
                                            (const double *)Z, h, (double *)psi0, (double *)Psi1,
                                            (double *)Psi2, accumulate != 0, workspace, st);
    }
    return e == hipSuccess ? GPPS_OK : GPPS_ERR_HIP;
}

gpps_status gpps_psi_grads(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, const void *mu,
                           const void *S, const void *Z, double sigma_f2, const double *l,
                           double dL_dpsi0, const void *dL_dPsi1, const void *dL_dPsi2,
                           void *dmu, void *dS, void *dZ, void *dsigma_f2, void *dl,
                           int accumulate, void *workspace, size_t workspace_bytes,
                           void *stream) {
    if (!valid_dtype(dt)) return GPPS_ERR_DTYPE;
    if (!valid_shape(N, M, Q)) return GPPS_ERR_SHAPE;
    if (!mu || !S || !Z || !dmu || !dS || !dZ || !dsigma_f2 || !dl) return GPPS_ERR_NULL;
    if (gpps_status r = check_hypers(sigma_f2, l, Q)) return r;
    if (!std::isfinite(dL_dpsi0)) return GPPS_ERR_HYPER;
    const gpps::Shape s = gpps::make_shape(N, M, Q);
    if (gpps_status r = check_workspace(dt, s, workspace, workspace_bytes)) return r;
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    for (const void *p : {mu, S, Z, dL_dPsi1, dL_dPsi2, (const void *)dmu, (const void *)dS,
                          (const void *)dZ, (const void *)dsigma_f2, (const void *)dl})
        if (p && !aligned(p, elem)) return GPPS_ERR_ALIGN;
    const int path = choose_path(dt, s);
    if (path < 0) return GPPS_ERR_PATH;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (dt == GPPS_F32) {
        const auto h = make_hyp<float>(sigma_f2, l, Q);
        if (path == GPPS_PATH_MFMA)
            e = gpps::mfma_psi_grads(s, (const float *)mu, (const float *)S, (const float *)Z, h,
                                     float(dL_dpsi0), (const float *)dL_dPsi1,
                                     (const float *)dL_dPsi2, (float *)dmu, (float *)dS,
                                     (float *)dZ, (float *)dsigma_f2, (float *)dl,
                                     accumulate != 0, workspace, st);
        else
            e = gpps::generic_psi_grads<float>(s, (const float *)mu, (const float *)S,
                                               (const float *)Z, h, float(dL_dpsi0),
                                               (const float *)dL_dPsi1, (const float *)dL_dPsi2,
                                               (float *)dmu, (float *)dS, (float *)dZ,
                                               (float *)dsigma_f2, (float *)dl, accumulate != 0,
                                               workspace, st);
    } else {
        const auto h = make_hyp<double>(sigma_f2, l, Q);
        e = gpps::generic_psi_grads<double>(s, (const double *)mu, (const double *)S,
                                            (const double *)Z, h, dL_dpsi0,
                                            (const double *)dL_dPsi1, (const double *)dL_dPsi2,
                                            (double *)dmu, (double *)dS, (double *)dZ,
                                            (double *)dsigma_f2, (double *)dl, accumulate != 0,
                                            workspace, st);
    }
    return e == hipSuccess ? GPPS_OK : GPPS_ERR_HIP;
}

gpps_status gpps_set_path(gpps_path path) {
    if (path != GPPS_PATH_AUTO && path != GPPS_PATH_GENERIC && path != GPPS_PATH_MFMA)
        return GPPS_ERR_PATH;
    g_path.store(path);
    return GPPS_OK;
}

gpps_path gpps_get_path(void) { return static_cast<gpps_path>(g_path.load()); }

const char *gpps_status_string(gpps_status status) {
    switch (status) {
        case GPPS_OK: return "success";
        case GPPS_ERR_NULL: return "a required pointer is NULL";
        case GPPS_ERR_SHAPE: return "invalid shape (need 1 <= N, 1 <= M <= GPPS_MAX_M, 1 <= Q <= GPPS_MAX_Q)";
        case GPPS_ERR_HYPER: return "sigma_f2, every l_q and dL_dpsi0 must be finite; sigma_f2 and l_q > 0";
        case GPPS_ERR_DTYPE: return "unknown dtype";
        case GPPS_ERR_WORKSPACE: return "workspace smaller than gpps_workspace_bytes()";
        case GPPS_ERR_ALIGN: return "workspace not 256-byte aligned or array not element-aligned";
        case GPPS_ERR_HIP: return "HIP runtime error or kernel launch failure";
        case GPPS_ERR_PATH: return "unknown path, or the requested path cannot run this call";
    }
    return "unknown status";
}

int gpps_version(void) { return 100; }

}  // extern "C"
