// C ABI of the gpps library: argument validation, workspace sizing and path
// dispatch.  Every check runs before the first HIP call, so a rejected call
// enqueues nothing and writes nothing.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace {

constexpr int kPathAuto = 0, kPathGeneric = 1, kPathMfma = 2;

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

// The path a call asks for through its flags (-1: unknown bits or both path
// flags; `allowed` are the bits the entry point accepts).
int requested_path(int flags, int allowed) {
    if (flags & ~allowed) return -1;
    const bool g = flags & GPPS_PATH_GENERIC, m = flags & GPPS_PATH_MFMA;
    if (g && m) return -1;
    return g ? kPathGeneric : (m ? kPathMfma : kPathAuto);
}

// Which path serves a call with variances S (or -1 if the requested one
// cannot).  Calls without S (known inputs) always take the known-input path.
constexpr int kPathKnown = 100;

int choose_path(gpps_dtype dt, const gpps::Shape &s, const void *S, int requested) {
    if (!S) return kPathKnown;
    const bool mfma_ok = dt == GPPS_F32 && gpps::mfma_supports(s);
    if (requested == kPathAuto) return mfma_ok ? kPathMfma : kPathGeneric;
    if (requested == kPathMfma) return mfma_ok ? kPathMfma : -1;
    return kPathGeneric;
}

// Bytes of the psi-statistic workspace before the route word (the largest
// region of any path), and the route word's offset.
size_t regions_bytes(gpps_dtype dt, const gpps::Shape &s) {
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    size_t b = std::max(gpps::generic_workspace_bytes(s, elem), gpps::known_workspace_bytes(s, elem));
    if (dt == GPPS_F32 && gpps::mfma_supports(s)) b = std::max(b, gpps::mfma_workspace_bytes(s));
    return gpps::align_up(b, 256);
}

int *route_word(gpps_dtype dt, const gpps::Shape &s, void *ws) {
    return reinterpret_cast<int *>(static_cast<char *>(ws) + regions_bytes(dt, s));
}

gpps_status check_workspace(gpps_dtype dt, const gpps::Shape &s, void *ws, size_t ws_bytes) {
    if (!ws) return GPPS_ERR_NULL;
    if (!aligned(ws, 256)) return GPPS_ERR_ALIGN;
    if (ws_bytes < gpps_workspace_bytes(dt, s.N, s.M, s.Q)) return GPPS_ERR_WORKSPACE;
    return GPPS_OK;
}

// The psi-statistics / their gradients on the chosen path (arguments already checked).
hipError_t run_stats(gpps_dtype dt, int path, const gpps::Shape &s, const void *mu, const void *S,
                     const void *Z, double sigma_f2, const double *l, void *psi0, void *Psi1,
                     void *Psi2, int accumulate, void *ws, hipStream_t st) {
    if (path == kPathKnown) {
        if (dt == GPPS_F32)
            return gpps::known_psi_stats<float>(s, (const float *)mu, (const float *)Z,
                                                make_hyp<float>(sigma_f2, l, s.Q), (float *)psi0,
                                                (float *)Psi1, (float *)Psi2, accumulate != 0, ws, st);
        return gpps::known_psi_stats<double>(s, (const double *)mu, (const double *)Z,
                                             make_hyp<double>(sigma_f2, l, s.Q), (double *)psi0,
                                             (double *)Psi1, (double *)Psi2, accumulate != 0, ws, st);
    }
    if (dt == GPPS_F32) {
        const auto h = make_hyp<float>(sigma_f2, l, s.Q);
        const int *gate = nullptr;
        if (path == kPathMfma) {
            // the matrix-core kernels, then the generic ones gated by the route
            // word: only one of the two sets does the work
            int *route = route_word(dt, s, ws);
            hipError_t e = gpps::mfma_psi_stats(s, (const float *)mu, (const float *)S,
                                                (const float *)Z, h, (float *)psi0, (float *)Psi1,
                                                (float *)Psi2, accumulate != 0, route, ws, st);
            if (e != hipSuccess) return e;
            gate = route;
        }
        return gpps::generic_psi_stats<float>(s, (const float *)mu, (const float *)S,
                                              (const float *)Z, h, (float *)psi0, (float *)Psi1,
                                              (float *)Psi2, accumulate != 0, ws, gate, st);
    }
    const auto h = make_hyp<double>(sigma_f2, l, s.Q);
    return gpps::generic_psi_stats<double>(s, (const double *)mu, (const double *)S,
                                           (const double *)Z, h, (double *)psi0, (double *)Psi1,
                                           (double *)Psi2, accumulate != 0, ws, nullptr, st);
}

hipError_t run_grads(gpps_dtype dt, int path, const gpps::Shape &s, const void *mu, const void *S,
                     const void *Z, double sigma_f2, const double *l, double dL_dpsi0,
                     const void *dL_dPsi1, const void *dL_dPsi2, void *dmu, void *dS, void *dZ,
                     void *dsigma_f2, void *dl, int accumulate, void *ws, hipStream_t st) {
    if (path == kPathKnown) {
        if (dt == GPPS_F32)
            return gpps::known_psi_grads<float>(
                s, (const float *)mu, (const float *)Z, make_hyp<float>(sigma_f2, l, s.Q),
                float(dL_dpsi0), (const float *)dL_dPsi1, (const float *)dL_dPsi2, (float *)dmu,
                (float *)dZ, (float *)dsigma_f2, (float *)dl, accumulate != 0, ws, st);
        return gpps::known_psi_grads<double>(
            s, (const double *)mu, (const double *)Z, make_hyp<double>(sigma_f2, l, s.Q), dL_dpsi0,
            (const double *)dL_dPsi1, (const double *)dL_dPsi2, (double *)dmu, (double *)dZ,
            (double *)dsigma_f2, (double *)dl, accumulate != 0, ws, st);
    }
    if (dt == GPPS_F32) {
        const auto h = make_hyp<float>(sigma_f2, l, s.Q);
        const int *gate = nullptr;
        if (path == kPathMfma) {
            int *route = route_word(dt, s, ws);
            hipError_t e = gpps::mfma_psi_grads(
                s, (const float *)mu, (const float *)S, (const float *)Z, h, float(dL_dpsi0),
                (const float *)dL_dPsi1, (const float *)dL_dPsi2, (float *)dmu, (float *)dS,
                (float *)dZ, (float *)dsigma_f2, (float *)dl, accumulate != 0, route, ws, st);
            if (e != hipSuccess) return e;
            gate = route;
        }
        return gpps::generic_psi_grads<float>(s, (const float *)mu, (const float *)S,
                                              (const float *)Z, h, float(dL_dpsi0),
                                              (const float *)dL_dPsi1, (const float *)dL_dPsi2,
                                              (float *)dmu, (float *)dS, (float *)dZ,
                                              (float *)dsigma_f2, (float *)dl, accumulate != 0,
                                              ws, gate, st);
    }
    const auto h = make_hyp<double>(sigma_f2, l, s.Q);
    return gpps::generic_psi_grads<double>(s, (const double *)mu, (const double *)S,
                                           (const double *)Z, h, dL_dpsi0,
                                           (const double *)dL_dPsi1, (const double *)dL_dPsi2,
                                           (double *)dmu, (double *)dS, (double *)dZ,
                                           (double *)dsigma_f2, (double *)dl, accumulate != 0, ws,
                                           nullptr, st);
}

}  // namespace

extern "C" {

size_t gpps_workspace_bytes(gpps_dtype dt, int64_t N, int64_t M, int64_t Q) {
    if (!valid_dtype(dt) || !valid_shape(N, M, Q)) return 0;
    return regions_bytes(dt, gpps::make_shape(N, M, Q)) + 256;  // + the route word
}

size_t gpps_route_word_offset(gpps_dtype dt, int64_t N, int64_t M, int64_t Q) {
    if (!valid_dtype(dt) || !valid_shape(N, M, Q)) return SIZE_MAX;
    return regions_bytes(dt, gpps::make_shape(N, M, Q));
}

}  // extern "C"

namespace gpps {

// Every check of gpps_psi_stats, without any HIP call; *path gets the path
// that will serve the call.
gpps_status check_stats(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, const void *mu,
                        const void *S, const void *Z, double sigma_f2, const double *l,
                        void *psi0, void *Psi1, void *Psi2, int flags, void *workspace,
                        size_t workspace_bytes, int *path_out) {
    if (!valid_dtype(dt)) return GPPS_ERR_DTYPE;
    if (!valid_shape(N, M, Q)) return GPPS_ERR_SHAPE;
    if (!mu || !Z || !psi0 || !Psi2) return GPPS_ERR_NULL;
    if (gpps_status r = check_hypers(sigma_f2, l, Q)) return r;
    const gpps::Shape s = gpps::make_shape(N, M, Q);
    if (gpps_status r = check_workspace(dt, s, workspace, workspace_bytes)) return r;
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    for (const void *p : {mu, S, Z, (const void *)psi0, (const void *)Psi1, (const void *)Psi2})
        if (p && !aligned(p, elem)) return GPPS_ERR_ALIGN;
    const int req = requested_path(flags, GPPS_ACCUMULATE | GPPS_PATH_GENERIC | GPPS_PATH_MFMA);
    if (req < 0) return GPPS_ERR_PATH;
    const int path = choose_path(dt, s, S, req);
    if (path < 0) return GPPS_ERR_PATH;
    *path_out = path;
    return GPPS_OK;
}

hipError_t launch_stats(gpps_dtype dt, int path, int64_t N, int64_t M, int64_t Q, const void *mu,
                        const void *S, const void *Z, double sigma_f2, const double *l, void *psi0,
                        void *Psi1, void *Psi2, int flags, void *workspace, hipStream_t st) {
    return run_stats(dt, path, make_shape(N, M, Q), mu, S, Z, sigma_f2, l, psi0, Psi1, Psi2,
                     flags & GPPS_ACCUMULATE, workspace, st);
}

// Every check of gpps_psi_grads, without any HIP call.
gpps_status check_grads(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, const void *mu,
                        const void *S, const void *Z, double sigma_f2, const double *l,
                        double dL_dpsi0, const void *dL_dPsi1, const void *dL_dPsi2, void *dmu,
                        void *dS, void *dZ, void *dsigma_f2, void *dl, int flags, void *workspace,
                        size_t workspace_bytes, int *path_out) {
    if (!valid_dtype(dt)) return GPPS_ERR_DTYPE;
    if (!valid_shape(N, M, Q)) return GPPS_ERR_SHAPE;
    if (!mu || !Z || !dmu || (S && !dS) || !dZ || !dsigma_f2 || !dl) return GPPS_ERR_NULL;
    if (gpps_status r = check_hypers(sigma_f2, l, Q)) return r;
    if (!std::isfinite(dL_dpsi0)) return GPPS_ERR_HYPER;
    const gpps::Shape s = gpps::make_shape(N, M, Q);
    if (gpps_status r = check_workspace(dt, s, workspace, workspace_bytes)) return r;
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    for (const void *p : {mu, S, Z, dL_dPsi1, dL_dPsi2, (const void *)dmu, (const void *)dS,
                          (const void *)dZ, (const void *)dsigma_f2, (const void *)dl})
        if (p && !aligned(p, elem)) return GPPS_ERR_ALIGN;
    const int req = requested_path(flags, GPPS_ACCUMULATE | GPPS_PATH_GENERIC | GPPS_PATH_MFMA);
    if (req < 0) return GPPS_ERR_PATH;
    const int path = choose_path(dt, s, S, req);
    if (path < 0) return GPPS_ERR_PATH;
    *path_out = path;
    return GPPS_OK;
}

hipError_t launch_grads(gpps_dtype dt, int path, int64_t N, int64_t M, int64_t Q, const void *mu,
                        const void *S, const void *Z, double sigma_f2, const double *l,
                        double dL_dpsi0, const void *dL_dPsi1, const void *dL_dPsi2, void *dmu,
                        void *dS, void *dZ, void *dsigma_f2, void *dl, int flags, void *workspace,
                        hipStream_t st) {
    return run_grads(dt, path, make_shape(N, M, Q), mu, S, Z, sigma_f2, l, dL_dpsi0, dL_dPsi1,
                     dL_dPsi2, dmu, dS, dZ, dsigma_f2, dl, flags & GPPS_ACCUMULATE, workspace, st);
}

}  // namespace gpps

extern "C" {

gpps_status gpps_psi_stats(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, const void *mu,
                           const void *S, const void *Z, double sigma_f2, const double *l,
                           void *psi0, void *Psi1, void *Psi2, int flags, void *workspace,
                           size_t workspace_bytes, void *stream) {
    int path = -1;
    if (gpps_status r = gpps::check_stats(dt, N, M, Q, mu, S, Z, sigma_f2, l, psi0, Psi1, Psi2,
                                          flags, workspace, workspace_bytes, &path))
        return r;
    const hipError_t e = gpps::launch_stats(dt, path, N, M, Q, mu, S, Z, sigma_f2, l, psi0, Psi1,
                                            Psi2, flags, workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? GPPS_OK : GPPS_ERR_HIP;
}

gpps_status gpps_psi_grads(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, const void *mu,
                           const void *S, const void *Z, double sigma_f2, const double *l,
                           double dL_dpsi0, const void *dL_dPsi1, const void *dL_dPsi2,
                           void *dmu, void *dS, void *dZ, void *dsigma_f2, void *dl,
                           int flags, void *workspace, size_t workspace_bytes,
                           void *stream) {
    int path = -1;
    if (gpps_status r = gpps::check_grads(dt, N, M, Q, mu, S, Z, sigma_f2, l, dL_dpsi0, dL_dPsi1,
                                          dL_dPsi2, dmu, dS, dZ, dsigma_f2, dl, flags, workspace,
                                          workspace_bytes, &path))
        return r;
    const hipError_t e = gpps::launch_grads(dt, path, N, M, Q, mu, S, Z, sigma_f2, l, dL_dpsi0,
                                            dL_dPsi1, dL_dPsi2, dmu, dS, dZ, dsigma_f2, dl, flags,
                                            workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? GPPS_OK : GPPS_ERR_HIP;
}

size_t gpps_bound_workspace_bytes(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, int64_t D) {
    if (!valid_dtype(dt) || !valid_shape(N, M, Q) || D < 1 || D > GPPS_MAX_D || M > GPPS_MAX_M_BOUND)
        return 0;
    const gpps::Shape s = gpps::make_shape(N, M, Q);
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    return gpps::bound_workspace_bytes(s, D, elem, gpps_workspace_bytes(dt, N, M, Q));
}

gpps_status gpps_bound(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, int64_t D, const void *mu,
                       const void *S, const void *Z, const void *Y, double sigma_f2, const double *l,
                       double beta, double jitter, void *L, void *dmu, void *dS, void *dZ,
                       void *dsigma_f2, void *dl, void *dbeta, int flags, void *workspace,
                       size_t workspace_bytes, void *stream) {
    if (!valid_dtype(dt)) return GPPS_ERR_DTYPE;
    if (!valid_shape(N, M, Q) || D < 1 || D > GPPS_MAX_D || M > GPPS_MAX_M_BOUND) return GPPS_ERR_SHAPE;
    if (!mu || !Z || !Y || !L || !dmu || (S && !dS) || !dZ || !dsigma_f2 || !dl || !dbeta)
        return GPPS_ERR_NULL;
    if (gpps_status r = check_hypers(sigma_f2, l, Q)) return r;
    if (!(beta > 0.0) || !std::isfinite(beta) || !(jitter >= 0.0) || !std::isfinite(jitter))
        return GPPS_ERR_HYPER;
    if (!workspace) return GPPS_ERR_NULL;
    if (!aligned(workspace, 256)) return GPPS_ERR_ALIGN;
    if (workspace_bytes < gpps_bound_workspace_bytes(dt, N, M, Q, D)) return GPPS_ERR_WORKSPACE;
    const size_t elem = dt == GPPS_F32 ? 4 : 8;
    for (const void *p : {mu, S, Z, Y, (const void *)L, (const void *)dmu, (const void *)dS,
                          (const void *)dZ, (const void *)dsigma_f2, (const void *)dl,
                          (const void *)dbeta})
        if (p && !aligned(p, elem)) return GPPS_ERR_ALIGN;
    const gpps::Shape s = gpps::make_shape(N, M, Q);
    const int req = requested_path(flags, GPPS_PATH_GENERIC | GPPS_PATH_MFMA);
    if (req < 0) return GPPS_ERR_PATH;
    const int path = choose_path(dt, s, S, req);
    if (path < 0) return GPPS_ERR_PATH;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const size_t psi_ws = gpps_workspace_bytes(dt, N, M, Q);
    const gpps::BoundBufs b = gpps::bound_buffers(s, D, elem, psi_ws);
    char *w = static_cast<char *>(workspace);
    void *psi0 = w + b.psi0, *Psi1 = w + b.psi1, *Psi2 = w + b.psi2, *G2 = w + b.g2;
    hipError_t e = run_stats(dt, path, s, mu, S, Z, sigma_f2, l, psi0, Psi1, Psi2, 0, workspace, st);
    if (e == hipSuccess) {
        if (dt == GPPS_F32)
            e = gpps::bound_middle<float>(s, D, (const float *)mu, (const float *)S, (const float *)Z,
                                          (const float *)Y, make_hyp<float>(sigma_f2, l, Q), beta,
                                          jitter, (float *)L, (float *)dbeta, workspace, psi_ws, st);
        else
            e = gpps::bound_middle<double>(s, D, (const double *)mu, (const double *)S,
                                           (const double *)Z, (const double *)Y,
                                           make_hyp<double>(sigma_f2, l, Q), beta, jitter,
                                           (double *)L, (double *)dbeta, workspace, psi_ws, st);
    }
    if (e == hipSuccess)
        e = run_grads(dt, path, s, mu, S, Z, sigma_f2, l, -0.5 * beta * (double)D, Psi1, G2, dmu, dS,
                      dZ, dsigma_f2, dl, 0, workspace, st);
    if (e == hipSuccess) {
        if (dt == GPPS_F32)
            e = gpps::bound_tail<float>(s, D, (const float *)mu, (const float *)S, (const float *)Z,
                                        make_hyp<float>(sigma_f2, l, Q), (float *)dmu, (float *)dS,
                                        (float *)dZ, (float *)dsigma_f2, (float *)dl, workspace,
                                        psi_ws, st);
        else
            e = gpps::bound_tail<double>(s, D, (const double *)mu, (const double *)S,
                                         (const double *)Z, make_hyp<double>(sigma_f2, l, Q),
                                         (double *)dmu, (double *)dS, (double *)dZ,
                                         (double *)dsigma_f2, (double *)dl, workspace, psi_ws, st);
    }
    return e == hipSuccess ? GPPS_OK : GPPS_ERR_HIP;
}

const char *gpps_status_string(gpps_status status) {
    switch (status) {
        case GPPS_OK: return "success";
        case GPPS_ERR_NULL: return "a required pointer is NULL";
        case GPPS_ERR_SHAPE: return "invalid shape (need 1 <= N, 1 <= M <= GPPS_MAX_M, 1 <= Q <= GPPS_MAX_Q, 1 <= D <= GPPS_MAX_D)";
        case GPPS_ERR_HYPER: return "sigma_f2, every l_q, dL_dpsi0, beta and jitter must be finite; sigma_f2, l_q, beta > 0, jitter >= 0";
        case GPPS_ERR_DTYPE: return "unknown dtype";
        case GPPS_ERR_WORKSPACE: return "workspace smaller than gpps_workspace_bytes()";
        case GPPS_ERR_ALIGN: return "workspace not 256-byte aligned or array not element-aligned";
        case GPPS_ERR_HIP: return "HIP runtime error or kernel launch failure";
        case GPPS_ERR_PATH: return "unknown flag bits, both path flags, or the requested path cannot run this call";
    }
    return "unknown status";
}

int gpps_version(void) { return 100; }

}  // extern "C"
