/*
 * gpps — RBF-ARD psi-statistics and their gradients on AMD Instinct MI355X (gfx950).
 *
 * C ABI of the HIP library libgpps.so.  Plain pointers and sizes only.
 *
 * Notation (Dai, Damianou, Hensman, Lawrence, "Gaussian Process Models with
 * Parallelization and GPU acceleration", section 2 and Alg. 1-2):
 *   N datapoints, M inducing inputs, Q latent dimensions.
 *   q(x_n) = N(mu_n, diag S_n)          variational posterior, factorised over n
 *   Z        inducing inputs (M x Q)
 *   k(x, z)  = sigma_f2 * exp(-1/2 sum_q (x_q - z_q)^2 / l_q^2)      ARD RBF kernel
 *   psi0     = sum_n E_q[k(x_n, x_n)]                     (scalar; the paper's phi)
 *   Psi1     = E_q[k(x_n, z_m)]              N x M         (the per-point Psi_nm of Alg. 1)
 *   Psi2     = sum_n E_q[k(x_n, z_m) k(x_n, z_m')]  M x M  (the paper's Phi, eq. (2)-(4))
 *
 * Conventions shared by every entry point:
 *   - dt selects the element type of EVERY device array of the call
 *     (GPPS_F32: float, GPPS_F64: double).  Arrays are dense, row-major,
 *     contiguous, aligned to their element size, and live in device memory
 *     of the current HIP device.
 *   - mu and S are N x Q (S holds the diagonal VARIANCES), Z is M x Q.
 *   - S = NULL means known inputs: every variance is zero and mu holds the
 *     inputs X themselves, the sparse GP regression case of section 2,
 *     eq. (boundF).  The statistics are then the plain kernel quantities
 *     (psi0 = N sigma_f2, Psi1 = Kfu, Psi2 = Kfu^T Kfu) and run on a separate
 *     matrix-core GEMM path (both dtypes) whatever path flag the call carries;
 *     dmu is dL/dX and dS may be NULL (it is not written).
 *   - sigma_f2 and l (Q values) are HOST doubles, so validation needs no
 *     device synchronisation.  In the F32 path they are rounded to float.
 *   - The caller owns every buffer.  The library allocates nothing, frees
 *     nothing and keeps no pointer after return.  Scratch memory is the
 *     caller's workspace of at least gpps_workspace_bytes(dt, N, M, Q) bytes,
 *     256-byte aligned; its contents on entry are ignored.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = default stream) and
 *     the call returns without synchronising: outputs are valid once the
 *     stream has been synchronised.  The workspace must not be reused by
 *     another call that may run concurrently.
 *   - flags is a bitwise or of GPPS_ACCUMULATE and at most one path flag.
 *     Without GPPS_ACCUMULATE the N-summed outputs are overwritten; with it
 *     they are added to.  This is how N is split into row chunks (section 2:
 *     every data-dependent quantity is a sum over datapoints, so partial
 *     results over disjoint row sets add up).  Per-row outputs (Psi1, dmu, dS)
 *     are always overwritten for the rows passed.  The path flags choose the
 *     kernels per call (the library keeps no path setting of its own).
 *   - Results are bitwise deterministic for fixed (dt, N, M, Q), path and
 *     device: no floating-point atomics are used; every reduction runs in a
 *     fixed order.
 *   - Errors: every argument is validated before any HIP call; on a
 *     validation error nothing is enqueued and nothing is written.  A failed
 *     kernel launch returns GPPS_ERR_HIP; faults during asynchronous execution
 *     surface at the caller's next synchronisation.  NaN or Inf inside device
 *     arrays is not checked and propagates.
 */
#ifndef GPPS_H
#define GPPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { GPPS_F32 = 0, GPPS_F64 = 1 } gpps_dtype;

typedef enum {
    GPPS_OK = 0,
    GPPS_ERR_NULL = 1,      /* a required pointer is NULL                              */
    GPPS_ERR_SHAPE = 2,     /* N < 1, M < 1, Q < 1, Q > GPPS_MAX_Q or M > GPPS_MAX_M   */
    GPPS_ERR_HYPER = 3,     /* sigma_f2 or some l_q is not finite and > 0              */
    GPPS_ERR_DTYPE = 4,     /* dt is not a gpps_dtype                                  */
    GPPS_ERR_WORKSPACE = 5, /* workspace smaller than gpps_workspace_bytes()           */
    GPPS_ERR_ALIGN = 6,     /* workspace not 256-byte aligned or an array misaligned   */
    GPPS_ERR_HIP = 7,       /* a HIP runtime call or kernel launch failed              */
    GPPS_ERR_PATH = 8       /* unknown flag bits, both path flags, or the requested path
                               cannot run this call */
} gpps_status;

/* Flags of gpps_psi_stats / gpps_psi_grads (and the path flags of gpps_bound).
 *
 * With neither path flag the call takes the fastest path that supports it: the
 * matrix-core path for F32 shapes within its limits (M rounded up to 32 at most
 * 512 with Q <= 31, or at most 256 with Q <= GPPS_MAX_Q_MFMA), the generic vector
 * path otherwise.  GPPS_PATH_GENERIC forces the generic path; GPPS_PATH_MFMA
 * asks for the matrix-core path and fails with GPPS_ERR_PATH where it cannot
 * take the call.  The matrix-core path carries its operands as two-part fp16
 * values; a device-side range guard bounds them over every row first, and when a
 * bound leaves the fp16 range the call is computed by the generic kernels
 * instead, with either flag (see gpps_route_word_offset).  Calls with S = NULL
 * always take the known-input path. */
#define GPPS_ACCUMULATE 1
#define GPPS_PATH_GENERIC 2
#define GPPS_PATH_MFMA 4

#define GPPS_MAX_Q 64
#define GPPS_MAX_M 4096
#define GPPS_MAX_Q_MFMA 62
#define GPPS_MAX_D 65536
#define GPPS_MAX_M_BOUND 512

/* Bytes of workspace gpps_psi_stats and gpps_psi_grads need for this shape
 * (the larger of the two, over every path).  0 for an invalid shape or dtype. */
size_t gpps_workspace_bytes(gpps_dtype dt, int64_t N, int64_t M, int64_t Q);

/* Allocation-free gpps_psi_stats, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same computation, arguments and flags as
 * gpps_psi_stats, with the workspace taken from a static device array of
 * GPPS_SCRATCH_BYTES that the library holds on every device it runs on until
 * the process ends.  The call allocates and frees nothing.
 *   - Calls whose workspace (gpps_workspace_bytes) exceeds GPPS_SCRATCH_BYTES
 *     return GPPS_ERR_WORKSPACE before any HIP call; split N into row chunks
 *     with GPPS_ACCUMULATE instead.
 *   - Every call on a device shares that device's array: calls that may
 *     overlap on one device (other streams or threads) race and must be
 *     ordered by the caller.  Contents left by a previous call are ignored.
 *   - The array's device address is looked up on the first call on each
 *     device (hipGetSymbolAddress); GPPS_ERR_HIP if that fails. */
#define GPPS_SCRATCH_BYTES (64 << 20)
gpps_status gpps_psi_stats_noalloc(gpps_dtype dt, int64_t N, int64_t M, int64_t Q,
                                   const void *mu, const void *S, const void *Z,
                                   double sigma_f2, const double *l,
                                   void *psi0, void *Psi1, void *Psi2,
                                   int flags, void *stream);

/* Diagnostics: byte offset, inside the workspace of a gpps_psi_stats,
 * gpps_psi_grads or gpps_bound call of this shape, of a 32-bit "route word".
 * Calls that take the matrix-core path (F32, S != NULL) write it: 0 when the
 * matrix cores computed the call, 1 when the range guard found an operand
 * outside the fp16 range and the generic kernels computed it.  Other calls
 * leave it unchanged.  Valid once the call's stream has been synchronised.
 * SIZE_MAX for an invalid shape or dtype. */
size_t gpps_route_word_offset(gpps_dtype dt, int64_t N, int64_t M, int64_t Q);

/*
 * Forward statistics — section 2, eq. (4) (phi, Phi, Psi as expectations under
 * q(X)); Alg. 1 (Psi_nm per datapoint and inducing input, Phi summed over
 * datapoints for every pair of inducing inputs).
 *
 *   S              device N x Q, or NULL for known inputs (see above).
 *   psi0  [1]      device.  += or = N * sigma_f2
 *   Psi1  [N x M]  device, may be NULL (not computed).  Always overwritten.
 *   Psi2  [M x M]  device.  Full symmetric matrix; both triangles are bitwise
 *                  equal.  += or = according to GPPS_ACCUMULATE in flags.
 */
gpps_status gpps_psi_stats(gpps_dtype dt, int64_t N, int64_t M, int64_t Q,
                           const void *mu, const void *S, const void *Z,
                           double sigma_f2, const double *l,
                           void *psi0, void *Psi1, void *Psi2,
                           int flags, void *workspace, size_t workspace_bytes,
                           void *stream);

/*
 * Gradients — Alg. 2: given dL/dPsi, the derivatives of
 *   L = dL_dpsi0 * psi0 + sum_{n,m} dL_dPsi1[n,m] Psi1[n,m]
 *                       + sum_{m,m'} dL_dPsi2[m,m'] Psi2[m,m']
 * with respect to mu, S, Z, sigma_f2 and every l_q (the lengthscales
 * themselves, not their logarithms; S as variances).
 *
 *   dL_dpsi0            host scalar.
 *   dL_dPsi1 [N x M]    device, or NULL for zero.
 *   dL_dPsi2 [M x M]    device, or NULL for zero.  Need not be symmetric: only its
 *                       symmetric part affects L, since Psi2 is symmetric.
 *   dmu, dS  [N x Q]    device, always overwritten (dS may be NULL when S is NULL).
 *   dZ       [M x Q]    device, += or = according to GPPS_ACCUMULATE in flags.
 *   dsigma_f2 [1]       device, += or =.
 *   dl       [Q]        device, += or =.
 */
gpps_status gpps_psi_grads(gpps_dtype dt, int64_t N, int64_t M, int64_t Q,
                           const void *mu, const void *S, const void *Z,
                           double sigma_f2, const double *l, double dL_dpsi0,
                           const void *dL_dPsi1, const void *dL_dPsi2,
                           void *dmu, void *dS, void *dZ, void *dsigma_f2, void *dl,
                           int flags, void *workspace, size_t workspace_bytes,
                           void *stream);

/*
 * Several views sharing one q(X) -- the multi-output compositions of section 1
 * (MRD: each view of the data has its own GP mapping from the same latent
 * points, so the bound is a sum over views plus one KL term of q(X)).
 *
 * View v (0 <= v < V, V <= 64) has M[v] inducing inputs Z[v] (device, M[v] x Q),
 * variance sigma_f2[v] and lengthscales l[v Q .. v Q + Q - 1] (host).  mu and S
 * (device N x Q; S = NULL for known inputs) are shared.  Every per-view output
 * is that of gpps_psi_stats / gpps_psi_grads for the view, with the same flags:
 *   psi0[v], Psi1[v] (may be NULL, or Psi1 itself NULL), Psi2[v],
 *   dZ[v], dsigma_f2[v], dl[v]         host arrays of V device pointers;
 *   dL_dpsi0[v] host, dL_dPsi1[v], dL_dPsi2[v] device (the arrays, or entries, NULL
 *                                       for zero);
 *   dmu, dS [N x Q]                    device: the SUM over views of the views'
 *                                       gradients (overwritten; dS may be NULL when
 *                                       S is NULL).
 * The views run in turn on the single-view kernels and path choice; every view
 * is validated before the first launch (a rejected call enqueues nothing), and
 * the views' dmu, dS are added in view order.  Workspace: at least
 * gpps_views_workspace_bytes(dt, V, N, M, Q) bytes, 256-byte aligned.
 * Errors as for the single-view calls, plus GPPS_ERR_SHAPE for V out of range.
 */
size_t gpps_views_workspace_bytes(gpps_dtype dt, int64_t V, int64_t N, const int64_t *M, int64_t Q);
gpps_status gpps_psi_stats_views(gpps_dtype dt, int64_t V, int64_t N, const int64_t *M, int64_t Q,
                                 const void *mu, const void *S, const void *const *Z,
                                 const double *sigma_f2, const double *l, void *const *psi0,
                                 void *const *Psi1, void *const *Psi2, int flags,
                                 void *workspace, size_t workspace_bytes, void *stream);
gpps_status gpps_psi_grads_views(gpps_dtype dt, int64_t V, int64_t N, const int64_t *M, int64_t Q,
                                 const void *mu, const void *S, const void *const *Z,
                                 const double *sigma_f2, const double *l, const double *dL_dpsi0,
                                 const void *const *dL_dPsi1, const void *const *dL_dPsi2,
                                 void *dmu, void *dS, void *const *dZ, void *const *dsigma_f2,
                                 void *const *dl, int flags, void *workspace,
                                 size_t workspace_bytes, void *stream);

/* Bytes of workspace gpps_bound needs for this shape with D output columns.
 * 0 for an invalid shape, D or dtype (or M > GPPS_MAX_M_BOUND). */
size_t gpps_bound_workspace_bytes(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, int64_t D);

/*
 * The Bayesian GP-LVM variational bound and its gradients — section 2:
 * eq. (boundF), with phi, Phi and the bold Psi turned into their expectations
 * under q(X) (psi0, Psi2 and Psi1^T Y), minus the KL term of eq. (boundBGPLVM)
 * for the prior p(x_n) = N(0, I):
 *
 *   L = -(N D / 2) log 2 pi + (N D / 2) log beta + (D / 2) log|Kmm| - (D / 2) log|A|
 *       - (beta / 2) tr(Y^T Y) + (beta^2 / 2) tr(Psi^T A^-1 Psi)
 *       - (beta D / 2) psi0 + (beta D / 2) tr(Kmm^-1 Psi2)
 *       - 1/2 sum_nq (mu_nq^2 + S_nq - log S_nq - 1),
 *   A = Kmm + beta Psi2,  Kmm = k(Z, Z) + jitter I,  Psi = Psi1^T Y,
 *
 * and dL w.r.t. mu, S, Z, sigma_f2, every l_q and beta (the parameters the paper
 * optimises).  The psi-statistics and their gradients run on the same kernels
 * as gpps_psi_stats / gpps_psi_grads, with the path chosen by the path flags of
 * `flags` (GPPS_ACCUMULATE is not allowed here); the M x M algebra runs in fp64
 * for either dtype.
 *
 *   Y        [N x D]   device, observed data (dtype dt).
 *   beta               host: noise precision, finite and > 0.
 *   jitter             host: added to the diagonal of k(Z, Z), finite and >= 0.
 *   L        [1]       device: the bound (overwritten).
 *   dmu, dS  [N x Q], dZ [M x Q], dsigma_f2 [1], dl [Q], dbeta [1]: device, overwritten.
 *   workspace          at least gpps_bound_workspace_bytes(dt, N, M, Q, D) bytes,
 *                      256-byte aligned, caller-owned (contents ignored).
 *
 * S = NULL (known inputs) gives the sparse GP regression bound of eq. (boundF)
 * itself: no KL term, dmu = dL/dX, and dS may be NULL.
 *
 * Errors as for gpps_psi_grads, plus GPPS_ERR_SHAPE for D < 1, D > GPPS_MAX_D or
 * M > GPPS_MAX_M_BOUND (the triangular inverse keeps a block column in LDS), and GPPS_ERR_HYPER
 * for beta or jitter out of range.  S must be > 0 (log S enters the KL term); a
 * non-positive S, or Kmm or A not positive definite in floating point, is not
 * detected before the call: L and dbeta are then NaN (a non-positive pivot in
 * the inversion is flagged on the device and turns L into NaN).
 */
gpps_status gpps_bound(gpps_dtype dt, int64_t N, int64_t M, int64_t Q, int64_t D,
                       const void *mu, const void *S, const void *Z, const void *Y,
                       double sigma_f2, const double *l, double beta, double jitter,
                       void *L, void *dmu, void *dS, void *dZ, void *dsigma_f2, void *dl,
                       void *dbeta, int flags, void *workspace, size_t workspace_bytes,
                       void *stream);

/* Kernel timing for benchmarks.  While enabled (on != 0), every kernel launch
 * of the library is bracketed by two HIP events recorded on the call's stream.
 * gpps_timing_collect() waits for those events, writes up to max_entries
 * (kernel name, summed milliseconds, launch count) triples into the caller's
 * arrays (any may be NULL), releases the events and returns the number of
 * distinct kernels, or -1 if an event call failed.  Names stay valid until the
 * next collect.  Timing is process-wide and off by default. */
gpps_status gpps_timing_enable(int on);
int gpps_timing_collect(int max_entries, const char **names, double *total_ms,
                        int64_t *launches);

/* Measurement support: sustained rates of the three units the psi-statistic
 * kernels spend their time in, measured on the current device by fixed-size
 * probe kernels enqueued on `stream` (the call synchronises that stream):
 *   rates[0]  fp32 vector flops/s (v_fma_f32, two flops each, unpacked),
 *   rates[1]  v_exp_f32 results/s,
 *   rates[2]  dense f16 matrix-core flops/s (v_mfma_f32_32x32x16_f16).
 * The benchmark prices the kernels' work against them beside the published
 * peaks.  sink: device scratch of at least gpps_probe_sink_bytes() bytes
 * (overwritten).  GPPS_ERR_NULL / GPPS_ERR_WORKSPACE for a missing or short
 * sink, GPPS_ERR_HIP if a probe fails. */
size_t gpps_probe_sink_bytes(void);
gpps_status gpps_probe_unit_rates(void *sink, size_t sink_bytes, double *rates, void *stream);

/* Static, NUL-terminated description of a status code. */
const char *gpps_status_string(gpps_status status);

/* Library version as major * 10000 + minor * 100 + patch. */
int gpps_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GPPS_H */
