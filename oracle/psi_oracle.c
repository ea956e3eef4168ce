/*
 * Plain fp64 CPU oracle for the RBF-ARD psi-statistics and their gradients.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file; only the tests, the smoke check and the bench's CPU-baseline leg do.
 * It shares no code, header, table or helper with the HIP library.
 *
 * What it computes (Dai, Damianou, Hensman, Lawrence, "Gaussian Process Models
 * with Parallelization and GPU acceleration"):
 *
 *   Section 2, eq. (3)-(4): in the Bayesian GP-LVM the three data-dependent
 *   statistics of the sparse bound become expectations under the factorised
 *   variational posterior q(x_n) = N(mu_n, diag S_n), each a sum over datapoints:
 *     psi0          = sum_n E_q[k(x_n, x_n)]
 *     Psi1[n, m]    = E_q[k(x_n, z_m)]                       (the per-point Psi_nm of Alg. 1)
 *     Psi2[m, m']   = sum_n E_q[k(x_n, z_m) k(x_n, z_m')]    (Phi = sum_n Phi^(n) of Alg. 1)
 *   Section 4 names an RBF kernel, Alg. 2 a per-dimension kernel parameter
 *   theta_q, so the kernel is the ARD RBF
 *     k(x, z) = sf2 * exp(-1/2 sum_q (x_q - z_q)^2 / l_q^2).
 *   Alg. 2: given dL/dPsi (here dL/dpsi0, G1 = dL/dPsi1, G2 = dL/dPsi2) the
 *   derivatives of L w.r.t. mu, S, Z and the kernel parameters (sf2, l_q).
 *
 * The paper does not print the closed forms.  The ones used here are exact
 * one-dimensional Gaussian integrals (the ARD kernel factorises over q):
 *   int N(x; mu, S) exp(-(x - z)^2 / (2 l^2)) dx
 *       = (1 + S/l^2)^(-1/2) exp(-(mu - z)^2 / (2 (l^2 + S)))
 * and, using (x - z)^2 + (x - z')^2 = 2 (x - zbar)^2 + (z - z')^2 / 2,
 *   int N(x; mu, S) exp(-((x - z)^2 + (x - z')^2) / (2 l^2)) dx
 *       = (1 + 2 S/l^2)^(-1/2) exp(-(z - z')^2 / (4 l^2) - (mu - zbar)^2 / (l^2 + 2 S)).
 *
 * The gradients are the derivative of
 *   L = dL_dpsi0 * psi0 + sum_{n,m} G1[n,m] Psi1[n,m] + sum_{m,m'} G2[m,m'] Psi2[m,m']
 * written term by term: for every datapoint n, every ordered pair (m, m') of the
 * full M x M matrix and every dimension q, the derivative of log of that term
 * times the term.  G2 is used through its symmetric part (G2 + G2^T)/2, which
 * leaves L unchanged because Psi2 is symmetric.
 *
 * Loops are plain n -> m -> m' -> q in fp64 with libm exp/log/sqrt; no
 * symmetry trick, no blocking, no reformulation.  OpenMP splits datapoints
 * over threads; each thread keeps private partial sums which are added in
 * thread order, so a run is deterministic for a fixed thread count.
 *
 * Return value of every entry point: 0 on success, 1 bad size, 2 null pointer,
 * 3 bad hyper-parameter, 4 out of memory.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int n_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

static int thread_id(void)
{
#ifdef _OPENMP
    return omp_get_thread_num();
#else
    return 0;
#endif
}

static int check_common(int64_t N, int64_t M, int64_t Q, const double *mu, const double *S,
                        const double *Z, double sf2, const double *l)
{
    if (N < 0 || M < 1 || Q < 1) return 1;
    if ((N > 0 && (!mu || !S)) || !Z || !l) return 2;
    if (!(sf2 > 0.0) || !isfinite(sf2)) return 3;
    for (int64_t q = 0; q < Q; ++q)
        if (!(l[q] > 0.0) || !isfinite(l[q])) return 3;
    return 0;
}

/* E_q[k(x_n, z_m)] for one (n, m): product over q of the 1-D integral above. */
static double psi1_term(int64_t Q, const double *mu_n, const double *S_n, const double *z_m,
                        double sf2, const double *l)
{
    double log_val = log(sf2);
    for (int64_t q = 0; q < Q; ++q) {
        double l2 = l[q] * l[q];
        double d = mu_n[q] - z_m[q];
        log_val += -0.5 * log(1.0 + S_n[q] / l2) - 0.5 * d * d / (l2 + S_n[q]);
    }
    return exp(log_val);
}

/* E_q[k(x_n, z_m) k(x_n, z_m')] for one (n, m, m'). */
static double psi2_term(int64_t Q, const double *mu_n, const double *S_n, const double *z_m,
                        const double *z_mp, double sf2, const double *l)
{
    double log_val = 2.0 * log(sf2);
    for (int64_t q = 0; q < Q; ++q) {
        double l2 = l[q] * l[q];
        double delta = z_m[q] - z_mp[q];
        double zbar = 0.5 * (z_m[q] + z_mp[q]);
        double e = mu_n[q] - zbar;
        log_val += -0.5 * log(1.0 + 2.0 * S_n[q] / l2) - delta * delta / (4.0 * l2) -
                   e * e / (l2 + 2.0 * S_n[q]);
    }
    return exp(log_val);
}

/*
 * Forward statistics (section 2, expectations under q(X) in eq. (4); Alg. 1
 * computes the same quantities).  psi0 [1], Psi1 [N x M] (may be NULL),
 * Psi2 [M x M]; all row-major, all overwritten.
 */
int oracle_psi_stats(int64_t N, int64_t M, int64_t Q, const double *mu, const double *S,
                     const double *Z, double sf2, const double *l, double *psi0, double *Psi1,
                     double *Psi2)
{
    int rc = check_common(N, M, Q, mu, S, Z, sf2, l);
    if (rc) return rc;
    if (!psi0 || !Psi2) return 2;

    /* psi0: sum_n E_q[k(x_n, x_n)]; the RBF kernel has k(x, x) = sf2 for every x. */
    double p0 = 0.0;
    for (int64_t n = 0; n < N; ++n) p0 += sf2;
    *psi0 = p0;

    if (Psi1) {
#pragma omp parallel for schedule(static)
        for (int64_t n = 0; n < N; ++n)
            for (int64_t m = 0; m < M; ++m)
                Psi1[n * M + m] = psi1_term(Q, mu + n * Q, S + n * Q, Z + m * Q, sf2, l);
    }

    int T = n_threads();
    double *part = (double *)calloc((size_t)T * (size_t)(M * M), sizeof(double));
    if (!part) return 4;
#pragma omp parallel
    {
        double *acc = part + (size_t)thread_id() * (size_t)(M * M);
#pragma omp for schedule(static)
        for (int64_t n = 0; n < N; ++n)
            for (int64_t m = 0; m < M; ++m)
                for (int64_t mp = 0; mp < M; ++mp)
                    acc[m * M + mp] +=
                        psi2_term(Q, mu + n * Q, S + n * Q, Z + m * Q, Z + mp * Q, sf2, l);
    }
    for (int64_t i = 0; i < M * M; ++i) {
        double s = 0.0;
        for (int t = 0; t < T; ++t) s += part[(size_t)t * (size_t)(M * M) + i];
        Psi2[i] = s;
    }
    free(part);
    return 0;
}

/*
 * Gradients (Alg. 2: derivatives w.r.t. mu_nq, S_nq, Z_mq and theta given
 * dL/dPsi).  G1 [N x M] or NULL (= 0), G2 [M x M] or NULL (= 0).
 * Outputs dmu, dS [N x Q], dZ [M x Q], dsf2 [1], dl [Q]; all overwritten.
 */
int oracle_psi_grads(int64_t N, int64_t M, int64_t Q, const double *mu, const double *S,
                     const double *Z, double sf2, const double *l, double dL_dpsi0,
                     const double *G1, const double *G2, double *dmu, double *dS, double *dZ,
                     double *dsf2, double *dl)
{
    int rc = check_common(N, M, Q, mu, S, Z, sf2, l);
    if (rc) return rc;
    if ((N > 0 && (!dmu || !dS)) || !dZ || !dsf2 || !dl) return 2;

    int T = n_threads();
    /* per-thread partials of the global gradients: dZ (M*Q), dl (Q), dsf2 (1) */
    size_t width = (size_t)(M * Q + Q + 1);
    double *part = (double *)calloc((size_t)T * width, sizeof(double));
    if (!part) return 4;

#pragma omp parallel
    {
        double *pz = part + (size_t)thread_id() * width;
        double *pl = pz + M * Q;
        double *ps = pl + Q;
#pragma omp for schedule(static)
        for (int64_t n = 0; n < N; ++n) {
            const double *mu_n = mu + n * Q, *S_n = S + n * Q;
            double *dmu_n = dmu + n * Q, *dS_n = dS + n * Q;
            for (int64_t q = 0; q < Q; ++q) dmu_n[q] = dS_n[q] = 0.0;

            /* Psi1 terms: L contains G1[n,m] * Psi1[n,m]. */
            if (G1) {
                for (int64_t m = 0; m < M; ++m) {
                    const double *z_m = Z + m * Q;
                    double t = G1[n * M + m] * psi1_term(Q, mu_n, S_n, z_m, sf2, l);
                    for (int64_t q = 0; q < Q; ++q) {
                        double l2 = l[q] * l[q];
                        double D1 = l2 + S_n[q];
                        double d = mu_n[q] - z_m[q];
                        dmu_n[q] += t * (-d / D1);
                        dS_n[q] += t * (0.5 * d * d / (D1 * D1) - 0.5 / D1);
                        pz[m * Q + q] += t * (d / D1);
                        pl[q] += t * (S_n[q] / (l[q] * D1) + l[q] * d * d / (D1 * D1));
                    }
                    *ps += t / sf2;
                }
            }

            /* Psi2 terms: L contains G2[m,m'] * Psi2_n[m,m'] over ordered pairs. */
            if (G2) {
                for (int64_t m = 0; m < M; ++m) {
                    const double *z_m = Z + m * Q;
                    for (int64_t mp = 0; mp < M; ++mp) {
                        const double *z_mp = Z + mp * Q;
                        double g = 0.5 * (G2[m * M + mp] + G2[mp * M + m]);
                        double t = g * psi2_term(Q, mu_n, S_n, z_m, z_mp, sf2, l);
                        for (int64_t q = 0; q < Q; ++q) {
                            double l2 = l[q] * l[q];
                            double D2 = l2 + 2.0 * S_n[q];
                            double delta = z_m[q] - z_mp[q];
                            double e = mu_n[q] - 0.5 * (z_m[q] + z_mp[q]);
                            dmu_n[q] += t * (-2.0 * e / D2);
                            dS_n[q] += t * (2.0 * e * e / (D2 * D2) - 1.0 / D2);
                            pz[m * Q + q] += t * (e / D2 - delta / (2.0 * l2));
                            pz[mp * Q + q] += t * (e / D2 + delta / (2.0 * l2));
                            pl[q] += t * (2.0 * S_n[q] / (l[q] * D2) +
                                          delta * delta / (2.0 * l2 * l[q]) +
                                          2.0 * l[q] * e * e / (D2 * D2));
                        }
                        *ps += 2.0 * t / sf2;
                    }
                }
            }
        }
    }

    for (size_t i = 0; i < width; ++i) {
        double s = 0.0;
        for (int t = 0; t < T; ++t) s += part[(size_t)t * width + i];
        if (i < (size_t)(M * Q))
            dZ[i] = s;
        else if (i < (size_t)(M * Q + Q))
            dl[i - (size_t)(M * Q)] = s;
        else
            *dsf2 = s;
    }
    /* psi0 = N * sf2 contributes dL_dpsi0 * N to the sf2 gradient and nothing else. */
    *dsf2 += dL_dpsi0 * (double)N;
    free(part);
    return 0;
}

/*
 * Selected entries Psi2[m, m'] (each a full sum over all N datapoints), for
 * checks at sizes where the full M x M oracle is too slow.  pairs holds
 * npairs (m, m') index pairs; out[k] receives Psi2[pairs[2k], pairs[2k+1]].
 */
int oracle_psi2_entries(int64_t N, int64_t M, int64_t Q, const double *mu, const double *S,
                        const double *Z, double sf2, const double *l, int64_t npairs,
                        const int64_t *pairs, double *out)
{
    int rc = check_common(N, M, Q, mu, S, Z, sf2, l);
    if (rc) return rc;
    if (npairs < 0) return 1;
    if (npairs > 0 && (!pairs || !out)) return 2;
    for (int64_t k = 0; k < npairs; ++k)
        if (pairs[2 * k] < 0 || pairs[2 * k] >= M || pairs[2 * k + 1] < 0 || pairs[2 * k + 1] >= M)
            return 1;
    int T = n_threads();
    double *part = (double *)calloc((size_t)T * (size_t)(npairs > 0 ? npairs : 1), sizeof(double));
    if (!part) return 4;
#pragma omp parallel
    {
        double *acc = part + (size_t)thread_id() * (size_t)npairs;
#pragma omp for schedule(static)
        for (int64_t n = 0; n < N; ++n)
            for (int64_t k = 0; k < npairs; ++k)
                acc[k] += psi2_term(Q, mu + n * Q, S + n * Q, Z + pairs[2 * k] * Q,
                                    Z + pairs[2 * k + 1] * Q, sf2, l);
    }
    for (int64_t k = 0; k < npairs; ++k) {
        double s = 0.0;
        for (int t = 0; t < T; ++t) s += part[(size_t)t * (size_t)npairs + k];
        out[k] = s;
    }
    free(part);
    return 0;
}

/*
 * Selected rows dL/dZ[m, :] (each a full sum over all N datapoints and all m'),
 * for checks at sizes where the full gradient oracle is too slow.  rows holds
 * nrows inducing-point indices; out is nrows x Q.  Same per-term derivatives
 * as oracle_psi_grads.
 */
int oracle_dZ_rows(int64_t N, int64_t M, int64_t Q, const double *mu, const double *S,
                   const double *Z, double sf2, const double *l, const double *G1,
                   const double *G2, int64_t nrows, const int64_t *rows, double *out)
{
    int rc = check_common(N, M, Q, mu, S, Z, sf2, l);
    if (rc) return rc;
    if (nrows < 0) return 1;
    if (nrows > 0 && (!rows || !out)) return 2;
    for (int64_t k = 0; k < nrows; ++k)
        if (rows[k] < 0 || rows[k] >= M) return 1;
    int T = n_threads();
    size_t width = (size_t)(nrows * Q);
    double *part = (double *)calloc((size_t)T * (width > 0 ? width : 1), sizeof(double));
    if (!part) return 4;
#pragma omp parallel
    {
        double *acc = part + (size_t)thread_id() * width;
#pragma omp for schedule(static)
        for (int64_t n = 0; n < N; ++n) {
            const double *mu_n = mu + n * Q, *S_n = S + n * Q;
            for (int64_t k = 0; k < nrows; ++k) {
                int64_t m = rows[k];
                const double *z_m = Z + m * Q;
                if (G1) {
                    double t = G1[n * M + m] * psi1_term(Q, mu_n, S_n, z_m, sf2, l);
                    for (int64_t q = 0; q < Q; ++q) {
                        double D1 = l[q] * l[q] + S_n[q];
                        acc[k * Q + q] += t * ((mu_n[q] - z_m[q]) / D1);
                    }
                }
                if (G2) {
                    /* z_m appears in the pairs (m, m') and (m', m) of the full matrix */
                    for (int64_t mp = 0; mp < M; ++mp) {
                        const double *z_mp = Z + mp * Q;
                        double g = 0.5 * (G2[m * M + mp] + G2[mp * M + m]);
                        double t = g * psi2_term(Q, mu_n, S_n, z_m, z_mp, sf2, l);
                        for (int64_t q = 0; q < Q; ++q) {
                            double l2 = l[q] * l[q];
                            double D2 = l2 + 2.0 * S_n[q];
                            double delta = z_m[q] - z_mp[q];
                            double e = mu_n[q] - 0.5 * (z_m[q] + z_mp[q]);
                            /* (m, m') term and its mirror (m', m) contribute equally */
                            acc[k * Q + q] += 2.0 * t * (e / D2 - delta / (2.0 * l2));
                        }
                    }
                }
            }
        }
    }
    for (size_t i = 0; i < width; ++i) {
        double s = 0.0;
        for (int t = 0; t < T; ++t) s += part[(size_t)t * width + i];
        out[i] = s;
    }
    free(part);
    return 0;
}

int oracle_num_threads(void) { return n_threads(); }
