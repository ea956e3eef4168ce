// The Bayesian GP-LVM bound and its gradients (section 2, eq. (boundF) with the
// kernel statistics turned into expectations under q(X), minus the KL term of
// eq. (boundBGPLVM)):
//
//   F = -(N D / 2) log 2 pi + (N D / 2) log beta + (D / 2) log|Kmm| - (D / 2) log|A|
//       - (beta / 2) tr(Y^T Y) + (beta^2 / 2) tr(Psi^T A^-1 Psi)
//       - (beta D / 2) psi0 + (beta D / 2) tr(Kmm^-1 Psi2),
//   A = Kmm + beta Psi2,   Kmm = k(Z, Z) + jitter I,   Psi = Psi1^T Y   (the paper's bold Psi),
//   KL = 1/2 sum_nq (mu^2 + S - log S - 1),   L = F - KL.
//
// Every term with a sum over datapoints is a data-parallel reduction (psi0, Psi1,
// Psi2 from the psi-statistic kernels, Psi1^T Y, tr(Y^T Y), the KL); the M x M
// algebra in between is the paper's "indistributable" part.  It runs here in
// fp64 whatever the element type of the call: Kmm and A (both symmetric positive
// definite) are factorised together by a blocked right-looking Cholesky, L L^T,
// which gives the log determinants as 2 sum log diag(L); the triangular factors
// are inverted block column by block column and the inverses formed as
// L^-T L^-1.  With C = A^-1 Psi and P = C C^T:
//
//   dL/dpsi0 = -beta D / 2,       dL/dPsi1 = beta^2 Y C^T,
//   dL/dPsi2 = -(beta D / 2) A^-1 - (beta^3 / 2) P + (beta D / 2) Kmm^-1,
//   dL/dKmm  = (D / 2) Kmm^-1 - (D / 2) A^-1 - (beta^2 / 2) P - (beta D / 2) Kmm^-1 Psi2 Kmm^-1,
//   dL/dbeta = N D / (2 beta) - tr(Y^T Y) / 2 - (D / 2) tr(A^-1 Psi2) + beta tr(Psi^T C)
//              - (beta^2 / 2) tr(P Psi2) - (D / 2) psi0 + (D / 2) tr(Kmm^-1 Psi2);
//
// dL/dPsi go through the psi-statistic gradient kernels, dL/dKmm through the
// kernel k(Z, Z) (to Z, sigma_f2, l), and the KL adds -mu to dmu and
// -(1 - 1/S) / 2 to dS.  All reductions run in a fixed order.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace gpps {
namespace {

constexpr int kB = 32;               // block edge of the M x M algebra
constexpr int kRowBlock = 256;       // rows per block of the row reductions
constexpr int64_t kPsiYRows = 256;   // rows per chunk of Psi1^T Y

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct BPlan {
    int64_t Mp;                       // M rounded up to kB
    int nbk;                          // Mp / kB
    int64_t rblocks, ychunks;
    size_t psi_ws;
    size_t off_psi0, off_psi1, off_psi2, off_g2, off_k0, off_gj, off_p2d, off_pm, off_t,
        off_kpk, off_gk, off_psi, off_c, off_ypart, off_rpart, off_tpart, off_ld, off_kdl,
        off_ksf, off_dg, total;
};

BPlan make_bplan(const Shape &s, int64_t D, size_t elem, size_t psi_ws) {
    BPlan p{};
    p.Mp = cdiv(s.M, kB) * kB;
    p.nbk = (int)(p.Mp / kB);
    p.rblocks = cdiv(s.N, kRowBlock);
    p.ychunks = cdiv(s.N, kPsiYRows);
    p.psi_ws = psi_ws;
    size_t o = align_up(psi_ws, 256);
    auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
    const size_t mm = sizeof(double) * p.Mp * p.Mp;
    p.off_psi0 = take(elem);
    p.off_psi1 = take(elem * s.N * s.M);             // Psi1, then dL/dPsi1
    p.off_psi2 = take(elem * s.M * s.M);
    p.off_g2 = take(elem * s.M * s.M);               // dL/dPsi2
    p.off_k0 = take(mm);                             // k(Z, Z) without jitter
    p.off_gj = take(6 * mm);                         // [Kmm, A] -> L; [2] L^-1; [2] inverses
    p.off_p2d = take(mm);                            // Psi2 (fp64, zero-padded)
    p.off_pm = take(mm);                             // P = C C^T
    p.off_t = take(mm);                              // Kmm^-1 Psi2
    p.off_kpk = take(mm);                            // Kmm^-1 Psi2 Kmm^-1
    p.off_gk = take(mm);                             // dL/dKmm
    p.off_psi = take(sizeof(double) * p.Mp * D);     // Psi = Psi1^T Y
    p.off_c = take(sizeof(double) * p.Mp * D);       // C = A^-1 Psi
    p.off_ypart = take(sizeof(double) * p.ychunks * s.M * D);
    p.off_rpart = take(sizeof(double) * p.rblocks * 2);
    p.off_tpart = take(sizeof(double) * p.Mp * 4);
    p.off_ld = take(sizeof(double) * 2 * (p.nbk + 1));  // log det per step and matrix; flag
    p.off_kdl = take(sizeof(double) * s.M * s.Q);
    p.off_ksf = take(sizeof(double) * s.M);
    p.off_dg = take(sizeof(double) * 2 * kB * kB);      // L_KK of the current Cholesky step
    p.total = o;
    return p;
}

template <typename P>
P *at(void *ws, size_t off) { return reinterpret_cast<P *>(static_cast<char *>(ws) + off); }

// ---------------------------------------------------------------- kernels
// Kmm = k(Z, Z) + jitter I and A = Kmm + beta Psi2, both fp64 and padded to Mp with
// the identity; K0 = k(Z, Z) and Psi2 (fp64, zero-padded) kept for later.
template <typename T>
__global__ void bound_kmm_kernel(int M, int Q, int Mp, const T *__restrict__ Z, Hyp<T> h,
                                 double jitter, double beta, const T *__restrict__ Psi2,
                                 double *__restrict__ K0, double *__restrict__ Kj,
                                 double *__restrict__ A, double *__restrict__ P2) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)Mp * Mp) return;
    const int m = (int)(i / Mp), mp = (int)(i - (int64_t)m * Mp);
    if (m < M && mp < M) {
        double s = 0.0;
        for (int q = 0; q < Q; ++q) {
            const double d = ((double)Z[(int64_t)m * Q + q] - (double)Z[(int64_t)mp * Q + q]) / (double)h.l[q];
            s += d * d;
        }
        const double k = (double)h.sf2 * exp(-0.5 * s);
        const double p2 = (double)Psi2[(int64_t)m * M + mp];
        K0[i] = k;
        Kj[i] = k + (m == mp ? jitter : 0.0);
        A[i] = Kj[i] + beta * p2;
        P2[i] = p2;
    } else {
        const double one = m == mp ? 1.0 : 0.0;
        K0[i] = 0.0;
        Kj[i] = one;
        A[i] = one;
        P2[i] = 0.0;
    }
}

// Per block of kRowBlock rows: sum_nd Y^2 and sum_nq (mu^2 + S - log S - 1) / 2
// (zero when S is null: known inputs).
template <typename T>
__global__ __launch_bounds__(256) void bound_rows_kernel(int64_t N, int Q, int64_t D,
                                                         const T *__restrict__ mu,
                                                         const T *__restrict__ S,
                                                         const T *__restrict__ Y,
                                                         double *__restrict__ part) {
    __shared__ double red[2][256];
    const int64_t n0 = (int64_t)blockIdx.x * kRowBlock;
    const int64_t rows = min<int64_t>(kRowBlock, N - n0);
    double yy = 0.0, kl = 0.0;
    for (int64_t k = threadIdx.x; k < rows * D; k += 256) {
        const double y = (double)Y[n0 * D + k];
        yy += y * y;
    }
    if (S) {  // no KL term for known inputs
        for (int64_t k = threadIdx.x; k < rows * Q; k += 256) {
            const double m = (double)mu[n0 * Q + k], s = (double)S[n0 * Q + k];
            kl += 0.5 * (m * m + s - log(s) - 1.0);
        }
    }
    red[0][threadIdx.x] = yy;
    red[1][threadIdx.x] = kl;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w) {
            red[0][threadIdx.x] += red[0][threadIdx.x + w];
            red[1][threadIdx.x] += red[1][threadIdx.x + w];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        part[blockIdx.x * 2] = red[0][0];
        part[blockIdx.x * 2 + 1] = red[1][0];
    }
}

// Psi1^T Y over one chunk of kPsiYRows rows: part[chunk][m][d].  Threads walk
// the (m, d) entries; each sums its chunk's rows in order.
template <typename T>
__global__ __launch_bounds__(256) void bound_psiy_kernel(int64_t N, int M, int64_t D,
                                                         const T *__restrict__ Psi1,
                                                         const T *__restrict__ Y,
                                                         double *__restrict__ part) {
    const int64_t n0 = (int64_t)blockIdx.x * kPsiYRows;
    const int64_t n1 = min<int64_t>(N, n0 + kPsiYRows);
    for (int64_t k = (int64_t)blockIdx.y * 256 + threadIdx.x; k < (int64_t)M * D;
         k += (int64_t)gridDim.y * 256) {
        const int m = (int)(k % M);
        const int64_t d = k / M;
        // row order; loads issued 16 rows at a time so that they overlap
        double s = 0.0;
        int64_t n = n0;
        for (; n + 16 <= n1; n += 16) {
            double a[16], b[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                a[j] = (double)Psi1[(n + j) * M + m];
                b[j] = (double)Y[(n + j) * D + d];
            }
#pragma unroll
            for (int j = 0; j < 16; ++j) s += a[j] * b[j];
        }
        for (; n < n1; ++n) s += (double)Psi1[n * M + m] * (double)Y[n * D + d];
        part[((int64_t)blockIdx.x * D + d) * M + m] = s;
    }
}

// Psi[m][d] = sum over chunks; padded rows zero.  32 outputs per workgroup,
// each summed by 8 groups of threads (group g: chunks g, g + 8, ... in order,
// loads issued 4 at a time), then the 8 group sums in order.
__global__ __launch_bounds__(256) void bound_psiy_reduce_kernel(int M, int Mp, int64_t D, int64_t chunks,
                                                                const double *__restrict__ part,
                                                                double *__restrict__ Psi) {
    __shared__ double gs[8][32];
    const int o = threadIdx.x & 31, g = threadIdx.x >> 5;
    const int64_t k = (int64_t)blockIdx.x * 32 + o;
    const bool in = k < (int64_t)Mp * D;
    const int m = in ? (int)(k / D) : M;
    const int64_t d = in ? k - (int64_t)m * D : 0;
    double s = 0.0;
    if (m < M) {
        const double *src = part + d * M + m;
        const int64_t stride = D * M;
        int64_t c = g;
        for (; c + 24 < chunks; c += 32) {
            double v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = src[(c + 8 * j) * stride];
#pragma unroll
            for (int j = 0; j < 4; ++j) s += v[j];
        }
        for (; c < chunks; c += 8) s += src[c * stride];
    }
    gs[g][o] = s;
    __syncthreads();
    if (g == 0 && in) {
        double t = 0.0;
        for (int j = 0; j < 8; ++j) t += gs[j][o];
        Psi[k] = t;
    }
}

// Lane l's value of v, read by every lane (l uniform).
__device__ inline double lane_bcast(double v, int l) {
    const long long u = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)u, l);
    const int hi = __builtin_amdgcn_readlane((int)(u >> 32), l);
    return __hiloint2double(hi, lo);
}

// Blocked Cholesky, panel step K: workgroup I = K + blockIdx.x of matrix
// blockIdx.y factors the diagonal block A_KK = L_KK L_KK^T (unblocked,
// right-looking) and, for I > K, solves X L_KK^T = A_IK in place.  One wave:
// lane r holds row r of the block (lanes 32-63 repeat rows 0-31); the pivot
// comes from its lane by readlane, and each finished column j of L goes to LDS
// and is read back as broadcasts (a readlane per entry would cost a scalar
// register round trip and its wait states).  Each element is updated in the
// same order as a column sweep over j.  Workgroup K writes L_KK (zero above the diagonal) to the side
// buffer Dg, since the others are still reading tile (K, K) (the update launch
// copies it in), the sum of its log-pivots to logdet[K], and adds the count of
// non-positive pivots to logdet[nbk].
__global__ __launch_bounds__(64) void bound_chol_panel_kernel(int Mp, int K, double *__restrict__ A0,
                                                              double *__restrict__ Dg,
                                                              double *__restrict__ logdet) {
    __shared__ double col[kB];         // column j of L
    __shared__ double Ls[kB][kB + 1];  // L_KK, for the panel solve
    const int I = K + blockIdx.x, mat = blockIdx.y, nbk = Mp / kB;
    double *A = A0 + (int64_t)mat * Mp * Mp;
    const int lane = threadIdx.x, r = lane & (kB - 1);
    const bool own = lane < kB;
    double a[kB];
#pragma unroll
    for (int c = 0; c < kB; ++c) a[c] = A[(int64_t)(K * kB + r) * Mp + K * kB + c];
    double ld = 0.0;
    bool bad = false;
#pragma unroll
    for (int j = 0; j < kB; ++j) {
        const double d = lane_bcast(a[j], j);  // A_jj after steps 0 .. j - 1
        if (I == K) {  // uniform: only the diagonal workgroup records the pivots
            bad |= !(d > 0.0);
            ld += log(d);
        }
        const double ljj = sqrt(d);
        a[j] = r > j ? a[j] / ljj : (r == j ? ljj : 0.0);  // column j of L; zero above
        __syncthreads();  // one wave: orders the previous step's reads before the store
        if (own) col[r] = a[j];
        __syncthreads();
        // trailing update; rows r < c only touch entries above the diagonal,
        // which step c sets to zero
#pragma unroll
        for (int c = j + 1; c < kB; ++c) a[c] -= a[j] * col[c];
    }
    if (I == K) {
        if (own)
#pragma unroll
            for (int c = 0; c < kB; ++c) Dg[(mat * kB + r) * kB + c] = a[c];
        if (lane == 0) {
            logdet[mat * (nbk + 1) + K] = ld;
            const double prev = K == 0 ? 0.0 : logdet[mat * (nbk + 1) + nbk];
            logdet[mat * (nbk + 1) + nbk] = prev + (bad ? 1.0 : 0.0);
        }
        return;
    }
    // X L_KK^T = A_IK, column sweep: x_j = a_j / L_jj, then a_c -= x_j L_cj for c > j
    if (own)
#pragma unroll
        for (int c = 0; c < kB; ++c) Ls[r][c] = a[c];
    double x[kB];
#pragma unroll
    for (int c = 0; c < kB; ++c) x[c] = A[(int64_t)(I * kB + r) * Mp + K * kB + c];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kB; ++j) {
        x[j] /= Ls[j][j];
#pragma unroll
        for (int c = j + 1; c < kB; ++c) x[c] -= x[j] * Ls[c][j];
    }
    if (own)
#pragma unroll
        for (int c = 0; c < kB; ++c) A[(int64_t)(I * kB + r) * Mp + K * kB + c] = x[c];
}

// Blocked Cholesky, trailing update after step K: A_IJ -= L_IK L_JK^T for
// K < J <= I (lower triangle); workgroup (K, K) copies L_KK in from Dg; the
// other workgroups return at once.
__global__ __launch_bounds__(256) void bound_chol_update_kernel(int Mp, int K, double *__restrict__ A0,
                                                                const double *__restrict__ Dg) {
    const int I = blockIdx.x, J = blockIdx.y, mat = blockIdx.z;
    double *A = A0 + (int64_t)mat * Mp * Mp;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    if (I == K && J == K) {
        for (int r = ty; r < kB; r += 8)
            A[(int64_t)(K * kB + r) * Mp + K * kB + tx] = Dg[(mat * kB + r) * kB + tx];
        return;
    }
    if (!(J > K && J <= I)) return;                      // workgroup-uniform
    __shared__ double Li[kB][kB + 1], Lj[kB][kB + 1];
    for (int r = ty; r < kB; r += 8) {
        Li[r][tx] = A[(int64_t)(I * kB + r) * Mp + K * kB + tx];
        Lj[r][tx] = A[(int64_t)(J * kB + r) * Mp + K * kB + tx];
    }
    __syncthreads();
    for (int r = ty; r < kB; r += 8) {
        double s = 0.0;
        for (int k = 0; k < kB; ++k) s += Li[r][k] * Lj[tx][k];
        A[(int64_t)(I * kB + r) * Mp + J * kB + tx] -= s;
    }
}

// Inverse of the lower-triangular factor, one workgroup per block column K and
// matrix: X_KK = L_KK^-1, X_IK = L_II^-1 (-sum_{J=K}^{I-1} L_IJ X_JK) for I > K, by
// forward substitution; the finished X_JK of the column stay in LDS (dynamic:
// one tile of L plus nbk - K tiles of X).  Tiles above the diagonal are written
// as zero.
__global__ __launch_bounds__(256) void bound_trinv_kernel(int Mp, const double *__restrict__ L0,
                                                          double *__restrict__ X0) {
    extern __shared__ double sh[];
    const int K = blockIdx.x, mat = blockIdx.y, nbk = Mp / kB;
    const double *L = L0 + (int64_t)mat * Mp * Mp;
    double *Xg = X0 + (int64_t)mat * Mp * Mp;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    constexpr int kT = kB * (kB + 1);                    // one padded tile
    double *Lt = sh;                                     // tile of L
    double *Xs = sh + kT;                                // X_JK, J = K .. nbk - 1
    auto lt = [&](int r, int c) -> double & { return Lt[r * (kB + 1) + c]; };
    auto xs = [&](int J, int r, int c) -> double & { return Xs[(J - K) * kT + r * (kB + 1) + c]; };
    for (int I = 0; I < K; ++I)
        for (int r = ty; r < kB; r += 8) Xg[(int64_t)(I * kB + r) * Mp + K * kB + tx] = 0.0;
    for (int I = K; I < nbk; ++I) {
        // T = identity (I == K) or -sum_J L_IJ X_JK
        double t[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) t[u] = (I == K && ty + 8 * u == tx) ? 1.0 : 0.0;
        for (int J = K; J < I; ++J) {
            __syncthreads();
            for (int r = ty; r < kB; r += 8) lt(r, tx) = L[(int64_t)(I * kB + r) * Mp + J * kB + tx];
            __syncthreads();
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int r = ty + 8 * u;
                double s = 0.0;
                for (int k = 0; k < kB; ++k) s += lt(r, k) * xs(J, k, tx);
                t[u] -= s;
            }
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < 4; ++u) xs(I, ty + 8 * u, tx) = t[u];
        for (int r = ty; r < kB; r += 8) lt(r, tx) = L[(int64_t)(I * kB + r) * Mp + I * kB + tx];
        __syncthreads();
        // X_IK = L_II^-1 T, column by column (forward substitution: x_j = t_j / L_jj,
        // then t_r -= L_rj x_j for r > j): column c in the registers of lane c of
        // the first wave, L_II read as LDS broadcasts, so no step needs a barrier
        if (threadIdx.x < kB) {
            const int c = threadIdx.x;
            double x[kB];
#pragma unroll
            for (int r = 0; r < kB; ++r) x[r] = xs(I, r, c);
#pragma unroll
            for (int j = 0; j < kB; ++j) {
                x[j] /= lt(j, j);
#pragma unroll
                for (int r = j + 1; r < kB; ++r) x[r] -= lt(r, j) * x[j];
            }
#pragma unroll
            for (int r = 0; r < kB; ++r) xs(I, r, c) = x[r];
        }
        __syncthreads();
        for (int r = ty; r < kB; r += 8) Xg[(int64_t)(I * kB + r) * Mp + K * kB + tx] = xs(I, r, tx);
    }
}

// C = alpha op(A) op(B), row-major fp64: op(A) is rows x inner, op(B) inner x cols.
// 16 x 16 threads per 16 x 16 output tile, inner dimension staged through LDS.
// One product of the M x M algebra: C = alpha op(A) op(B).
struct GemmJob {
    int64_t rows, cols, inner;
    const double *A;
    int64_t lda;
    bool ta;
    const double *B;
    int64_t ldb;
    bool tb;
    double alpha;
    double *C;
    int64_t ldc;
};

// Output tile (bx, by) of job j (the caller keeps it inside the job's tiles).
__device__ inline void gemm_tile(const GemmJob &j, int64_t bx, int64_t by) {
    __shared__ double As[16][17], Bs[16][17];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int64_t r = by * 16 + ty, c = bx * 16 + tx;
    double s = 0.0;
    for (int64_t k0 = 0; k0 < j.inner; k0 += 16) {
        {
            const int64_t ar = by * 16 + ty, ak = k0 + tx;
            As[ty][tx] = (ar < j.rows && ak < j.inner) ? (j.ta ? j.A[ak * j.lda + ar] : j.A[ar * j.lda + ak])
                                                        : 0.0;
            const int64_t bk = k0 + ty, bc = bx * 16 + tx;
            Bs[ty][tx] = (bk < j.inner && bc < j.cols) ? (j.tb ? j.B[bc * j.ldb + bk] : j.B[bk * j.ldb + bc])
                                                        : 0.0;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 16; ++k) s += As[ty][k] * Bs[k][tx];
        __syncthreads();
    }
    if (r < j.rows && c < j.cols) j.C[r * j.ldc + c] = j.alpha * s;
}

// Two independent products in one launch (blockIdx.z selects the job); tiles
// past a job's edge return at once (workgroup-uniform, before any barrier).
__global__ __launch_bounds__(256) void bound_gemm2_kernel(GemmJob j0, GemmJob j1) {
    const GemmJob &j = blockIdx.z == 0 ? j0 : j1;
    if ((int64_t)blockIdx.x * 16 >= j.cols || (int64_t)blockIdx.y * 16 >= j.rows) return;
    gemm_tile(j, blockIdx.x, blockIdx.y);
}

// dL/dPsi2 (element type T, M x M), dL/dKmm (fp64, Mp x Mp) and, per row m, the
// partial traces tr(A^-1 Psi2), tr(P Psi2), tr(Kmm^-1 Psi2) (all symmetric).
template <typename T>
__global__ __launch_bounds__(256) void bound_assemble_kernel(
    int M, int Mp, int64_t D, double beta, const double *__restrict__ Kinv,
    const double *__restrict__ Ainv, const double *__restrict__ Pm, const double *__restrict__ KPK,
    const double *__restrict__ P2, T *__restrict__ G2, double *__restrict__ GK,
    double *__restrict__ tpart) {
    __shared__ double red[3][256];
    const int m = blockIdx.x;
    const double hd = 0.5 * (double)D;
    double ta = 0.0, tp = 0.0, tk = 0.0;
    for (int mp = threadIdx.x; mp < Mp; mp += 256) {
        const int64_t i = (int64_t)m * Mp + mp;
        const double ki = Kinv[i], ai = Ainv[i], pm = Pm[i], p2 = P2[i];
        GK[i] = hd * ki - hd * ai - 0.5 * beta * beta * pm - beta * hd * KPK[i];
        if (m < M && mp < M) {
            G2[(int64_t)m * M + mp] = (T)(-beta * hd * ai - 0.5 * beta * beta * beta * pm + beta * hd * ki);
            ta += ai * p2;
            tp += pm * p2;
            tk += ki * p2;
        }
    }
    red[0][threadIdx.x] = ta;
    red[1][threadIdx.x] = tp;
    red[2][threadIdx.x] = tk;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w)
            for (int j = 0; j < 3; ++j) red[j][threadIdx.x] += red[j][threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        for (int j = 0; j < 3; ++j) tpart[(int64_t)m * 4 + j] = red[j][0];
}

// dL/dPsi1[n][m] = beta^2 sum_d Y[n][d] C[m][d]  (written over Psi1).
template <typename T>
__global__ void bound_g1_kernel(int64_t N, int M, int64_t D, double beta2, const T *__restrict__ Y,
                                const double *__restrict__ C, T *__restrict__ G1) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= N * M) return;
    int64_t n;
    int m;
    if (i <= 0x7fffffff) {  // 32-bit division where the index fits
        const unsigned u = (unsigned)i, nn = u / (unsigned)M;
        n = nn;
        m = (int)(u - nn * (unsigned)M);
    } else {
        n = i / M;
        m = (int)(i - n * M);
    }
    double s = 0.0;
    for (int64_t d = 0; d < D; ++d) s += (double)Y[n * D + d] * C[(int64_t)m * D + d];
    G1[i] = (T)(beta2 * s);
}

// The bound and dL/dbeta from the reductions (one workgroup, fixed order).
template <typename T>
__global__ __launch_bounds__(256) void bound_scalar_kernel(
    int64_t N, int M, int Mp, int64_t D, int nbk, double beta, double psi0, int64_t rblocks,
    const double *__restrict__ rpart, const double *__restrict__ tpart,
    const double *__restrict__ logdet, const double *__restrict__ Psi, const double *__restrict__ C,
    T *__restrict__ Lout, T *__restrict__ dbeta) {
    __shared__ double red[6][256];
    double yy = 0.0, kl = 0.0, ta = 0.0, tp = 0.0, tk = 0.0, pc = 0.0;
    for (int64_t b = threadIdx.x; b < rblocks; b += 256) {
        yy += rpart[b * 2];
        kl += rpart[b * 2 + 1];
    }
    for (int m = threadIdx.x; m < Mp; m += 256) {
        ta += tpart[(int64_t)m * 4];
        tp += tpart[(int64_t)m * 4 + 1];
        tk += tpart[(int64_t)m * 4 + 2];
    }
    for (int64_t k = threadIdx.x; k < (int64_t)M * D; k += 256) pc += Psi[k] * C[k];
    red[0][threadIdx.x] = yy;
    red[1][threadIdx.x] = kl;
    red[2][threadIdx.x] = ta;
    red[3][threadIdx.x] = tp;
    red[4][threadIdx.x] = tk;
    red[5][threadIdx.x] = pc;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w)
            for (int j = 0; j < 6; ++j) red[j][threadIdx.x] += red[j][threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    yy = red[0][0]; kl = red[1][0]; ta = red[2][0]; tp = red[3][0]; tk = red[4][0]; pc = red[5][0];
    double ldk = 0.0, lda = 0.0;
    for (int K = 0; K < nbk; ++K) {
        ldk += logdet[K];
        lda += logdet[(nbk + 1) + K];
    }
    const bool bad = logdet[nbk] != 0.0 || logdet[(nbk + 1) + nbk] != 0.0;
    const double Nd = (double)N, Dd = (double)D;
    const double F = -0.5 * Nd * Dd * log(2.0 * M_PI) + 0.5 * Nd * Dd * log(beta) + 0.5 * Dd * ldk -
                     0.5 * Dd * lda - 0.5 * beta * yy + 0.5 * beta * beta * pc -
                     0.5 * beta * Dd * psi0 + 0.5 * beta * Dd * tk;
    const double db = 0.5 * Nd * Dd / beta - 0.5 * yy - 0.5 * Dd * ta + beta * pc -
                      0.5 * beta * beta * tp - 0.5 * Dd * psi0 + 0.5 * Dd * tk;
    Lout[0] = bad ? (T)NAN : (T)(F - kl);
    dbeta[0] = bad ? (T)NAN : (T)db;
}

// Chain rule through Kmm = k(Z, Z) + jitter I for dL/dKmm = GK (symmetrised):
// with W = GKs o K0,  dZ[m][q] += -(2 / l^2) sum_m' W (z_mq - z_m'q) (added in
// place), and per row m the partial sums of dl_q (sum_m' W (z_mq - z_m'q)^2 / l^3)
// and of dsigma_f2 (sum_m' W / sigma_f2).
template <typename T>
__global__ __launch_bounds__(64) void bound_kmm_grad_kernel(int M, int Q, int Mp,
                                                            const T *__restrict__ Z, Hyp<T> h,
                                                            const double *__restrict__ K0,
                                                            const double *__restrict__ GK,
                                                            T *__restrict__ dZ, double *__restrict__ kdl,
                                                            double *__restrict__ ksf) {
    const int m = blockIdx.x, q = threadIdx.x;
    double zq = 0.0, gz = 0.0, gl = 0.0, sw = 0.0;
    const double l = q < Q ? (double)h.l[q] : 1.0;
    if (q < Q) zq = (double)Z[(int64_t)m * Q + q];
    // partners in order; loads issued 8 at a time so that they overlap
    for (int mp0 = 0; mp0 < M; mp0 += 8) {
        double w[8], zp[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int mp = mp0 + j;
            const bool in = mp < M;
            w[j] = in ? 0.5 * (GK[(int64_t)m * Mp + mp] + GK[(int64_t)mp * Mp + m]) * K0[(int64_t)m * Mp + mp]
                      : 0.0;
            zp[j] = (in && q < Q) ? (double)Z[(int64_t)mp * Q + q] : 0.0;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (mp0 + j >= M) break;
            sw += w[j];
            if (q < Q) {
                const double d = zq - zp[j];
                gz += w[j] * d;
                gl += w[j] * d * d;
            }
        }
    }
    if (q < Q) {
        dZ[(int64_t)m * Q + q] = (T)((double)dZ[(int64_t)m * Q + q] - 2.0 * gz / (l * l));
        kdl[(int64_t)m * Q + q] = gl / (l * l * l);
    }
    if (q == 0) ksf[m] = sw / (double)h.sf2;
}

// dl[q] += sum_m kdl[m][q], dsigma_f2 += sum_m ksf[m] (fixed order).
template <typename T>
__global__ void bound_kmm_reduce_kernel(int M, int Q, const double *__restrict__ kdl,
                                        const double *__restrict__ ksf, T *__restrict__ dl,
                                        T *__restrict__ dsf2) {
    const int q = threadIdx.x;
    // m in order; loads issued 8 at a time so that they overlap
    if (q <= Q) {
        double s = 0.0;
        int m = 0;
        for (; m + 8 <= M; m += 8) {
            double v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = q < Q ? kdl[(int64_t)(m + j) * Q + q] : ksf[m + j];
#pragma unroll
            for (int j = 0; j < 8; ++j) s += v[j];
        }
        for (; m < M; ++m) s += q < Q ? kdl[(int64_t)m * Q + q] : ksf[m];
        if (q < Q) dl[q] = (T)((double)dl[q] + s);
        else dsf2[0] = (T)((double)dsf2[0] + s);
    }
}

// The KL term's gradient: dmu -= mu, dS -= (1 - 1/S) / 2.
template <typename T>
__global__ void bound_kl_grad_kernel(int64_t NQ, const T *__restrict__ mu, const T *__restrict__ S,
                                     T *__restrict__ dmu, T *__restrict__ dS) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= NQ) return;
    dmu[i] = dmu[i] - mu[i];
    dS[i] = dS[i] - (T)0.5 * ((T)1 - (T)1 / S[i]);
}

}  // namespace

size_t bound_workspace_bytes(const Shape &s, int64_t D, size_t elem, size_t psi_ws) {
    return make_bplan(s, D, elem, psi_ws).total;
}

BoundBufs bound_buffers(const Shape &s, int64_t D, size_t elem, size_t psi_ws) {
    const BPlan p = make_bplan(s, D, elem, psi_ws);
    return BoundBufs{p.off_psi0, p.off_psi1, p.off_psi2, p.off_g2};
}

template <typename T>
hipError_t bound_middle(const Shape &s, int64_t D, const T *mu, const T *S, const T *Z, const T *Y,
                        const Hyp<T> &h, double beta, double jitter, T *L, T *dbeta, void *ws,
                        size_t psi_ws, hipStream_t st) {
    const BPlan p = make_bplan(s, D, sizeof(T), psi_ws);
    const int M = (int)s.M, Q = (int)s.Q, Mp = (int)p.Mp;
    const int64_t mm = p.Mp * p.Mp;
    T *Psi1 = at<T>(ws, p.off_psi1), *Psi2 = at<T>(ws, p.off_psi2), *G2 = at<T>(ws, p.off_g2);
    double *K0 = at<double>(ws, p.off_k0), *gj = at<double>(ws, p.off_gj);
    double *P2 = at<double>(ws, p.off_p2d), *Pm = at<double>(ws, p.off_pm);
    double *Tm = at<double>(ws, p.off_t), *KPK = at<double>(ws, p.off_kpk), *GK = at<double>(ws, p.off_gk);
    double *Psi = at<double>(ws, p.off_psi), *C = at<double>(ws, p.off_c);
    double *ld = at<double>(ws, p.off_ld);

    // Kmm, A; the row reductions; Psi = Psi1^T Y
    {
        TimedScope ts(st, "bound_kmm");
        bound_kmm_kernel<T><<<(unsigned)cdiv(mm, 256), 256, 0, st>>>(M, Q, Mp, Z, h, jitter, beta, Psi2,
                                                                    K0, gj, gj + mm, P2);
    }
    {
        TimedScope ts(st, "bound_rows");
        bound_rows_kernel<T><<<(unsigned)p.rblocks, 256, 0, st>>>(s.N, Q, D, mu, S, Y,
                                                                 at<double>(ws, p.off_rpart));
    }
    {
        TimedScope ts(st, "bound_psiy");
        dim3 g((unsigned)p.ychunks, (unsigned)std::min<int64_t>(cdiv((int64_t)M * D, 256), 16));
        bound_psiy_kernel<T><<<g, 256, 0, st>>>(s.N, M, D, Psi1, Y, at<double>(ws, p.off_ypart));
        bound_psiy_reduce_kernel<<<(unsigned)cdiv(p.Mp * D, 32), 256, 0, st>>>(
            M, Mp, D, p.ychunks, at<double>(ws, p.off_ypart), Psi);
    }
    // Kmm = L_k L_k^T and A = L_a L_a^T (blocked Cholesky, in place), log determinants,
    // the triangular inverses and Kmm^-1 = L_k^-T L_k^-1, A^-1 = L_a^-T L_a^-1
    double *Lf = gj, *Li = gj + 2 * mm, *Kinv = gj + 4 * mm, *Ainv = gj + 5 * mm;
    {
        TimedScope ts(st, "bound_chol");
        double *Dg = at<double>(ws, p.off_dg);
        for (int K = 0; K < p.nbk; ++K) {
            bound_chol_panel_kernel<<<dim3(p.nbk - K, 2), 64, 0, st>>>(Mp, K, Lf, Dg, ld);
            bound_chol_update_kernel<<<dim3(p.nbk, p.nbk, 2), 256, 0, st>>>(Mp, K, Lf, Dg);
        }
        const size_t shb = sizeof(double) * kB * (kB + 1) * (p.nbk + 1);
        hipError_t e = hipFuncSetAttribute((const void *)bound_trinv_kernel,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)shb);
        if (e != hipSuccess) return e;
        bound_trinv_kernel<<<dim3(p.nbk, 2), 256, shb, st>>>(Mp, Lf, Li);
    }
    // C = A^-1 Psi, P = C C^T, Kmm^-1 Psi2 Kmm^-1; dL/dPsi2, dL/dKmm, dL/dPsi1; the scalars
    {
        TimedScope ts(st, "bound_gemm");
        // three stages of two independent products each, one launch per stage
        auto pair = [&](const GemmJob &a, const GemmJob &b) {
            const int64_t gx = std::max(cdiv(a.cols, 16), cdiv(b.cols, 16));
            const int64_t gy = std::max(cdiv(a.rows, 16), cdiv(b.rows, 16));
            bound_gemm2_kernel<<<dim3((unsigned)gx, (unsigned)gy, 2), 256, 0, st>>>(a, b);
        };
        const int64_t P = p.Mp;
        pair(GemmJob{P, P, P, Li, P, true, Li, P, false, 1.0, Kinv, P},                // Kmm^-1
             GemmJob{P, P, P, Li + mm, P, true, Li + mm, P, false, 1.0, Ainv, P});     // A^-1
        pair(GemmJob{P, D, P, Ainv, P, false, Psi, D, false, 1.0, C, D},               // C = A^-1 Psi
             GemmJob{P, P, P, Kinv, P, false, P2, P, false, 1.0, Tm, P});              // Kmm^-1 Psi2
        pair(GemmJob{P, P, D, C, D, false, C, D, true, 1.0, Pm, P},                    // C C^T
             GemmJob{P, P, P, Tm, P, false, Kinv, P, false, 1.0, KPK, P});             // Kmm^-1 Psi2 Kmm^-1
    }
    {
        TimedScope ts(st, "bound_assemble");
        bound_assemble_kernel<T><<<(unsigned)p.Mp, 256, 0, st>>>(M, Mp, D, beta, Kinv, Ainv, Pm, KPK, P2,
                                                                G2, GK, at<double>(ws, p.off_tpart));
        bound_g1_kernel<T><<<(unsigned)cdiv(s.N * M, 256), 256, 0, st>>>(s.N, M, D, beta * beta, Y, C,
                                                                        Psi1);
        bound_scalar_kernel<T><<<1, 256, 0, st>>>(s.N, M, Mp, D, p.nbk, beta, (double)s.N * (double)h.sf2,
                                                 p.rblocks, at<double>(ws, p.off_rpart),
                                                 at<double>(ws, p.off_tpart), ld, Psi, C, L, dbeta);
    }
    return hipGetLastError();
}

template <typename T>
hipError_t bound_tail(const Shape &s, int64_t D, const T *mu, const T *S, const T *Z, const Hyp<T> &h,
                      T *dmu, T *dS, T *dZ, T *dsf2, T *dl, void *ws, size_t psi_ws, hipStream_t st) {
    const BPlan p = make_bplan(s, D, sizeof(T), psi_ws);
    const int M = (int)s.M, Q = (int)s.Q;
    TimedScope ts(st, "bound_kmm_grad");
    bound_kmm_grad_kernel<T><<<(unsigned)M, 64, 0, st>>>(M, Q, (int)p.Mp, Z, h, at<double>(ws, p.off_k0),
                                                        at<double>(ws, p.off_gk), dZ,
                                                        at<double>(ws, p.off_kdl), at<double>(ws, p.off_ksf));
    bound_kmm_reduce_kernel<T><<<1, 128, 0, st>>>(M, Q, at<double>(ws, p.off_kdl), at<double>(ws, p.off_ksf),
                                                 dl, dsf2);
    if (S) bound_kl_grad_kernel<T><<<(unsigned)cdiv(s.N * Q, 256), 256, 0, st>>>(s.N * Q, mu, S, dmu, dS);
    return hipGetLastError();
}

#define GPPS_BOUND_INST(T)                                                                            \
    template hipError_t bound_middle<T>(const Shape &, int64_t, const T *, const T *, const T *,       \
                                        const T *, const Hyp<T> &, double, double, T *, T *, void *,   \
                                        size_t, hipStream_t);                                         \
    template hipError_t bound_tail<T>(const Shape &, int64_t, const T *, const T *, const T *,         \
                                      const Hyp<T> &, T *, T *, T *, T *, T *, void *, size_t,         \
                                      hipStream_t);
GPPS_BOUND_INST(float)
GPPS_BOUND_INST(double)
#undef GPPS_BOUND_INST

}  // namespace gpps
