// Known inputs (S = 0): the sparse GP regression case of section 2, eq. (boundF).
//
// With every variance zero the expectations of eq. (4) collapse to the plain
// kernel quantities: psi0 = N sf2, Psi1 = Kfu with Kfu[n, m] = k(x_n, z_m), and
// Psi2 = Kfu^T Kfu.  Psi2 is then a dense contraction over the datapoints, so
// unlike the S > 0 path (where an exp sits between the per-datapoint Gram and
// the sum over n) the work here is GEMM-shaped and runs on the matrix cores:
//
//   stats:  Kfu on the vector ALU (Q differences and one exp per entry), then
//           Psi2 = Kfu^T Kfu as a split-N symmetric rank-k update (upper tiles
//           only), one partial tile set per row chunk, chunks summed in a
//           fixed order;
//   grads:  dL/dKfu = G1 + 2 Kfu G2s (G2s the symmetric part of dL/dPsi2) as a
//           GEMM over the inducing inputs, E = dL/dKfu o Kfu, and the chain
//           rule through the kernel.  With xs = (x - c) / l and zs = (z - c) / l
//           per dimension (c the mean of Z; the kernel depends on differences
//           only, and centring keeps the expanded sums below well scaled):
//             r_n = sum_m E,  U_nq = sum_m E zs_mq,  c_m = sum_n E,  V_mq = sum_n E xs_nq
//             dx_nq = -(xs_nq r_n - U_nq) / l_q
//             dz_mq = (V_mq - zs_mq c_m) / l_q
//             dl_q  = (sum_n (r_n xs_nq^2 - 2 xs_nq U_nq) + sum_m c_m zs_mq^2) / l_q
//             dsf2  = sum E / sf2 + N dL/dpsi0.
//
// Matrix-core products: fp32 v_mfma_f32_32x32x2f32 (fp32 products, fp32
// accumulation), fp64 v_mfma_f64_16x16x4f64.  Every tiled kernel works on
// 64 x 64 output blocks, one wave per block.  No atomics; results are bitwise
// deterministic for a fixed shape.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace gpps {
namespace {

constexpr int kEdge = 64;              // output block edge of every tiled kernel
constexpr int kUnroll = 4;             // matrix-core k-steps per batch of loads
constexpr float kLog2eF = 1.4426950408889634f;

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return cdiv(a, b) * b; }

template <typename T>
T *at(void *ws, size_t off) { return reinterpret_cast<T *>(static_cast<char *>(ws) + off); }

// One matrix-core product per element type.  Lane l supplies A[l % TILE][l / TILE]
// and B[l / TILE][l % TILE]; accumulator element v of lane l is C[row(v, l)][l % TILE].
template <typename T>
struct Mma;
template <>
struct Mma<float> {
    static constexpr int TILE = 32, KS = 2, NACC = 16;
    typedef float acc_t __attribute__((ext_vector_type(16)));
    __device__ static acc_t mma(float a, float b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
    __device__ static int row(int v, int lane) { return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3); }
};
template <>
struct Mma<double> {
    static constexpr int TILE = 16, KS = 4, NACC = 4;
    typedef double acc_t __attribute__((ext_vector_type(4)));
    __device__ static acc_t mma(double a, double b, acc_t c) {
        return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
    }
    // rows interleave over the lane groups (measured: register v of lane group
    // g holds row 4 v + g), unlike the 4 consecutive rows of the fp32 16 x 16 forms
    __device__ static int row(int v, int lane) { return 4 * v + (lane >> 4); }
};

// sf2 exp(-s / 2) from the prefactor pre(h) and the squared scaled distance s.
__device__ inline float kpre(const Hyp<float> &h) { return h.log_sf2 * kLog2eF; }
__device__ inline double kpre(const Hyp<double> &h) { return h.log_sf2; }
__device__ inline float kval(float pre, float s) {
    return __builtin_amdgcn_exp2f(fmaf(-0.5f * kLog2eF, s, pre));
}
__device__ inline double kval(double pre, double s) { return exp(pre - 0.5 * s); }

// ---------------------------------------------------------------- launch plan
struct KPlan {
    int tile;                   // matrix-core tile edge (32 fp32, 16 fp64)
    int64_t nb, ntp, ntu, nbp;  // 64-blocks per edge, tiles per edge, upper tiles, upper block pairs
    int64_t chunks, rows;       // Psi2 row chunks and rows per chunk
    int64_t grid_syrk;          // Psi2 workgroups (XCD-rounded)
    int64_t rblocks;            // row-kernel blocks (256 datapoints each)
    int64_t cchunks, crows;     // column-kernel row chunks and rows per chunk
    size_t off_cz, off_xs, off_zs, off_k, off_e, off_g2s, off_part, off_rowp, off_colp, off_vc;
    size_t total;
};

KPlan make_kplan(const Shape &s, size_t elem) {
    KPlan p{};
    p.tile = elem == 4 ? 32 : 16;
    p.nb = cdiv(s.M, kEdge);
    p.ntp = p.nb * (kEdge / p.tile);
    p.ntu = p.ntp * (p.ntp + 1) / 2;
    p.nbp = p.nb * (p.nb + 1) / 2;
    // about two waves per SIMD for the rank-k update; each chunk a multiple of
    // the unrolled k-step so that only the last one is ragged
    p.chunks = std::max<int64_t>(1, std::min<int64_t>(cdiv(s.N, 256), 2048 / p.nbp));
    p.rows = round_up(cdiv(s.N, p.chunks), 16);
    p.chunks = cdiv(s.N, p.rows);
    p.grid_syrk = round_up(p.chunks, 8) * p.nbp;
    p.rblocks = cdiv(s.N, 256);
    p.cchunks = std::max<int64_t>(1, std::min<int64_t>(cdiv(s.N, kEdge), std::max<int64_t>(1, 2048 / p.nb)));
    p.crows = round_up(cdiv(s.N, p.cchunks), kEdge);
    p.cchunks = cdiv(s.N, p.crows);
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
    p.off_cz = take(elem * s.Q);
    p.off_xs = take(elem * s.N * s.Q);
    p.off_zs = take(elem * s.M * s.Q);
    p.off_k = take(elem * s.N * s.M);
    p.off_e = take(elem * s.N * s.M);
    p.off_g2s = take(elem * s.M * s.M);
    p.off_part = take(elem * p.chunks * p.ntu * p.tile * p.tile);
    p.off_rowp = take(elem * p.rblocks * (s.Q + 1));
    p.off_colp = take(elem * p.cchunks * s.M * (s.Q + 1));
    p.off_vc = take(elem * s.M * (s.Q + 1));
    p.total = o;
    return p;
}

// ---------------------------------------------------------------- centring
// cz[q] = mean_m z_mq, zs = (Z - cz) / l.  One workgroup: G = 256 / Q groups of
// Q threads sum rows m = g, g + G, ... (coalesced), then the G partial sums of
// each dimension are added in group order.
template <typename T>
__global__ __launch_bounds__(256) void known_centre_kernel(int M, int Q, const T *__restrict__ Z,
                                                           Hyp<T> h, T *__restrict__ cz,
                                                           T *__restrict__ zs) {
    __shared__ T part[256];
    __shared__ T c[GPPS_MAX_Q];
    const int t = threadIdx.x, G = 256 / Q;
    if (t < G * Q) {
        const int g = t / Q, q = t - g * Q;
        T s = 0;
        for (int m = g; m < M; m += G) s += Z[(int64_t)m * Q + q];
        part[t] = s;
    }
    __syncthreads();
    if (t < Q) {
        T s = 0;
        for (int g = 0; g < G; ++g) s += part[g * Q + t];
        c[t] = s / T(M);
        cz[t] = c[t];
    }
    __syncthreads();
    for (int i = t; i < M * Q; i += 256) zs[i] = (Z[i] - c[i % Q]) / h.l[i % Q];
}

// ---------------------------------------------------------------- Kfu
// One 64 x 64 block of Kfu per workgroup.  TRANS = false writes out[n][m]
// (N x M, the Psi1 layout), TRANS = true writes out[m][n] (M x N, the layout
// the gradient GEMM streams).  Grid: (row blocks, column blocks); the
// workgroups of the first column block also write xs.  Dynamic LDS: 2 * 64 * Q elements.
template <typename T, bool TRANS>
__global__ __launch_bounds__(256) void known_kfu_kernel(int64_t N, int M, int Q,
                                                        const T *__restrict__ X,
                                                        const T *__restrict__ cz,
                                                        const T *__restrict__ zs, Hyp<T> h,
                                                        T *__restrict__ out, T *__restrict__ xs) {
    extern __shared__ double known_smem[];
    T *sx = reinterpret_cast<T *>(known_smem);  // [q][64] scaled rows
    T *sz = sx + Q * kEdge;                     // [q][64] scaled inducing inputs
    const int tid = threadIdx.x;
    const int64_t n0 = (int64_t)blockIdx.x * kEdge;
    const int m0 = blockIdx.y * kEdge;
    for (int i = tid; i < kEdge * Q; i += 256) {
        const int r = i / Q, q = i - r * Q;
        const int64_t n = n0 + r;
        T v = 0;
        if (n < N) {
            v = (X[n * Q + q] - cz[q]) / h.l[q];
            if (blockIdx.y == 0) xs[n * Q + q] = v;
        }
        sx[q * kEdge + r] = v;
        const int m = m0 + r;
        sz[q * kEdge + r] = m < M ? zs[(int64_t)m * Q + q] : T(0);
    }
    __syncthreads();
    const T pre = kpre(h);
    T s[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) s[j] = 0;
    if (!TRANS) {
        const int c = tid & 63, rg = tid >> 6;
        for (int q = 0; q < Q; ++q) {
            const T zc = sz[q * kEdge + c];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const T d = sx[q * kEdge + rg + 4 * j] - zc;
                s[j] = fma(d, d, s[j]);
            }
        }
        const int m = m0 + c;
        if (m < M) {
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int64_t n = n0 + rg + 4 * j;
                if (n < N) out[n * M + m] = kval(pre, s[j]);
            }
        }
    } else {
        const int r = tid & 63, cg = tid >> 6;
        for (int q = 0; q < Q; ++q) {
            const T xr = sx[q * kEdge + r];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const T d = xr - sz[q * kEdge + cg + 4 * j];
                s[j] = fma(d, d, s[j]);
            }
        }
        const int64_t n = n0 + r;
        if (n < N) {
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int m = m0 + cg + 4 * j;
                if (m < M) out[(int64_t)m * N + n] = kval(pre, s[j]);
            }
        }
    }
}

// Upper block pair index -> (I, J), I <= J, over nb blocks per edge.
__device__ inline void block_pair(int64_t bp, int64_t nb, int &I, int &J) {
    int64_t i = 0;
    while (bp >= nb - i) { bp -= nb - i; ++i; }
    I = (int)i;
    J = (int)(i + bp);
}

// ---------------------------------------------------------------- Psi2 = Kfu^T Kfu
// One wave per (row chunk, upper 64-block pair (I, J)): the partial sums of the
// chunk's rows for every upper tile of the block pair, on the matrix cores.
// Workgroups are dispatched round-robin over the 8 XCDs, so the block pairs of
// one chunk are given ids that land on the same XCD and share its L2.
template <typename T>
__global__ __launch_bounds__(64) void known_syrk_kernel(int64_t N, int M, int64_t rows,
                                                        int64_t chunks, int64_t nb, int64_t ntp,
                                                        int64_t ntu, const T *__restrict__ K,
                                                        T *__restrict__ part) {
    using A = Mma<T>;
    constexpr int TILE = A::TILE, KS = A::KS, BT = kEdge / TILE;
    const int64_t nbp = nb * (nb + 1) / 2;
    const int64_t id = blockIdx.x, slot = id >> 3;
    const int64_t chunk = (slot / nbp) * 8 + (id & 7);
    if (chunk >= chunks) return;
    int I, J;
    block_pair(slot % nbp, nb, I, J);
    const int lane = threadIdx.x, li = lane % TILE, lk = lane / TILE;
    const int64_t r0 = chunk * rows, r1 = min(N, r0 + rows);
    typename A::acc_t acc[BT][BT];
#pragma unroll
    for (int ti = 0; ti < BT; ++ti)
#pragma unroll
        for (int tj = 0; tj < BT; ++tj)
#pragma unroll
            for (int v = 0; v < A::NACC; ++v) acc[ti][tj][v] = 0;
    const int ci = I * kEdge + li, cj = J * kEdge + li;
    for (int64_t n = r0; n < r1; n += KS * kUnroll) {
        T a[kUnroll][BT], b[kUnroll][BT];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t row = n + u * KS + lk;
            const bool ok = row < r1;
#pragma unroll
            for (int t = 0; t < BT; ++t) {
                const int mi = ci + t * TILE, mj = cj + t * TILE;
                a[u][t] = (ok && mi < M) ? K[row * M + mi] : T(0);
                b[u][t] = (ok && mj < M) ? K[row * M + mj] : T(0);
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
            for (int ti = 0; ti < BT; ++ti)
#pragma unroll
                for (int tj = 0; tj < BT; ++tj)
                    if (I < J || ti <= tj) acc[ti][tj] = A::mma(a[u][ti], b[u][tj], acc[ti][tj]);
    }
#pragma unroll
    for (int ti = 0; ti < BT; ++ti)
#pragma unroll
        for (int tj = 0; tj < BT; ++tj) {
            if (!(I < J || ti <= tj)) continue;
            const int64_t gi = (int64_t)I * BT + ti, gj = (int64_t)J * BT + tj;
            const int64_t p = gi * ntp - gi * (gi - 1) / 2 + (gj - gi);
            T *dst = part + (chunk * ntu + p) * (TILE * TILE);
#pragma unroll
            for (int v = 0; v < A::NACC; ++v) dst[A::row(v, lane) * TILE + li] = acc[ti][tj][v];
        }
}

// Fixed-order sum of the chunk partials of every upper tile; writes both
// triangles of Psi2 (bitwise equal) and psi0.
template <typename T>
__global__ __launch_bounds__(256) void known_syrk_reduce_kernel(int64_t N, int M, int64_t ntp,
                                                                int64_t ntu, int64_t chunks,
                                                                const T *__restrict__ part,
                                                                Hyp<T> h, T *__restrict__ psi0,
                                                                T *__restrict__ Psi2,
                                                                int accumulate) {
    constexpr int TILE = Mma<T>::TILE, TT = TILE * TILE;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx == 0) psi0[0] = (accumulate ? psi0[0] : T(0)) + T(N) * h.sf2;
    if (idx >= ntu * TT) return;
    const int64_t p = idx / TT;
    const int e = (int)(idx - p * TT);
    int gi, gj;
    block_pair(p, ntp, gi, gj);
    const int m = gi * TILE + e / TILE, mp = gj * TILE + e % TILE;
    if (m >= M || mp >= M || m > mp) return;
    // chunk order; loads issued 16 at a time so that they overlap
    const T *src = part + p * TT + e;
    const int64_t stride = ntu * TT;
    T s = 0;
    int64_t c = 0;
    for (; c + 16 <= chunks; c += 16) {
        T v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = src[(c + j) * stride];
#pragma unroll
        for (int j = 0; j < 16; ++j) s += v[j];
    }
    for (; c < chunks; ++c) s += src[c * stride];
    const T v = (accumulate ? Psi2[(int64_t)m * M + mp] : T(0)) + s;
    Psi2[(int64_t)m * M + mp] = v;
    Psi2[(int64_t)mp * M + m] = v;
}

// ---------------------------------------------------------------- gradients
template <typename T>
__global__ void known_sym_kernel(int M, const T *__restrict__ G2, T *__restrict__ G2s) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)M * M) return;
    const int m = (int)(i / M), mp = (int)(i - (int64_t)m * M);
    G2s[i] = T(0.5) * (G2[(int64_t)m * M + mp] + G2[(int64_t)mp * M + m]);
}

// E^T[m][n] = (G1[n][m] + 2 sum_k G2s[m][k] Kt[k][n]) Kt[m][n], one wave per
// 64 x 64 block (m, n) on the matrix cores.  G2s is symmetric, so its A operand
// G2s[m][k] is read as G2s[k][m], a contiguous row.  Same XCD grouping as the
// rank-k update: the m-blocks of one column block n share an XCD.
template <typename T, bool HAS_G2>
__global__ __launch_bounds__(64) void known_dkfu_kernel(int64_t N, int M, int64_t nblk, int64_t mb,
                                                        const T *__restrict__ Kt,
                                                        const T *__restrict__ G1,
                                                        const T *__restrict__ G2s,
                                                        T *__restrict__ Et) {
    using A = Mma<T>;
    constexpr int TILE = A::TILE, KS = A::KS, BT = kEdge / TILE;
    const int64_t id = blockIdx.x, slot = id >> 3;
    const int64_t nbi = (slot / mb) * 8 + (id & 7);
    if (nbi >= nblk) return;
    const int64_t n0 = nbi * kEdge;
    const int m0 = (int)(slot % mb) * kEdge;
    const int lane = threadIdx.x, li = lane % TILE, lk = lane / TILE;
    typename A::acc_t acc[BT][BT];
#pragma unroll
    for (int ti = 0; ti < BT; ++ti)
#pragma unroll
        for (int tj = 0; tj < BT; ++tj)
#pragma unroll
            for (int v = 0; v < A::NACC; ++v) acc[ti][tj][v] = 0;
    if (HAS_G2) {
        for (int k = 0; k < M; k += KS * kUnroll) {
            T a[kUnroll][BT], b[kUnroll][BT];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int kr = k + u * KS + lk;
                const bool ok = kr < M;
#pragma unroll
                for (int t = 0; t < BT; ++t) {
                    const int m = m0 + t * TILE + li;
                    const int64_t n = n0 + t * TILE + li;
                    a[u][t] = (ok && m < M) ? G2s[(int64_t)kr * M + m] : T(0);
                    b[u][t] = (ok && n < N) ? Kt[(int64_t)kr * N + n] : T(0);
                }
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                for (int tm = 0; tm < BT; ++tm)
#pragma unroll
                    for (int tn = 0; tn < BT; ++tn)
                        acc[tm][tn] = A::mma(a[u][tm], b[u][tn], acc[tm][tn]);
        }
    }
#pragma unroll
    for (int tm = 0; tm < BT; ++tm)
#pragma unroll
        for (int tn = 0; tn < BT; ++tn)
#pragma unroll
            for (int v = 0; v < A::NACC; ++v) {
                const int m = m0 + tm * TILE + A::row(v, lane);
                const int64_t n = n0 + tn * TILE + li;
                if (m < M && n < N) {
                    const T g1 = G1 ? G1[n * M + m] : T(0);
                    const int64_t o = (int64_t)m * N + n;
                    Et[o] = (g1 + T(2) * acc[tm][tn][v]) * Kt[o];
                }
            }
}

// Fixed-order sum over the 256 threads of a workgroup (wave butterflies, then
// the four wave sums in order); the result is valid in thread 0.
template <typename T>
__device__ inline T block_sum(T v, T *red4) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red4[threadIdx.x >> 6] = v;
    __syncthreads();
    return ((red4[0] + red4[1]) + red4[2]) + red4[3];
}

// 16-byte vectors for LDS reads of the scaled-input tables.
template <typename T>
struct Vec;
template <>
struct Vec<float> {
    typedef float t __attribute__((ext_vector_type(4)));
    static constexpr int W = 4;
};
template <>
struct Vec<double> {
    typedef double t __attribute__((ext_vector_type(2)));
    static constexpr int W = 2;
};

// acc[0..QM) += e * row[0..QM) for an LDS row that is zero beyond Q (no
// per-dimension guard: a runtime bound inside the unrolled loop makes the
// compiler shuffle the accumulators).
template <typename T, int QM>
__device__ inline void axpy_row(T e, const T *row, T *acc) {
    using V = typename Vec<T>::t;
    constexpr int W = Vec<T>::W;
    const V *r = reinterpret_cast<const V *>(row);
#pragma unroll
    for (int v = 0; v < QM / W; ++v) {
        const V z = r[v];
#pragma unroll
        for (int w = 0; w < W; ++w) acc[v * W + w] = fma(e, z[w], acc[v * W + w]);
    }
}

// One thread per datapoint: r_n and U_n (sums over m of E^T[m][n] and of
// E^T[m][n] zs_m; coalesced over n, loads issued 16 at a time), dx_n, and
// per-block partials of sum_n (r xs^2 - 2 xs U) (dl) and sum_n r (dsf2).
template <typename T, int QM>
__global__ __launch_bounds__(256) void known_rows_kernel(int64_t N, int M, int Q,
                                                         const T *__restrict__ Et,
                                                         const T *__restrict__ xs,
                                                         const T *__restrict__ zs, Hyp<T> h,
                                                         T *__restrict__ dX,
                                                         T *__restrict__ rowpart) {
    __shared__ __align__(16) T sz[kEdge][QM];  // zero beyond Q and beyond the block's rows
    __shared__ T red4[4];
    const int tid = threadIdx.x;
    const int64_t n = (int64_t)blockIdx.x * 256 + tid;
    const bool valid = n < N;
    T r = 0, U[QM];
#pragma unroll
    for (int q = 0; q < QM; ++q) U[q] = 0;
    for (int mb = 0; mb < M; mb += kEdge) {
        const int cnt = min(kEdge, M - mb);
        __syncthreads();
        for (int i = tid; i < kEdge * QM; i += 256) {
            const int c = i / QM, q = i - c * QM;
            sz[c][q] = (c < cnt && q < Q) ? zs[(int64_t)(mb + c) * Q + q] : T(0);
        }
        __syncthreads();
        if (valid) {
            for (int c0 = 0; c0 < cnt; c0 += 16) {
                T e[16];
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    e[j] = c0 + j < cnt ? Et[(int64_t)(mb + c0 + j) * N + n] : T(0);
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    r += e[j];
                    axpy_row<T, QM>(e[j], &sz[c0 + j][0], U);
                }
            }
        }
    }
#pragma unroll
    for (int q = 0; q <= QM; ++q) {
        if (q < Q || q == QM) {
            T v = 0;
            if (q < Q) {
                const T x = valid ? xs[n * Q + q] : T(0);
                if (valid) dX[n * Q + q] = -(x * r - U[q]) / h.l[q];
                v = valid ? r * x * x - T(2) * x * U[q] : T(0);
            } else {
                v = valid ? r : T(0);
            }
            const T s = block_sum(v, red4);
            if (tid == 0) rowpart[blockIdx.x * (Q + 1) + (q < Q ? q : Q)] = s;
        }
    }
}

// One workgroup per (64 inducing inputs, row chunk): c_m and V_m over the
// chunk from E^T tiles staged in LDS -> colpart[chunk][m][Q + 1] (V, then c).
template <typename T, int QM>
__global__ __launch_bounds__(256) void known_cols_kernel(int64_t N, int M, int Q, int64_t rows,
                                                         const T *__restrict__ Et,
                                                         const T *__restrict__ xs,
                                                         T *__restrict__ colpart) {
    __shared__ T se[kEdge][kEdge + 1];         // E^T tile [m][n], zero outside
    __shared__ __align__(16) T sx[kEdge][QM];  // xs rows of the tile, zero outside
    __shared__ T red[4][kEdge];
    const int tid = threadIdx.x;
    const int m0 = blockIdx.x * kEdge;
    const int64_t r0 = (int64_t)blockIdx.y * rows, r1 = min(N, r0 + rows);
    const int mr = tid & 63, quarter = tid >> 6;
    T c = 0, V[QM];
#pragma unroll
    for (int q = 0; q < QM; ++q) V[q] = 0;
    for (int64_t nb = r0; nb < r1; nb += kEdge) {
        const int cnt = (int)min<int64_t>(kEdge, r1 - nb);
        __syncthreads();
        for (int i = tid; i < kEdge * kEdge; i += 256) {
            const int row = i >> 6, col = i & 63;
            const int m = m0 + row;
            se[row][col] = (m < M && col < cnt) ? Et[(int64_t)m * N + nb + col] : T(0);
        }
        for (int i = tid; i < kEdge * QM; i += 256) {
            const int rr = i / QM, q = i - rr * QM;
            sx[rr][q] = (rr < cnt && q < Q) ? xs[(nb + rr) * Q + q] : T(0);
        }
        __syncthreads();
#pragma unroll 4
        for (int j = 0; j < 16; ++j) {
            const int col = quarter * 16 + j;
            const T e = se[mr][col];
            c += e;
            axpy_row<T, QM>(e, &sx[col][0], V);
        }
    }
    const int m = m0 + mr;
#pragma unroll
    for (int q = 0; q <= QM; ++q) {
        if (q < Q || q == QM) {
            __syncthreads();
            red[quarter][mr] = q < Q ? V[q] : c;
            __syncthreads();
            if (quarter == 0 && m < M)
                colpart[((int64_t)blockIdx.y * M + m) * (Q + 1) + (q < Q ? q : Q)] =
                    ((red[0][mr] + red[1][mr]) + red[2][mr]) + red[3][mr];
        }
    }
}

// One workgroup per inducing input m: Vc[m][k] = sum over the column chunks of
// colpart[chunk][m][k], k <= Q.  G = 256 / (Q + 1) groups of Q + 1 threads take
// chunks g, g + G, ... (coalesced over k); the G partials are added in order.
template <typename T>
__global__ __launch_bounds__(256) void known_col_reduce_kernel(int M, int Q, int64_t cchunks,
                                                               const T *__restrict__ colpart,
                                                               T *__restrict__ Vc) {
    __shared__ T part[256];
    const int t = threadIdx.x, Q1 = Q + 1, G = 256 / Q1;
    const int64_t m = blockIdx.x;
    if (t < G * Q1) {
        const int g = t / Q1, k = t - g * Q1;
        T s = 0;
        for (int64_t c = g; c < cchunks; c += G) s += colpart[(c * M + m) * Q1 + k];
        part[t] = s;
    }
    __syncthreads();
    if (t < Q1) {
        T s = 0;
        for (int g = 0; g < G; ++g) s += part[g * Q1 + t];
        Vc[m * Q1 + t] = s;
    }
}

// dZ[m][q] = (V_mq - zs_mq c_m) / l_q elementwise (blocks below zblocks), then
// one workgroup per dl_q and one for dsf2, each a fixed-order block sum.
template <typename T>
__global__ __launch_bounds__(256) void known_grad_final_kernel(
    int64_t N, int M, int Q, int64_t zblocks, int64_t rblocks, const T *__restrict__ Vc,
    const T *__restrict__ rowpart, const T *__restrict__ zs, Hyp<T> h, T dL_dpsi0,
    T *__restrict__ dZ, T *__restrict__ dsf2, T *__restrict__ dl, int accumulate) {
    __shared__ T red4[4];
    const int64_t Q1 = Q + 1;
    if ((int64_t)blockIdx.x < zblocks) {
        const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
        if (i >= (int64_t)M * Q) return;
        const int64_t m = i / Q, q = i - m * Q;
        const T v = (Vc[m * Q1 + q] - zs[i] * Vc[m * Q1 + Q]) / h.l[q];
        dZ[i] = (accumulate ? dZ[i] : T(0)) + v;
        return;
    }
    const int k = (int)(blockIdx.x - zblocks);  // k < Q: dl_k; k == Q: dsf2
    T s = 0;
    for (int64_t b = threadIdx.x; b < rblocks; b += 256) s += rowpart[b * Q1 + k];
    if (k < Q)
        for (int m = threadIdx.x; m < M; m += 256) {
            const T z = zs[(int64_t)m * Q + k];
            s += Vc[(int64_t)m * Q1 + Q] * z * z;
        }
    s = block_sum(s, red4);
    if (threadIdx.x == 0) {
        if (k < Q) dl[k] = (accumulate ? dl[k] : T(0)) + s / h.l[k];
        else dsf2[0] = (accumulate ? dsf2[0] : T(0)) + (s / h.sf2 + dL_dpsi0 * T(N));
    }
}

template <typename T>
void launch_centre_kfu(const Shape &s, const KPlan &p, const T *X, const T *Z, const Hyp<T> &h,
                       bool trans, T *out, void *ws, hipStream_t st) {
    T *cz = at<T>(ws, p.off_cz), *zs = at<T>(ws, p.off_zs), *xs = at<T>(ws, p.off_xs);
    {
        TimedScope ts(st, "known_centre");
        known_centre_kernel<T><<<1, 256, 0, st>>>((int)s.M, (int)s.Q, Z, h, cz, zs);
    }
    dim3 grid((unsigned)cdiv(s.N, kEdge), (unsigned)cdiv(s.M, kEdge));
    const size_t lds = 2 * kEdge * s.Q * sizeof(T);
    TimedScope ts(st, "known_kfu");
    if (trans)
        known_kfu_kernel<T, true><<<grid, 256, lds, st>>>(s.N, (int)s.M, (int)s.Q, X, cz, zs, h, out, xs);
    else
        known_kfu_kernel<T, false><<<grid, 256, lds, st>>>(s.N, (int)s.M, (int)s.Q, X, cz, zs, h, out, xs);
}

template <typename T, int QM>
void launch_chain(const Shape &s, const KPlan &p, const T *Et, const Hyp<T> &h, T *dX, void *ws,
                  hipStream_t st) {
    const T *xs = at<T>(ws, p.off_xs), *zs = at<T>(ws, p.off_zs);
    {
        TimedScope ts(st, "known_rows");
        known_rows_kernel<T, QM><<<(unsigned)p.rblocks, 256, 0, st>>>(
            s.N, (int)s.M, (int)s.Q, Et, xs, zs, h, dX, at<T>(ws, p.off_rowp));
    }
    TimedScope ts(st, "known_cols");
    known_cols_kernel<T, QM><<<dim3((unsigned)p.nb, (unsigned)p.cchunks), 256, 0, st>>>(
        s.N, (int)s.M, (int)s.Q, p.crows, Et, xs, at<T>(ws, p.off_colp));
}

}  // namespace

size_t known_workspace_bytes(const Shape &s, size_t elem) { return make_kplan(s, elem).total; }

template <typename T>
hipError_t known_psi_stats(const Shape &s, const T *X, const T *Z, const Hyp<T> &h, T *psi0,
                           T *Psi1, T *Psi2, int accumulate, void *ws, hipStream_t st) {
    const KPlan p = make_kplan(s, sizeof(T));
    T *K = Psi1 ? Psi1 : at<T>(ws, p.off_k);
    launch_centre_kfu<T>(s, p, X, Z, h, false, K, ws, st);
    T *part = at<T>(ws, p.off_part);
    {
        TimedScope ts(st, "known_syrk");
        known_syrk_kernel<T><<<(unsigned)p.grid_syrk, 64, 0, st>>>(s.N, (int)s.M, p.rows, p.chunks,
                                                                  p.nb, p.ntp, p.ntu, K, part);
    }
    const int64_t elems = p.ntu * p.tile * p.tile;
    TimedScope ts(st, "known_syrk_reduce");
    known_syrk_reduce_kernel<T><<<(unsigned)cdiv(elems, 256), 256, 0, st>>>(
        s.N, (int)s.M, p.ntp, p.ntu, p.chunks, part, h, psi0, Psi2, accumulate);
    return hipGetLastError();
}

template <typename T>
hipError_t known_psi_grads(const Shape &s, const T *X, const T *Z, const Hyp<T> &h, T dL_dpsi0,
                           const T *G1, const T *G2, T *dX, T *dZ, T *dsf2, T *dl, int accumulate,
                           void *ws, hipStream_t st) {
    const KPlan p = make_kplan(s, sizeof(T));
    T *Kt = at<T>(ws, p.off_k), *Et = at<T>(ws, p.off_e);
    launch_centre_kfu<T>(s, p, X, Z, h, true, Kt, ws, st);
    const int64_t nblk = cdiv(s.N, kEdge), mb = p.nb;
    const unsigned grid = (unsigned)(round_up(nblk, 8) * mb);
    if (G2) {
        T *G2s = at<T>(ws, p.off_g2s);
        {
            TimedScope ts(st, "known_sym");
            known_sym_kernel<T><<<(unsigned)cdiv(s.M * s.M, 256), 256, 0, st>>>((int)s.M, G2, G2s);
        }
        TimedScope ts(st, "known_dkfu");
        known_dkfu_kernel<T, true><<<grid, 64, 0, st>>>(s.N, (int)s.M, nblk, mb, Kt, G1, G2s, Et);
    } else {
        TimedScope ts(st, "known_dkfu");
        known_dkfu_kernel<T, false><<<grid, 64, 0, st>>>(s.N, (int)s.M, nblk, mb, Kt, G1, nullptr, Et);
    }
    if (s.Q <= 4) launch_chain<T, 4>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 8) launch_chain<T, 8>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 16) launch_chain<T, 16>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 32) launch_chain<T, 32>(s, p, Et, h, dX, ws, st);
    else launch_chain<T, 64>(s, p, Et, h, dX, ws, st);
    TimedScope ts(st, "known_grad_reduce");
    T *Vc = at<T>(ws, p.off_vc);
    known_col_reduce_kernel<T><<<(unsigned)s.M, 256, 0, st>>>((int)s.M, (int)s.Q, p.cchunks,
                                                             at<T>(ws, p.off_colp), Vc);
    const int64_t zblocks = cdiv(s.M * s.Q, 256);
    known_grad_final_kernel<T><<<(unsigned)(zblocks + s.Q + 1), 256, 0, st>>>(
        s.N, (int)s.M, (int)s.Q, zblocks, p.rblocks, Vc, at<T>(ws, p.off_rowp), at<T>(ws, p.off_zs),
        h, dL_dpsi0, dZ, dsf2, dl, accumulate);
    return hipGetLastError();
}

#define GPPS_KNOWN_INST(T)                                                                          \
    template hipError_t known_psi_stats<T>(const Shape &, const T *, const T *, const Hyp<T> &, T *, \
                                           T *, T *, int, void *, hipStream_t);                      \
    template hipError_t known_psi_grads<T>(const Shape &, const T *, const T *, const Hyp<T> &, T,  \
                                           const T *, const T *, T *, T *, T *, T *, int, void *,   \
                                           hipStream_t);
GPPS_KNOWN_INST(float)
GPPS_KNOWN_INST(double)
#undef GPPS_KNOWN_INST

}  // namespace gpps
