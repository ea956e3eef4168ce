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
//           only) and d_nmq = xs_nq - zs_mq:
//             dx_nq = -sum_m E d / l_q
//             dz_mq =  sum_n E d / l_q
//             dl_q  =  sum_nm E d^2 / l_q
//             dsf2  =  sum E / sf2 + N dL/dpsi0.
//
// Matrix-core products: fp32 v_mfma_f32_32x32x2f32 (fp32 products, fp32
// accumulation), fp64 v_mfma_f64_16x16x4f64, on 128 x 128 blocks staged
// through LDS (block_product).  No atomics; results are bitwise deterministic
// for a fixed shape.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace gpps {
namespace {

constexpr int kEdge = 64;              // block edge of the Kfu and chain-rule kernels
constexpr int kBlk = 128;              // block edge of the matrix-core products
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

// 16-byte vectors (global loads into LDS, LDS row reads).
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
    int64_t nb;                 // 64-blocks of inducing inputs (column kernel)
    int64_t nb2, ntp, ntu, nbp; // kBlk-blocks per edge, tiles per edge, upper tiles, upper block pairs
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
    p.nb2 = cdiv(s.M, kBlk);
    p.ntp = p.nb2 * (kBlk / p.tile);
    p.ntu = p.ntp * (p.ntp + 1) / 2;
    p.nbp = p.nb2 * (p.nb2 + 1) / 2;
    // at most one round of two workgroups per CU for the rank-k update (the
    // chunk count a multiple of the 8 XCDs, so the XCD-rounded grid stays
    // within it); each chunk a multiple of the LDS slab so that only the last
    // one is ragged
    const int64_t bk = elem == 4 ? 32 : 16;
    const int64_t fit = 512 / p.nbp >= 8 ? 512 / p.nbp / 8 * 8 : std::max<int64_t>(1, 512 / p.nbp);
    p.chunks = std::max<int64_t>(1, std::min<int64_t>(cdiv(s.N, 4 * bk), fit));
    p.rows = round_up(cdiv(s.N, p.chunks), bk);
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
    p.off_rowp = take(elem * p.rblocks);
    p.off_colp = take(elem * p.cchunks * s.M * 2 * s.Q);
    p.off_vc = take(elem * s.M * 2 * s.Q);
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
    using VT = typename Vec<T>::t;
    constexpr int W = Vec<T>::W;
    T s[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) s[j] = 0;
    // each thread owns 16 consecutive rows (columns) of the block, read from
    // the LDS table as 16-byte vectors
    if (!TRANS) {
        const int c = tid & 63, rg = tid >> 6;
        for (int q = 0; q < Q; ++q) {
            const T zc = sz[q * kEdge + c];
            const VT *xr = reinterpret_cast<const VT *>(sx + q * kEdge + 16 * rg);
#pragma unroll
            for (int v = 0; v < 16 / W; ++v) {
                const VT xv = xr[v];
#pragma unroll
                for (int w = 0; w < W; ++w) {
                    const T d = xv[w] - zc;
                    s[v * W + w] = fma(d, d, s[v * W + w]);
                }
            }
        }
        const int m = m0 + c;
        if (m < M) {
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int64_t n = n0 + 16 * rg + j;
                if (n < N) out[n * M + m] = kval(pre, s[j]);
            }
        }
    } else {
        const int r = tid & 63, cg = tid >> 6;
        for (int q = 0; q < Q; ++q) {
            const T xr = sx[q * kEdge + r];
            const VT *zr = reinterpret_cast<const VT *>(sz + q * kEdge + 16 * cg);
#pragma unroll
            for (int v = 0; v < 16 / W; ++v) {
                const VT zv = zr[v];
#pragma unroll
                for (int w = 0; w < W; ++w) {
                    const T d = xr - zv[w];
                    s[v * W + w] = fma(d, d, s[v * W + w]);
                }
            }
        }
        const int64_t n = n0 + r;
        if (n < N) {
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int m = m0 + 16 * cg + j;
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

// ---------------------------------------------------------------- matrix-core block product
// C[i][j] = sum_k A[k][i] B[k][j] over one kBlk x kBlk block, both operands
// stored k-major (row k contiguous in i, resp. j): the layout of Kfu (rows n)
// for Psi2 and of G2s and Kfu^T (rows m) for the gradient.  Four waves in a
// 2 x 2 grid own 64 x 64 each.  k advances in LDS slabs of BK rows, double
// buffered: the next slab's global loads (16-byte vectors where the rows
// allow it) are in flight while the current slab feeds the matrix cores, so
// bounds are tested once per loaded vector and never per product.

template <typename T>
struct Slab {
    static constexpr int BK = sizeof(T) == 4 ? 32 : 16;   // k rows per stage
    static constexpr int VW = Vec<T>::W;                  // elements per vector
    static constexpr int RV = kBlk / VW;                  // vectors per slab row
    static constexpr int PER = BK * RV / 256;             // vectors per thread (4)
    static constexpr int SZ = BK * kBlk;                  // elements per slab
    static constexpr size_t LDS = 4 * SZ * sizeof(T);     // two buffers of (A, B)
};

template <typename T, bool VEC>
__device__ inline void slab_load(const T *__restrict__ src, int64_t ld, int64_t k0, int64_t k1,
                                 int64_t c0, int64_t c1, typename Vec<T>::t (&r)[Slab<T>::PER]) {
    constexpr int VW = Slab<T>::VW, RV = Slab<T>::RV;
#pragma unroll
    for (int u = 0; u < Slab<T>::PER; ++u) {
        const int f = threadIdx.x + 256 * u;
        const int kr = f / RV, cv = (f - kr * RV) * VW;
        const int64_t k = k0 + kr, c = c0 + cv;
        typename Vec<T>::t v;
        if (VEC && k < k1 && c + VW <= c1) {
            v = *reinterpret_cast<const typename Vec<T>::t *>(src + k * ld + c);
        } else {
#pragma unroll
            for (int w = 0; w < VW; ++w) v[w] = (k < k1 && c + w < c1) ? src[k * ld + c + w] : T(0);
        }
        r[u] = v;
    }
}

template <typename T>
__device__ inline void slab_store(T *lds, const typename Vec<T>::t (&r)[Slab<T>::PER]) {
    constexpr int VW = Slab<T>::VW, RV = Slab<T>::RV;
#pragma unroll
    for (int u = 0; u < Slab<T>::PER; ++u) {
        const int f = threadIdx.x + 256 * u;
        const int kr = f / RV, cv = (f - kr * RV) * VW;
        *reinterpret_cast<typename Vec<T>::t *>(lds + kr * kBlk + cv) = r[u];
    }
}

// acc[ti][tj]: tile (ti, tj) of this wave's 64 x 64 part.  Columns [a0, a_end)
// of A and [b0, b_end) of B over rows [k0, k1).  same: the two column ranges
// are one (a diagonal block of a symmetric product: B is not loaded, and
// tiles below the diagonal are skipped).
template <typename T, bool VEC>
__device__ inline void block_product(const T *__restrict__ A, int64_t lda, int64_t a0, int64_t a_end,
                                     const T *__restrict__ B, int64_t ldb, int64_t b0, int64_t b_end,
                                     int64_t k0, int64_t k1, bool same, T *lds,
                                     typename Mma<T>::acc_t (&acc)[64 / Mma<T>::TILE][64 / Mma<T>::TILE]) {
    using MM = Mma<T>;
    using SL = Slab<T>;
    constexpr int TILE = MM::TILE, KS = MM::KS, BT = 64 / TILE, BK = SL::BK, SZ = SL::SZ;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w & 1, wn = w >> 1;
    const int li = lane % TILE, lk = lane / TILE;
#pragma unroll
    for (int ti = 0; ti < BT; ++ti)
#pragma unroll
        for (int tj = 0; tj < BT; ++tj)
#pragma unroll
            for (int v = 0; v < MM::NACC; ++v) acc[ti][tj][v] = 0;
    const bool active = !(same && wm > wn);
    const bool diag = same && wm == wn;
    const int64_t stages = k1 > k0 ? (k1 - k0 + BK - 1) / BK : 0;
    // slabs are fetched two stages ahead into two register sets: the loads of
    // stage s + 2 are in flight while stage s computes and stage s + 1 (fetched
    // one stage earlier) waits in registers for its LDS buffer.  The stage loop
    // is unrolled by two so that each register set has a fixed name.
    using VT = typename Vec<T>::t;
    VT ra0[SL::PER], rb0[SL::PER], ra1[SL::PER], rb1[SL::PER];
    if (stages > 0) {
        slab_load<T, VEC>(A, lda, k0, k1, a0, a_end, ra0);
        if (!same) slab_load<T, VEC>(B, ldb, k0, k1, b0, b_end, rb0);
    }
    if (stages > 1) {
        slab_load<T, VEC>(A, lda, k0 + BK, k1, a0, a_end, ra1);
        if (!same) slab_load<T, VEC>(B, ldb, k0 + BK, k1, b0, b_end, rb1);
    }
    if (stages > 0) {
        slab_store<T>(lds, ra0);
        if (!same) slab_store<T>(lds + SZ, rb0);
        __syncthreads();
    }
    auto step = [&](int64_t s, VT(&rac)[SL::PER], VT(&rbc)[SL::PER], VT(&ran)[SL::PER],
                    VT(&rbn)[SL::PER]) {
        const T *sa = lds + (s & 1) * 2 * SZ;
        const T *sb = same ? sa : sa + SZ;
        if (s + 2 < stages) {  // the current set was stored to LDS one stage ago
            slab_load<T, VEC>(A, lda, k0 + (s + 2) * BK, k1, a0, a_end, rac);
            if (!same) slab_load<T, VEC>(B, ldb, k0 + (s + 2) * BK, k1, b0, b_end, rbc);
        }
        if (active) {
#pragma unroll
            for (int ks = 0; ks < BK / KS; ++ks) {
                const int row = (ks * KS + lk) * kBlk;
                T a[BT], b[BT];
#pragma unroll
                for (int t = 0; t < BT; ++t) {
                    a[t] = sa[row + wm * 64 + t * TILE + li];
                    b[t] = sb[row + wn * 64 + t * TILE + li];
                }
#pragma unroll
                for (int ti = 0; ti < BT; ++ti)
#pragma unroll
                    for (int tj = 0; tj < BT; ++tj)
                        if (!diag || ti <= tj) acc[ti][tj] = MM::mma(a[ti], b[tj], acc[ti][tj]);
            }
        }
        if (s + 1 < stages) {
            T *nb = lds + ((s + 1) & 1) * 2 * SZ;
            slab_store<T>(nb, ran);
            if (!same) slab_store<T>(nb + SZ, rbn);
        }
        __syncthreads();
    };
    for (int64_t s = 0; s < stages; s += 2) {
        step(s, ra0, rb0, ra1, rb1);
        if (s + 1 < stages) step(s + 1, ra1, rb1, ra0, rb0);
    }
}

// ---------------------------------------------------------------- Psi2 = Kfu^T Kfu
// One workgroup per (row chunk, upper kBlk-block pair (I, J)): the chunk's
// partial sums for every upper matrix-core tile of the pair.  Workgroups are
// dispatched round-robin over the 8 XCDs, so the block pairs of one chunk get
// ids on the same XCD and share its L2.
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void known_syrk_kernel(int64_t N, int M, int64_t rows,
                                                         int64_t chunks, int64_t nb, int64_t ntp,
                                                         int64_t ntu, const T *__restrict__ K,
                                                         T *__restrict__ part) {
    using MM = Mma<T>;
    constexpr int TILE = MM::TILE, BT = 64 / TILE;
    __shared__ __align__(16) T lds[4 * Slab<T>::SZ];
    const int64_t nbp = nb * (nb + 1) / 2;
    const int64_t id = blockIdx.x, slot = id >> 3;
    const int64_t chunk = (slot / nbp) * 8 + (id & 7);
    if (chunk >= chunks) return;
    int I, J;
    block_pair(slot % nbp, nb, I, J);
    const int64_t r0 = chunk * rows, r1 = min(N, r0 + rows);
    typename MM::acc_t acc[BT][BT];
    block_product<T, VEC>(K, M, (int64_t)I * kBlk, M, K, M, (int64_t)J * kBlk, M, r0, r1, I == J, lds,
                          acc);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w & 1, wn = w >> 1;
#pragma unroll
    for (int ti = 0; ti < BT; ++ti)
#pragma unroll
        for (int tj = 0; tj < BT; ++tj) {
            const int64_t gi = ((int64_t)I * kBlk + wm * 64) / TILE + ti;
            const int64_t gj = ((int64_t)J * kBlk + wn * 64) / TILE + tj;
            if (gi > gj) continue;
            const int64_t p = gi * ntp - gi * (gi - 1) / 2 + (gj - gi);
            T *dst = part + (chunk * ntu + p) * (TILE * TILE);
#pragma unroll
            for (int v = 0; v < MM::NACC; ++v) dst[MM::row(v, lane) * TILE + lane % TILE] = acc[ti][tj][v];
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

// E^T[m][n] = (G1[n][m] + 2 sum_k G2s[m][k] Kt[k][n]) Kt[m][n], one workgroup
// per kBlk x kBlk block (m, n) on the matrix cores.  G2s is symmetric, so its
// A operand G2s[m][k] is read as G2s[k][m], a contiguous row.  Same XCD
// grouping as the rank-k update: the m-blocks of one column block n share an XCD.
template <typename T, bool HAS_G2, bool VEC>
__global__ __launch_bounds__(256) void known_dkfu_kernel(int64_t N, int M, int64_t nblk, int64_t mb,
                                                         const T *__restrict__ Kt,
                                                         const T *__restrict__ G1,
                                                         const T *__restrict__ G2s,
                                                         T *__restrict__ Et) {
    using MM = Mma<T>;
    constexpr int TILE = MM::TILE, BT = 64 / TILE;
    __shared__ __align__(16) T lds[4 * Slab<T>::SZ];
    const int64_t id = blockIdx.x, slot = id >> 3;
    const int64_t nbi = (slot / mb) * 8 + (id & 7);
    if (nbi >= nblk) return;
    const int64_t n0 = nbi * kBlk;
    const int64_t m0 = (slot % mb) * kBlk;
    typename MM::acc_t acc[BT][BT];
    block_product<T, VEC>(G2s, M, m0, M, Kt, N, n0, N, 0, HAS_G2 ? M : 0, false, lds, acc);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w & 1, wn = w >> 1;
#pragma unroll
    for (int tm = 0; tm < BT; ++tm)
#pragma unroll
        for (int tn = 0; tn < BT; ++tn)
#pragma unroll
            for (int v = 0; v < MM::NACC; ++v) {
                const int64_t m = m0 + wm * 64 + tm * TILE + MM::row(v, lane);
                const int64_t n = n0 + wn * 64 + tn * TILE + lane % TILE;
                if (m < M && n < N) {
                    const T g1 = G1 ? G1[n * M + m] : T(0);
                    const int64_t o = m * N + n;
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

// Chain-rule kernels.  Every difference xs_nq - zs_mq is formed before it is
// weighted by E, so no large sums are subtracted afterwards (the expanded forms,
// sum_n E xs - zs sum_n E and the like, can cancel to a small remainder where E
// is concentrated around z_m far from the centre).  LDS rows are zero beyond Q,
// and so are the register
// copies of the fixed point, so the padded dimensions contribute nothing (no
// per-dimension guard: a runtime bound inside the unrolled loops makes the
// compiler shuffle the accumulators).

// One thread per datapoint: dx_nq = -sum_m E^T[m][n] (xs_nq - zs_mq) / l_q
// (coalesced over n, loads issued 16 at a time) and a per-block partial of
// sum E (dsf2).
template <typename T, int QM>
__global__ __launch_bounds__(256) void known_rows_kernel(int64_t N, int M, int Q,
                                                         const T *__restrict__ Et,
                                                         const T *__restrict__ xs,
                                                         const T *__restrict__ zs, Hyp<T> h,
                                                         T *__restrict__ dX,
                                                         T *__restrict__ rowpart) {
    using V = typename Vec<T>::t;
    constexpr int W = Vec<T>::W;
    __shared__ __align__(16) T sz[kEdge][QM];  // zero beyond Q and beyond the block's rows
    __shared__ T red4[4];
    const int tid = threadIdx.x;
    const int64_t n = (int64_t)blockIdx.x * 256 + tid;
    const bool valid = n < N;
    T r = 0, U[QM], x[QM];
#pragma unroll
    for (int q = 0; q < QM; ++q) {
        U[q] = 0;
        x[q] = (valid && q < Q) ? xs[n * Q + q] : T(0);
    }
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
                    const V *zr = reinterpret_cast<const V *>(&sz[c0 + j][0]);
#pragma unroll
                    for (int v = 0; v < QM / W; ++v) {
                        const V z = zr[v];
#pragma unroll
                        for (int w = 0; w < W; ++w)
                            U[v * W + w] = fma(e[j], x[v * W + w] - z[w], U[v * W + w]);
                    }
                }
            }
        }
    }
    if (valid) {
#pragma unroll
        for (int q = 0; q < QM; ++q)
            if (q < Q) dX[n * Q + q] = -U[q] / h.l[q];
    }
    const T sr = block_sum(valid ? r : T(0), red4);
    if (tid == 0) rowpart[blockIdx.x] = sr;
}

// One workgroup per (64 inducing inputs, row chunk), E^T tiles staged in LDS:
// per inducing input m the chunk's sum_n E (xs_nq - zs_mq) (dZ) and
// sum_n E (xs_nq - zs_mq)^2 (dl) -> colpart[chunk][m][2 Q].
template <typename T, int QM>
__global__ __launch_bounds__(256) void known_cols_kernel(int64_t N, int M, int Q, int64_t rows,
                                                         const T *__restrict__ Et,
                                                         const T *__restrict__ xs,
                                                         const T *__restrict__ zs,
                                                         T *__restrict__ colpart) {
    using Vv = typename Vec<T>::t;
    constexpr int W = Vec<T>::W;
    __shared__ T se[kEdge][kEdge + 1];         // E^T tile [m][n], zero outside
    __shared__ __align__(16) T sx[kEdge][QM];  // xs rows of the tile, zero outside
    __shared__ T red[4][kEdge];
    const int tid = threadIdx.x;
    const int m0 = blockIdx.x * kEdge;
    const int64_t r0 = (int64_t)blockIdx.y * rows, r1 = min(N, r0 + rows);
    const int mr = tid & 63, quarter = tid >> 6;
    const int m = m0 + mr;
    T V[QM], D[QM], z[QM];
#pragma unroll
    for (int q = 0; q < QM; ++q) {
        V[q] = D[q] = 0;
        z[q] = (m < M && q < Q) ? zs[(int64_t)m * Q + q] : T(0);
    }
    for (int64_t nb = r0; nb < r1; nb += kEdge) {
        const int cnt = (int)min<int64_t>(kEdge, r1 - nb);
        __syncthreads();
        for (int i = tid; i < kEdge * kEdge; i += 256) {
            const int row = i >> 6, col = i & 63;
            const int mm = m0 + row;
            se[row][col] = (mm < M && col < cnt) ? Et[(int64_t)mm * N + nb + col] : T(0);
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
            const Vv *xr = reinterpret_cast<const Vv *>(&sx[col][0]);
#pragma unroll
            for (int v = 0; v < QM / W; ++v) {
                const Vv xv = xr[v];
#pragma unroll
                for (int w = 0; w < W; ++w) {
                    const int q = v * W + w;
                    const T d = xv[w] - z[q];
                    const T t = e * d;
                    V[q] += t;
                    D[q] = fma(t, d, D[q]);
                }
            }
        }
    }
#pragma unroll
    for (int k = 0; k < 2 * QM; ++k) {
        const int q = k < QM ? k : k - QM;
        if (q < Q) {
            __syncthreads();
            red[quarter][mr] = k < QM ? V[q] : D[q];
            __syncthreads();
            if (quarter == 0 && m < M)
                colpart[((int64_t)blockIdx.y * M + m) * (2 * Q) + (k < QM ? q : Q + q)] =
                    ((red[0][mr] + red[1][mr]) + red[2][mr]) + red[3][mr];
        }
    }
}

// One workgroup per inducing input m: Vc[m][k] = sum over the column chunks of
// colpart[chunk][m][k], k < 2 Q.  G = 256 / (2 Q) groups of 2 Q threads take
// chunks g, g + G, ... (coalesced over k); the G partials are added in order.
template <typename T>
__global__ __launch_bounds__(256) void known_col_reduce_kernel(int M, int Q, int64_t cchunks,
                                                               const T *__restrict__ colpart,
                                                               T *__restrict__ Vc) {
    __shared__ T part[256];
    const int t = threadIdx.x, K = 2 * Q, G = 256 / K;
    const int64_t m = blockIdx.x;
    if (t < G * K) {
        const int g = t / K, k = t - g * K;
        T s = 0;
        for (int64_t c = g; c < cchunks; c += G) s += colpart[(c * M + m) * K + k];
        part[t] = s;
    }
    __syncthreads();
    if (t < K) {
        T s = 0;
        for (int g = 0; g < G; ++g) s += part[g * K + t];
        Vc[m * K + t] = s;
    }
}

// dZ[m][q] = Vc[m][q] / l_q elementwise (blocks below zblocks), then one
// workgroup per dl_q (sum_m Vc[m][Q + q] / l_q) and one for dsf2 (sum E / sf2 +
// N dL/dpsi0), each a fixed-order block sum.
template <typename T>
__global__ __launch_bounds__(256) void known_grad_final_kernel(
    int64_t N, int M, int Q, int64_t zblocks, int64_t rblocks, const T *__restrict__ Vc,
    const T *__restrict__ rowpart, Hyp<T> h, T dL_dpsi0, T *__restrict__ dZ, T *__restrict__ dsf2,
    T *__restrict__ dl, int accumulate) {
    __shared__ T red4[4];
    const int64_t K = 2 * Q;
    if ((int64_t)blockIdx.x < zblocks) {
        const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
        if (i >= (int64_t)M * Q) return;
        const int64_t m = i / Q, q = i - m * Q;
        dZ[i] = (accumulate ? dZ[i] : T(0)) + Vc[m * K + q] / h.l[q];
        return;
    }
    const int k = (int)(blockIdx.x - zblocks);  // k < Q: dl_k; k == Q: dsf2
    T s = 0;
    if (k < Q)
        for (int m = threadIdx.x; m < M; m += 256) s += Vc[(int64_t)m * K + Q + k];
    else
        for (int64_t b = threadIdx.x; b < rblocks; b += 256) s += rowpart[b];
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
        s.N, (int)s.M, (int)s.Q, p.crows, Et, xs, zs, at<T>(ws, p.off_colp));
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
        // 16-byte loads need rows that start on 16 bytes
        if (s.M % Vec<T>::W == 0 && reinterpret_cast<uintptr_t>(K) % 16 == 0)
            known_syrk_kernel<T, true><<<(unsigned)p.grid_syrk, 256, 0, st>>>(
                s.N, (int)s.M, p.rows, p.chunks, p.nb2, p.ntp, p.ntu, K, part);
        else
            known_syrk_kernel<T, false><<<(unsigned)p.grid_syrk, 256, 0, st>>>(
                s.N, (int)s.M, p.rows, p.chunks, p.nb2, p.ntp, p.ntu, K, part);
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
    const int64_t nblk = cdiv(s.N, kBlk), mb = p.nb2;
    const unsigned grid = (unsigned)(round_up(nblk, 8) * mb);
    const bool vec = s.M % Vec<T>::W == 0 && s.N % Vec<T>::W == 0;  // workspace rows start on 16 bytes
    if (G2) {
        T *G2s = at<T>(ws, p.off_g2s);
        {
            TimedScope ts(st, "known_sym");
            known_sym_kernel<T><<<(unsigned)cdiv(s.M * s.M, 256), 256, 0, st>>>((int)s.M, G2, G2s);
        }
        TimedScope ts(st, "known_dkfu");
        if (vec)
            known_dkfu_kernel<T, true, true><<<grid, 256, 0, st>>>(s.N, (int)s.M, nblk, mb, Kt, G1, G2s, Et);
        else
            known_dkfu_kernel<T, true, false><<<grid, 256, 0, st>>>(s.N, (int)s.M, nblk, mb, Kt, G1, G2s, Et);
    } else {
        TimedScope ts(st, "known_dkfu");
        known_dkfu_kernel<T, false, false><<<grid, 256, 0, st>>>(s.N, (int)s.M, nblk, mb, Kt, G1, nullptr,
                                                                 Et);
    }
    // the chain kernels pad Q to QM (a multiple of the 16-byte vector)
    if (s.Q <= 4) launch_chain<T, 4>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 8) launch_chain<T, 8>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 12) launch_chain<T, 12>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 16) launch_chain<T, 16>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 20) launch_chain<T, 20>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 24) launch_chain<T, 24>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 32) launch_chain<T, 32>(s, p, Et, h, dX, ws, st);
    else if (s.Q <= 48) launch_chain<T, 48>(s, p, Et, h, dX, ws, st);
    else launch_chain<T, 64>(s, p, Et, h, dX, ws, st);
    TimedScope ts(st, "known_grad_reduce");
    T *Vc = at<T>(ws, p.off_vc);
    known_col_reduce_kernel<T><<<(unsigned)s.M, 256, 0, st>>>((int)s.M, (int)s.Q, p.cchunks,
                                                             at<T>(ws, p.off_colp), Vc);
    const int64_t zblocks = cdiv(s.M * s.Q, 256);
    known_grad_final_kernel<T><<<(unsigned)(zblocks + s.Q + 1), 256, 0, st>>>(
        s.N, (int)s.M, (int)s.Q, zblocks, p.rblocks, Vc, at<T>(ws, p.off_rowp), h, dL_dpsi0, dZ,
        dsf2, dl, accumulate);
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
