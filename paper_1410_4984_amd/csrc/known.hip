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
    int64_t tiles;              // 64-row tiles of the datapoints (chain kernel)
    int64_t gmax;               // chain kernel: most tile groups per inducing-input block
    size_t off_cz, off_xs, off_zs, off_k, off_e, off_g2s, off_part, off_ep, off_colp, off_vc, off_dxp;
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
    // the chain kernel's grid is one round of resident workgroups, at most 8
    // per CU on 256 CUs
    p.tiles = cdiv(s.N, kEdge);
    p.gmax = std::max<int64_t>(1, std::min<int64_t>(p.tiles, std::max<int64_t>(1, 2048 / p.nb)));
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
    p.off_cz = take(elem * s.Q);
    p.off_xs = take(elem * s.N * s.Q);
    p.off_zs = take(elem * s.M * s.Q);
    p.off_k = take(elem * s.N * s.M);
    p.off_e = take(elem * s.N * s.M);
    p.off_g2s = take(elem * s.M * s.M);
    p.off_part = take(elem * p.chunks * p.ntu * p.tile * p.tile);
    p.off_ep = take(elem * p.nb * p.gmax);
    p.off_colp = take(elem * p.gmax * s.M * 2 * s.Q);
    p.off_vc = take(elem * s.M * 2 * s.Q);
    p.off_dxp = take(elem * p.nb * s.N * s.Q);
    p.total = o;
    return p;
}

// ---------------------------------------------------------------- centring
// cz[q] = mean_m z_mq, zs = (Z - cz) / l.  One workgroup: G = 1024 / Q groups of
// Q threads sum rows m = g, g + G, ... (coalesced; loads issued 8 at a time so
// that they overlap), then the G partial sums of each dimension are added in
// group order.
template <typename T>
__global__ __launch_bounds__(1024) void known_centre_kernel(int M, int Q, const T *__restrict__ Z,
                                                           Hyp<T> h, T *__restrict__ cz,
                                                           T *__restrict__ zs) {
    __shared__ T part[1024];
    __shared__ T c[GPPS_MAX_Q];
    const int t = threadIdx.x, G = 1024 / Q;
    if (t < G * Q) {
        const int g = t / Q, q = t - g * Q;
        T s = 0;
        int m = g;
        for (; m + 7 * G < M; m += 8 * G) {
            T v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = Z[(int64_t)(m + j * G) * Q + q];
#pragma unroll
            for (int j = 0; j < 8; ++j) s += v[j];
        }
        for (; m < M; m += G) s += Z[(int64_t)m * Q + q];
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
#pragma unroll 4
    for (int i = t; i < M * Q; i += 1024) zs[i] = (Z[i] - c[i % Q]) / h.l[i % Q];
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
__global__ __launch_bounds__(256, sizeof(T) == 4 ? 2 : 1) void known_dkfu_kernel(int64_t N, int M, int64_t nblk, int64_t mb,
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
    // Per tile, every load of the epilogue is issued before the first use, from
    // clamped (valid) addresses; only the stores test the bounds.  (Loads under
    // the bounds test were each waited for in turn: one memory round trip per
    // output element.)
#pragma unroll
    for (int tm = 0; tm < BT; ++tm)
#pragma unroll
        for (int tn = 0; tn < BT; ++tn) {
            T g1[MM::NACC], kv[MM::NACC];
            const int64_t n = n0 + wn * 64 + tn * TILE + lane % TILE;
            const int64_t nc = min(n, N - 1);
#pragma unroll
            for (int v = 0; v < MM::NACC; ++v) {
                const int64_t m = min<int64_t>(m0 + wm * 64 + tm * TILE + MM::row(v, lane), M - 1);
                kv[v] = Kt[m * N + nc];
                g1[v] = G1 ? G1[nc * M + m] : T(0);
            }
#pragma unroll
            for (int v = 0; v < MM::NACC; ++v) {
                const int64_t m = m0 + wm * 64 + tm * TILE + MM::row(v, lane);
                if (m < M && n < N) Et[m * N + n] = (g1[v] + T(2) * acc[tm][tn][v]) * kv[v];
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

// Chain-rule sums, both from one pass over E^T.  Every difference xs_nq - zs_mq
// is formed before it is weighted by E, so no large sums are subtracted
// afterwards (the expanded forms, sum_n E xs - zs sum_n E and the like, can
// cancel to a small remainder where E is concentrated around z_m far from the
// centre).  LDS rows are zero beyond Q and beyond the edge of the data, so the
// padded dimensions and rows contribute nothing (no per-dimension guard: a
// runtime bound inside the unrolled loops makes the compiler shuffle the
// accumulators).
//
// Workgroup (64-block of inducing inputs b, group g) takes the 64-row tiles of
// the datapoints g, g + G, g + 2G, ...  Each E^T tile [64 m][64 n] is loaded
// once (the next one is in flight while the current one is used) and read
// twice from LDS.  Wave w owns the dimensions q = w, w + 4, w + 8, ...:
//   columns: thread (m, w) adds E d and E d^2 over the tile's 64 n to
//            registers kept over the workgroup's tiles -> colpart[g][m][2 Q];
//   rows:    thread (n, w) sums E d over the block's 64 m -> dxpart[b][q][n];
// and sum E per workgroup -> epart[g * nb + b] (dsf2).
// A wave's dimensions sit in a slot of QP = QM/4 rounded up to the 16-byte
// vector, so that each is read as whole vectors: xs and zs rows are
// [64][4 slots][QP], zero in the padding.
template <typename T>
constexpr int chain_qp(int QM) { return (QM / 4 + Vec<T>::W - 1) / Vec<T>::W * Vec<T>::W; }

template <typename T>
size_t chain_lds_bytes(int QM) {  // sx [64][4][QP], sz [64][4][QP], se [64][65], red4
    return sizeof(T) * (2 * (size_t)kEdge * 4 * chain_qp<T>(QM) + (size_t)kEdge * (kEdge + 1) + 4);
}

template <typename T, int QM, bool VEC>
__global__ __launch_bounds__(256) void known_chain_kernel(int64_t N, int M, int Q, int64_t tiles,
                                                          int64_t G, const T *__restrict__ Et,
                                                          const T *__restrict__ xs,
                                                          const T *__restrict__ zs,
                                                          T *__restrict__ dxpart,
                                                          T *__restrict__ colpart,
                                                          T *__restrict__ epart) {
    using Vv = typename Vec<T>::t;
    constexpr int W = Vec<T>::W;
    constexpr int RV = kEdge / W;               // vectors per tile row
    constexpr int EV = kEdge * RV / 256;        // tile vectors per thread
    constexpr int XP = kEdge * QM / 256;        // xs tile elements per thread
    constexpr int QC = QM / 4;                  // dimensions per thread
    constexpr int QP = chain_qp<T>(QM);         // their padded slot
    constexpr int RS = 4 * QP;                  // xs / zs row stride in LDS
    static_assert(QM % 4 == 0, "QM is a multiple of 4");
    extern __shared__ __align__(16) unsigned char chain_smem[];
    T *sx = reinterpret_cast<T *>(chain_smem);  // [64][4][QP]
    T *sz = sx + kEdge * RS;                    // [64][4][QP]
    T *se = sz + kEdge * RS;                    // [64][65], E^T tile [m][n]
    T *red4 = se + kEdge * (kEdge + 1);         // [4]
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int blk = blockIdx.x, nbk = gridDim.x;
    const int64_t g = blockIdx.y;
    const int m0 = blk * kEdge;

    // slot w, entry i holds dimension q = w + 4 i (zero where q >= Q and in the padding)
    for (int i = tid; i < kEdge * RS; i += 256) {
        const int r = i / RS, k = i - r * RS, w = k / QP, j = k - w * QP, q = w + 4 * j;
        sz[i] = (m0 + r < M && j < QC && q < Q) ? zs[(int64_t)(m0 + r) * Q + q] : T(0);
        sx[i] = T(0);
    }
    __syncthreads();
    T zq[QC], Vc[QC], Dc[QC];
#pragma unroll
    for (int i = 0; i < QC; ++i) {
        zq[i] = sz[lane * RS + wv * QP + i];
        Vc[i] = Dc[i] = 0;
    }
    T esum = 0;

    Vv ev[EV];
    T xv[XP];
    auto load = [&](int64_t t) {
        const int64_t n0 = t * kEdge;
#pragma unroll
        for (int u = 0; u < EV; ++u) {
            const int f = tid + 256 * u;
            const int row = f / RV, cv = (f - row * RV) * W;
            const int m = m0 + row;
            const int64_t n = n0 + cv;
            if (VEC && m < M && n + W <= N) {
                ev[u] = *reinterpret_cast<const Vv *>(Et + (int64_t)m * N + n);
            } else {
#pragma unroll
                for (int w = 0; w < W; ++w)
                    ev[u][w] = (m < M && n + w < N) ? Et[(int64_t)m * N + n + w] : T(0);
            }
        }
#pragma unroll
        for (int u = 0; u < XP; ++u) {
            const int f = tid + 256 * u;
            const int r = f / QM, q = f - r * QM;
            xv[u] = (n0 + r < N && q < Q) ? xs[(n0 + r) * Q + q] : T(0);
        }
    };
    if (g < tiles) load(g);
    for (int64_t t = g; t < tiles; t += G) {
        __syncthreads();  // the previous tile's LDS reads are done
#pragma unroll
        for (int u = 0; u < EV; ++u) {
            const int f = tid + 256 * u;
            const int row = f / RV, cv = (f - row * RV) * W;
#pragma unroll
            for (int w = 0; w < W; ++w) se[row * (kEdge + 1) + cv + w] = ev[u][w];
        }
#pragma unroll
        for (int u = 0; u < XP; ++u) {
            const int f = tid + 256 * u;
            const int r = f / QM, q = f - r * QM;
            sx[r * RS + (q & 3) * QP + (q >> 2)] = xv[u];
        }
        __syncthreads();
        if (t + G < tiles) load(t + G);
        // columns: m = m0 + lane over the tile's 64 n
#pragma unroll 4
        for (int c = 0; c < kEdge; ++c) {
            const T e = se[lane * (kEdge + 1) + c];
            T xr[QP];
#pragma unroll
            for (int v = 0; v < QP / W; ++v) {
                const Vv xq = reinterpret_cast<const Vv *>(sx + c * RS + wv * QP)[v];
#pragma unroll
                for (int w = 0; w < W; ++w) xr[v * W + w] = xq[w];
            }
#pragma unroll
            for (int i = 0; i < QC; ++i) {
                const T d = xr[i] - zq[i];
                const T te = e * d;
                Vc[i] += te;
                Dc[i] = fma(te, d, Dc[i]);
            }
        }
        // rows: n = n0 + lane over the block's 64 m
        T x[QC], U[QC];
#pragma unroll
        for (int i = 0; i < QC; ++i) {
            x[i] = sx[lane * RS + wv * QP + i];
            U[i] = 0;
        }
#pragma unroll 4
        for (int r = 0; r < kEdge; ++r) {
            const T e = se[r * (kEdge + 1) + lane];
            if (wv == 0) esum += e;
            T zr[QP];
#pragma unroll
            for (int v = 0; v < QP / W; ++v) {
                const Vv zv = reinterpret_cast<const Vv *>(sz + r * RS + wv * QP)[v];
#pragma unroll
                for (int w = 0; w < W; ++w) zr[v * W + w] = zv[w];
            }
#pragma unroll
            for (int i = 0; i < QC; ++i) U[i] = fma(e, x[i] - zr[i], U[i]);
        }
        const int64_t n = t * kEdge + lane;
        if (n < N) {
#pragma unroll
            for (int i = 0; i < QC; ++i) {
                const int q = wv + 4 * i;
                if (q < Q) dxpart[((int64_t)blk * Q + q) * N + n] = U[i];
            }
        }
    }
    const int m = m0 + lane;
    if (m < M && g < tiles) {
#pragma unroll
        for (int i = 0; i < QC; ++i) {
            const int q = wv + 4 * i;
            if (q < Q) {
                colpart[(g * M + m) * (2 * Q) + q] = Vc[i];
                colpart[(g * M + m) * (2 * Q) + Q + q] = Dc[i];
            }
        }
    }
    const T se_all = block_sum(esum, red4);
    if (tid == 0) epart[g * nbk + blk] = se_all;
}

// dX = -(sum over the inducing-input blocks of dxpart, in block order) / l.
// One workgroup per 64 datapoints: the sums are read coalesced over n from
// dxpart [b][q][n] and written through an LDS transpose as the block's 64 Q
// contiguous elements of dX.
template <typename T>
__global__ __launch_bounds__(256) void known_dx_kernel(int64_t N, int Q, int nbk,
                                                       const T *__restrict__ dxpart, Hyp<T> h,
                                                       T *__restrict__ dX) {
    __shared__ T tile[kEdge][GPPS_MAX_Q + 1];
    const int tid = threadIdx.x, nn = tid & 63;
    const int64_t n0 = (int64_t)blockIdx.x * kEdge, n = n0 + nn;
    const int cnt = (int)min<int64_t>(kEdge, N - n0);
    if (n < N) {
        for (int q = tid >> 6; q < Q; q += 4) {
            T s = 0;
            for (int b = 0; b < nbk; ++b) s += dxpart[((int64_t)b * Q + q) * N + n];
            tile[nn][q] = -s / h.l[q];
        }
    }
    __syncthreads();
    for (int i = tid; i < cnt * Q; i += 256) {
        const int r = i / Q, q = i - r * Q;
        dX[n0 * Q + i] = tile[r][q];
    }
}

// One workgroup per inducing input m: Vc[m][k] = sum over the chain kernel's
// tile groups of colpart[group][m][k], k < 2 Q.  S = 256 / (2 Q) sets of 2 Q
// threads take groups s, s + S, ... (coalesced over k); the S partials are
// added in order.
template <typename T>
__global__ __launch_bounds__(256) void known_col_reduce_kernel(int M, int Q, int64_t groups,
                                                               const T *__restrict__ colpart,
                                                               T *__restrict__ Vc) {
    __shared__ T part[256];
    const int t = threadIdx.x, K = 2 * Q, S = 256 / K;
    const int64_t m = blockIdx.x;
    if (t < S * K) {
        const int j = t / K, k = t - j * K;
        // groups j, j + S, ... in order; loads issued 8 at a time so that they overlap
        T s = 0;
        int64_t c = j;
        for (; c + 7 * S < groups; c += 8 * S) {
            T v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = colpart[((c + u * S) * M + m) * K + k];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; c < groups; c += S) s += colpart[(c * M + m) * K + k];
        part[t] = s;
    }
    __syncthreads();
    if (t < K) {
        T s = 0;
        for (int j = 0; j < S; ++j) s += part[j * K + t];
        Vc[m * K + t] = s;
    }
}

// dZ[m][q] = Vc[m][q] / l_q elementwise (blocks below zblocks), then one
// workgroup per dl_q (sum_m Vc[m][Q + q] / l_q) and one for dsf2 (sum E / sf2 +
// N dL/dpsi0, sum E from the chain kernel's nep partials), each a fixed-order
// block sum.
template <typename T>
__global__ __launch_bounds__(256) void known_grad_final_kernel(
    int64_t N, int M, int Q, int64_t zblocks, int64_t nep, const T *__restrict__ Vc,
    const T *__restrict__ epart, Hyp<T> h, T dL_dpsi0, T *__restrict__ dZ, T *__restrict__ dsf2,
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
        for (int64_t b = threadIdx.x; b < nep; b += 256) s += epart[b];
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
        known_centre_kernel<T><<<1, 1024, 0, st>>>((int)s.M, (int)s.Q, Z, h, cz, zs);
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
hipError_t launch_chain(const Shape &s, const KPlan &p, const T *Et, const Hyp<T> &h, T *dX,
                        void *ws, hipStream_t st, int64_t &G) {
    const T *xs = at<T>(ws, p.off_xs), *zs = at<T>(ws, p.off_zs);
    // workspace rows of E^T start on 16 bytes when N is a multiple of the vector
    auto k = s.N % Vec<T>::W == 0 ? known_chain_kernel<T, QM, true> : known_chain_kernel<T, QM, false>;
    const size_t lds = chain_lds_bytes<T>(QM);
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0, occ = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, k, 256, lds)) != hipSuccess) return e;
    // one round of resident workgroups over the inducing-input blocks
    G = std::max<int64_t>(1, std::min<int64_t>(p.gmax, (int64_t)std::max(1, occ) * cus / p.nb));
    {
        TimedScope ts(st, "known_chain");
        k<<<dim3((unsigned)p.nb, (unsigned)G), 256, lds, st>>>(
            s.N, (int)s.M, (int)s.Q, p.tiles, G, Et, xs, zs, at<T>(ws, p.off_dxp),
            at<T>(ws, p.off_colp), at<T>(ws, p.off_ep));
    }
    TimedScope ts(st, "known_dx");
    known_dx_kernel<T><<<(unsigned)p.tiles, 256, 0, st>>>(s.N, (int)s.Q, (int)p.nb,
                                                         at<T>(ws, p.off_dxp), h, dX);
    return hipGetLastError();
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
    // the chain kernel pads Q to QM (a multiple of 4)
    int64_t G = 1;
    hipError_t e;
    if (s.Q <= 4) e = launch_chain<T, 4>(s, p, Et, h, dX, ws, st, G);
    else if (s.Q <= 8) e = launch_chain<T, 8>(s, p, Et, h, dX, ws, st, G);
    else if (s.Q <= 12) e = launch_chain<T, 12>(s, p, Et, h, dX, ws, st, G);
    else if (s.Q <= 16) e = launch_chain<T, 16>(s, p, Et, h, dX, ws, st, G);
    else if (s.Q <= 20) e = launch_chain<T, 20>(s, p, Et, h, dX, ws, st, G);
    else if (s.Q <= 24) e = launch_chain<T, 24>(s, p, Et, h, dX, ws, st, G);
    else if (s.Q <= 32) e = launch_chain<T, 32>(s, p, Et, h, dX, ws, st, G);
    else if (s.Q <= 48) e = launch_chain<T, 48>(s, p, Et, h, dX, ws, st, G);
    else e = launch_chain<T, 64>(s, p, Et, h, dX, ws, st, G);
    if (e != hipSuccess) return e;
    TimedScope ts(st, "known_grad_reduce");
    T *Vc = at<T>(ws, p.off_vc);
    known_col_reduce_kernel<T><<<(unsigned)s.M, 256, 0, st>>>((int)s.M, (int)s.Q, G,
                                                             at<T>(ws, p.off_colp), Vc);
    const int64_t zblocks = cdiv(s.M * s.Q, 256);
    known_grad_final_kernel<T><<<(unsigned)(zblocks + s.Q + 1), 256, 0, st>>>(
        s.N, (int)s.M, (int)s.Q, zblocks, p.nb * G, Vc, at<T>(ws, p.off_ep), h, dL_dpsi0, dZ,
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
