// Generic vector-ALU path: RBF-ARD psi-statistics and gradients, templated on
// the element type (float or double).
//
// What is computed (section 2, eq. (4): phi, Phi and Psi become expectations
// under q(x_n) = N(mu_n, diag S_n); Alg. 1 and Alg. 2).  With
//   w1 = 1 / (l^2 + S),  w2 = 1 / (l^2 + 2 S)                          per (n, q)
//   lp1_n = log sf2   - 1/2 sum_q log(1 + S/l^2)
//   lp2_n = 2 log sf2 - 1/2 sum_q log(1 + 2 S/l^2)
// the exact Gaussian integrals give
//   Psi1[n, m]    = exp(lp1_n - 1/2 sum_q (mu - z_m)^2 w1)
//   Psi2_n[m, m'] = exp(lp2_n - sum_q [(z_m - z_m')^2 / (4 l^2) + (mu - zbar)^2 w2])
// with zbar = (z_m + z_m') / 2, and Psi2 = sum_n Psi2_n.
//
// Work split: Psi1 one thread per output; Psi2 one thread per unique pair
// (m <= m'), partial sums per row chunk reduced in a fixed order.  Gradients,
// by the first form that applies:
//   * pairs kernels (small Q): one thread per inducing input m, the Z table in
//     LDS, per row the sums r and V over the partners m' (symmetric form: each
//     unordered pair evaluated once);
//   * the wide kernel (Q up to 32 in fp64, 64 in fp32): the same ordered sums
//     with two lanes per m, each holding half of the dimensions;
//   * otherwise a row kernel (one thread per datapoint and range of pair rows m:
//     dmu, dS and dl / dsf2 partials) and a column kernel (one thread per
//     inducing input, row chunk and range of partners: dZ partials).
// Fixed-order reduce kernels combine the partials.  No atomics anywhere.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace gpps {
namespace {

constexpr int kRowTile = 32;     // rows staged in LDS at a time
constexpr int kFwdTile = 128;    // ... by the forward pair kernel
constexpr int kPairTile = 16;    // pair tile edge (16 x 16 threads)
constexpr int kRowBlock = 64;    // threads (rows) per block in the gradient row kernel
constexpr int kColBlock = 64;    // threads (inducing inputs) per block in the column kernel
constexpr int kBand = 8;         // symmetric pairs kernel: pair offsets k per LDS exchange
constexpr int kSlotBand = 4;     // ... the same with several rows at a time
constexpr int64_t kGridCap = 2048;  // workgroups of the grid-stride kernels

__device__ inline float dexp(float x) { return __expf(x); }
__device__ inline double dexp(double x) { return exp(x); }
__device__ inline float dlog1p(float x) { return log1pf(x); }
__device__ inline double dlog1p(double x) { return log1p(x); }

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Register width (latent dimensions, padded) of the pairs kernel for Q.
inline int64_t pairs_qm(int64_t Q) { return Q <= 1 ? 1 : Q <= 2 ? 2 : Q <= 4 ? 4 : Q <= 8 ? 8 : 16; }
// Register width (dimensions, padded) of the forward pair kernel for Q, and its
// pairs per thread (two where a dimension's LDS read would otherwise serve one
// pair's three operations; one at small widths and for wide fp64 rows).
inline int fwd_qm(int64_t Q) {
    for (int qm : {1, 2, 4, 8, 12, 16, 20, 24, 32, 48})
        if (Q <= qm) return qm;
    return 64;
}
inline int fwd_ppt(int64_t Q, size_t elem) {
    const int qm = fwd_qm(Q);
    return qm >= 8 && !(elem == 8 && qm >= 48) ? 2 : 1;
}
// Dimensions per lane of the wide gradient kernel for Q (0: none fits; fp64
// keeps seven arrays of QH doubles live, fp32 the same in floats).
inline int wide_qh(int64_t Q, size_t elem) {
    for (int qh : {4, 6, 8, 10, 12, 16, 24, 32})
        if (2 * qh >= Q) return (elem == 8 && qh > 16) ? 0 : qh;
    return 0;
}

struct Plan {
    int64_t tiles_edge;              // pair tiles per edge (Psi2 reduce)
    int64_t pblocks;                 // forward: blocks of 256 unique pairs
    int64_t nc2;                     // row chunks of the Psi2 forward kernel
    int64_t rows2;                   // rows per chunk (forward)
    int64_t ncc, rowsc;              // column-kernel chunks and rows per chunk
    int64_t col_blocks;              // column-kernel blocks per chunk
    int64_t row_blocks;              // row-kernel blocks
    int64_t rr;                      // row kernel: ranges of pair rows m (m = r mod rr)
    int64_t cr;                      // column kernel: ranges of partners m'
    bool pairs;                      // gradients by grad_pairs_kernel (Z table fits in LDS)
    bool psym;                       // ... in its symmetric form (one workgroup spans all of M)
    bool pslots;                     // ... with R rows at a time (grad_pairs_slots_kernel)
    int prs, psthreads;              // its rows at a time and threads per workgroup
    int pthreads;                    // pairs kernel: threads (inducing inputs) per workgroup
    int64_t pmb, pchunks, prows;     // pairs kernel: m-blocks, row chunks, rows per chunk
    bool wide;                       // gradients by grad_wide_kernel (wider Q, Z table in LDS)
    int wqh;                         // its dimensions per lane
    int64_t wmb, wchunks, wrows;     // its blocks of 128 inducing inputs, row chunks, rows
    // workspace offsets in bytes
    size_t off_w1, off_w2, off_lp1, off_lp2, off_p2, off_g2s, off_gc, off_colp, off_rowp, off_rowg,
        total;
};

Plan make_plan(const Shape &s, size_t elem) {
    Plan p{};
    p.tiles_edge = cdiv(s.M, kPairTile);
    p.pblocks = cdiv(s.P, 256 * fwd_ppt(s.Q, elem));
    int64_t nc2 = cdiv(s.N, 256);
    int64_t cap2 = std::max<int64_t>(1, 2048 / p.pblocks);
    p.nc2 = std::max<int64_t>(1, std::min(nc2, cap2));
    p.rows2 = cdiv(s.N, p.nc2);
    p.nc2 = cdiv(s.N, p.rows2);
    p.col_blocks = cdiv(s.M, kColBlock);
    int64_t ncc = cdiv(s.N, 64);
    int64_t capc = std::max<int64_t>(1, 2048 / p.col_blocks);
    p.ncc = std::max<int64_t>(1, std::min(ncc, capc));
    p.rowsc = cdiv(s.N, p.ncc);
    p.ncc = cdiv(s.N, p.rowsc);
    p.row_blocks = cdiv(s.N, kRowBlock);
    p.rr = std::max<int64_t>(1, std::min<int64_t>(std::min<int64_t>(s.M, 64), cdiv(2048, p.row_blocks)));
    p.cr = std::max<int64_t>(1, std::min<int64_t>(std::min<int64_t>(s.M, 64),
                                                  cdiv(2048, p.col_blocks * p.ncc)));
    // the pairs kernel keeps the whole Z table (padded to QM) in LDS and a dozen
    // per-dimension values per thread in registers: small Q only (beyond that
    // it spills and the row and column kernels below take over)
    p.pairs = pairs_qm(s.Q) <= (elem == 4 ? 8 : 4) && s.M * pairs_qm(s.Q) * elem <= 65536;
    p.pthreads = (int)std::min<int64_t>(256, cdiv(s.M, 64) * 64);
    p.pmb = cdiv(s.M, p.pthreads);
    p.pchunks = std::max<int64_t>(1, std::min<int64_t>(s.N, 2048 / p.pmb));
    p.prows = cdiv(s.N, p.pchunks);
    p.pchunks = cdiv(s.N, p.prows);
    // symmetric form: every pair exchange stays inside one workgroup, and the Z
    // table plus two bands of kBand x M pair values fit in LDS
    p.psym = p.pairs && p.pmb == 1 && (pairs_qm(s.Q) + 2 * kBand) * s.M * elem <= 65536;
    p.prs = (int)std::min<int64_t>(8, 512 / s.M);
    p.psthreads = (int)(cdiv(p.prs * s.M, 64) * 64);
    p.pslots = p.psym && p.prs >= 2 &&
               (s.M * pairs_qm(s.Q) + p.prs * 2 * kSlotBand * s.M + p.prs * s.M * 2 * pairs_qm(s.Q)) * elem <=
                   65536;
    if (p.pslots) {
        // chunks a whole number of passes of R rows, about five rounds of two
        // 512-thread workgroups per CU
        p.pchunks = std::max<int64_t>(1, std::min<int64_t>(s.N, 2560));
        p.prows = cdiv(cdiv(s.N, p.pchunks), p.prs) * p.prs;
        p.pchunks = cdiv(s.N, p.prows);
    }
    // wide form: where the pairs kernel does not apply and the padded Z table
    // fits in LDS
    p.wqh = wide_qh(s.Q, elem);
    p.wide = !p.pairs && p.wqh > 0 && (s.M + 128) * 2 * p.wqh * elem <= 65536;
    p.wmb = cdiv(s.M, 128);
    p.wchunks = std::max<int64_t>(1, std::min<int64_t>(s.N, 2048 / p.wmb));
    p.wrows = cdiv(s.N, p.wchunks);
    p.wchunks = cdiv(s.N, p.wrows);
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
    p.off_w1 = take(elem * s.N * s.Q);
    p.off_w2 = take(elem * s.N * s.Q);
    p.off_lp1 = take(elem * s.N);
    p.off_lp2 = take(elem * s.N);
    p.off_p2 = take(elem * p.nc2 * s.P);
    p.off_g2s = take(elem * s.M * s.M);
    p.off_gc = take(elem * (s.M / 2 + 1) * s.M);
    p.off_colp = take(elem * std::max({p.ncc * p.cr, p.pchunks, p.wchunks}) * s.M * s.Q);
    p.off_rowp =
        take(elem * std::max({p.rr * p.row_blocks, p.pmb * p.pchunks, p.wmb * p.wchunks}) * (s.Q + 1));
    p.off_rowg = take(elem * std::max({p.rr, p.pmb, p.wmb}) * s.N * s.Q * 2);
    p.total = o;
    return p;
}

template <typename T>
T *at(void *ws, size_t off) { return reinterpret_cast<T *>(static_cast<char *>(ws) + off); }

// ---------------------------------------------------------------- per-row tables
template <typename T>
__global__ void rows_pre_kernel(const int *__restrict__ gate, int64_t N, int Q, const T *__restrict__ S, Hyp<T> h,
                                T *__restrict__ w1, T *__restrict__ w2, T *__restrict__ lp1,
                                T *__restrict__ lp2) {
    if (gate && gate[0] == 0) return;
    int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= N) return;
    T a = h.log_sf2, b = T(2) * h.log_sf2;
    for (int q = 0; q < Q; ++q) {
        T s = S[n * Q + q];
        T l2 = h.l2[q];
        w1[n * Q + q] = T(1) / (l2 + s);
        w2[n * Q + q] = T(1) / (l2 + T(2) * s);
        a -= T(0.5) * dlog1p(s / l2);
        b -= T(0.5) * dlog1p(T(2) * s / l2);
    }
    lp1[n] = a;
    lp2[n] = b;
}

// ---------------------------------------------------------------- Psi1 (Alg. 1, Psi)
template <typename T>
__global__ void psi1_kernel(const int *__restrict__ gate, int64_t N, int M, int Q, const T *__restrict__ mu,
                            const T *__restrict__ Z, const T *__restrict__ w1,
                            const T *__restrict__ lp1, T *__restrict__ Psi1) {
    if (gate && gate[0] == 0) return;
    // grid-stride over the N x M entries (the grid is capped, so that a call
    // whose gate is closed dispatches few workgroups)
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N * M;
         i += (int64_t)gridDim.x * blockDim.x) {
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
        T s = 0;
        for (int q = 0; q < Q; ++q) {
            T d = mu[n * Q + q] - Z[(int64_t)m * Q + q];
            s += d * d * w1[n * Q + q];
        }
        Psi1[i] = dexp(lp1[n] - T(0.5) * s);
    }
}

__device__ inline int64_t pair_index(int64_t m, int64_t mp, int64_t M) {
    return m * M - m * (m - 1) / 2 + (mp - m);
}

// Inverse of pair_index: the pair (m, mp), m <= mp, at position t < M (M + 1) / 2
// of the row-major upper triangle.  Row m starts at m (2M - m + 1) / 2; the
// square-root estimate of m is corrected by exact integer tests.
__device__ inline void pair_coords(int64_t t, int64_t M, int &m, int &mp) {
    auto start = [&](int64_t r) { return r * (2 * M - r + 1) / 2; };
    const double b = 2.0 * (double)M + 1.0;
    int64_t r = (int64_t)((b - sqrt(fmax(b * b - 8.0 * (double)t, 0.0))) * 0.5);
    r = r < 0 ? 0 : (r >= M ? M - 1 : r);
    while (r > 0 && start(r) > t) --r;
    while (r + 1 < M && start(r + 1) <= t) ++r;
    m = (int)r;
    mp = (int)(r + (t - start(r)));
}

// ---------------------------------------------------------------- Psi2 partials (Alg. 1, Phi)
// One thread per PPT unique pairs (pairs t = block base + k 256 + thread,
// k < PPT: consecutive pairs of the row-major upper triangle, so no lane idles
// below the diagonal) and row chunk.  The rows' (mu, w2) are staged in LDS as
// pairs, one read per (row, dimension) serving the thread's PPT pairs.
template <typename T>
struct Two;
template <>
struct Two<float> {
    typedef float2 t;
};
template <>
struct Two<double> {
    typedef double2 t;
};

template <typename T, int QM, int PPT>
__global__ __launch_bounds__(256) void psi2_partial_kernel(const int *__restrict__ gate,
    int64_t N, int M, int Q, int64_t P, int64_t rows_per_chunk,
    const T *__restrict__ mu, const T *__restrict__ Z, const T *__restrict__ w2,
    const T *__restrict__ lp2, Hyp<T> h, T *__restrict__ partial) {
    if (gate && gate[0] == 0) return;
    using T2 = typename Two<T>::t;
    __shared__ T2 s_mw[kFwdTile][QM];
    __shared__ T s_lp[kFwdTile];
    const int64_t t0 = (int64_t)blockIdx.x * 256 * PPT + threadIdx.x;
    // loads from clamped (valid) addresses, masked by a multiplication: a select
    // around each load would let the compiler wait for the loads one at a time
    T zbar[PPT][QM], C[PPT];
    bool valid[PPT];
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
        const int64_t t = t0 + k * 256;
        valid[k] = t < P;
        int m = 0, mp = 0;
        if (valid[k]) pair_coords(t, M, m, mp);
        C[k] = 0;
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            const int qc = min(q, Q - 1);
            const T a = Z[(int64_t)m * Q + qc], b = Z[(int64_t)mp * Q + qc];
            const T on = q < Q ? T(1) : T(0);
            zbar[k][q] = on * (T(0.5) * (a + b));
            C[k] -= on * ((a - b) * (a - b) / (T(4) * h.l2[qc]));
        }
    }
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    T acc[PPT];
#pragma unroll
    for (int k = 0; k < PPT; ++k) acc[k] = 0;
    for (int64_t base = r0; base < r1; base += kFwdTile) {
        const int cnt = (int)min<int64_t>(kFwdTile, r1 - base);
        __syncthreads();
        // zero beyond Q, so that the padded dimensions need no test below; four
        // entries per thread have their loads in flight together
        for (int i0 = threadIdx.x; i0 < cnt * QM; i0 += 4 * blockDim.x) {
            T a[4], b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = min(i0 + u * (int)blockDim.x, cnt * QM - 1);
                const int r = i / QM, q = min(i - r * QM, Q - 1);
                a[u] = mu[(base + r) * Q + q];
                b[u] = w2[(base + r) * Q + q];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + u * (int)blockDim.x;
                const int r = i / QM, q = i - r * QM;
                if (i < cnt * QM) {
                    T2 v;
                    v.x = q < Q ? a[u] : T(0);
                    v.y = q < Q ? b[u] : T(0);
                    s_mw[r][q] = v;
                }
            }
        }
        for (int r = threadIdx.x; r < cnt; r += blockDim.x) s_lp[r] = lp2[base + r];
        __syncthreads();
        // two-level sum: the tile's rows first, then into the chunk total, so
        // that rounding grows with tile + tiles per chunk, not rows per chunk
        T tacc[PPT];
#pragma unroll
        for (int k = 0; k < PPT; ++k) tacc[k] = 0;
#pragma unroll 4
        for (int r = 0; r < cnt; ++r) {
            T e[PPT];
#pragma unroll
            for (int k = 0; k < PPT; ++k) e[k] = s_lp[r] + C[k];
#pragma unroll
            for (int q = 0; q < QM; ++q) {
                const T2 v = s_mw[r][q];
#pragma unroll
                for (int k = 0; k < PPT; ++k) {
                    const T d = v.x - zbar[k][q];
                    e[k] -= d * d * v.y;
                }
            }
#pragma unroll
            for (int k = 0; k < PPT; ++k) tacc[k] += dexp(e[k]);
        }
#pragma unroll
        for (int k = 0; k < PPT; ++k) acc[k] += tacc[k];
    }
#pragma unroll
    for (int k = 0; k < PPT; ++k)
        if (valid[k]) partial[(int64_t)blockIdx.y * P + t0 + k * 256] = acc[k];
}

// Fixed-order sum of the chunk partials; writes both triangles and psi0.
template <typename T>
__global__ void psi2_reduce_kernel(const int *__restrict__ gate, int64_t N, int M, int64_t P, int64_t nchunks,
                                   const T *__restrict__ partial, Hyp<T> h, T *__restrict__ psi0,
                                   T *__restrict__ Psi2, int accumulate) {
    if (gate && gate[0] == 0) return;
    const int mp = blockIdx.x * kPairTile + threadIdx.x % kPairTile;
    const int m = blockIdx.y * kPairTile + threadIdx.x / kPairTile;
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
        psi0[0] = (accumulate ? psi0[0] : T(0)) + T(N) * h.sf2;
    if (m >= M || mp >= M || m > mp) return;
    const int64_t p = pair_index(m, mp, M);
    // chunk order; loads issued 16 at a time so that they overlap
    T s = 0;
    int64_t c = 0;
    for (; c + 16 <= nchunks; c += 16) {
        T v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = partial[(c + j) * P + p];
#pragma unroll
        for (int j = 0; j < 16; ++j) s += v[j];
    }
    for (; c < nchunks; ++c) s += partial[c * P + p];
    T v = (accumulate ? Psi2[(int64_t)m * M + mp] : T(0)) + s;
    Psi2[(int64_t)m * M + mp] = v;
    Psi2[(int64_t)mp * M + m] = v;
}

// ---------------------------------------------------------------- gradients (Alg. 2)
template <typename T>
__global__ void sym_kernel(const int *__restrict__ gate, int M, const T *__restrict__ G2, T *__restrict__ G2s) {
    if (gate && gate[0] == 0) return;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)M * M) return;
    int m = (int)(i / M), mp = (int)(i - (int64_t)m * M);
    G2s[i] = T(0.5) * (G2[(int64_t)m * M + mp] + G2[(int64_t)mp * M + m]);
}

// Gc[k][m] = G2s[m][(m + k) mod M], k = 0 .. M/2: the symmetric pairs kernel
// reads the pair (m, m + k) of every thread m as one coalesced row.
template <typename T>
__global__ void circ_kernel(const int *__restrict__ gate, int M, const T *__restrict__ G2s, T *__restrict__ Gc) {
    if (gate && gate[0] == 0) return;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)(M / 2 + 1) * M) return;
    const int k = (int)(i / M), m = (int)(i - (int64_t)k * M);
    int mp = m + k;
    if (mp >= M) mp -= M;
    Gc[i] = G2s[(int64_t)m * M + mp];
}

// One thread per datapoint and range r of pair rows (m = r, r + rr, ...; the
// Psi1 terms in the column tiles t = r, r + rr, ...): partial dmu_n, dS_n of the
// range (rowg[r][2][N][Q]) and per-block partials of dl and dsf2.
template <typename T, int QM>
__global__ __launch_bounds__(kRowBlock) void grad_rows_kernel(const int *__restrict__ gate, 
    int64_t N, int M, int Q, int rr, const T *__restrict__ mu, const T *__restrict__ S,
    const T *__restrict__ Z, const T *__restrict__ w1, const T *__restrict__ w2,
    const T *__restrict__ lp1, const T *__restrict__ lp2, Hyp<T> h, const T *__restrict__ G1,
    const T *__restrict__ G2s, T *__restrict__ rowg, T *__restrict__ rowpart) {
    if (gate && gate[0] == 0) return;
    const int range = blockIdx.y;
    __shared__ T s_g1[kRowBlock][kRowBlock + 1];
    __shared__ T s_red[QM + 1][kRowBlock];
    const int tid = threadIdx.x;
    const int64_t n0 = (int64_t)blockIdx.x * kRowBlock;
    const int64_t n = n0 + tid;
    const bool valid = n < N;
    T m_[QM], s_[QM], a1[QM], a2[QM];
    T gmu[QM], gS[QM], gl[QM];
    T l1 = 0, l2v = 0, gsf = 0;
#pragma unroll
    for (int q = 0; q < QM; ++q) {
        m_[q] = s_[q] = a1[q] = a2[q] = gmu[q] = gS[q] = gl[q] = 0;
        if (q < Q && valid) {
            m_[q] = mu[n * Q + q];
            s_[q] = S[n * Q + q];
            a1[q] = w1[n * Q + q];
            a2[q] = w2[n * Q + q];
        }
    }
    if (valid) { l1 = lp1[n]; l2v = lp2[n]; }

    if (G1) {
        const int rows = (int)min<int64_t>(kRowBlock, N - n0);
        for (int mt = range * kRowBlock; mt < M; mt += rr * kRowBlock) {
            const int cols = min(kRowBlock, M - mt);
            __syncthreads();
            for (int i = tid; i < rows * cols; i += kRowBlock) {
                int r = i / cols, c = i - r * cols;
                s_g1[r][c] = G1[(n0 + r) * M + mt + c];
            }
            __syncthreads();
            if (valid) {
                for (int c = 0; c < cols; ++c) {
                    const int m = mt + c;
                    T e = 0;
#pragma unroll
                    for (int q = 0; q < QM; ++q)
                        if (q < Q) {
                            T d = m_[q] - Z[(int64_t)m * Q + q];
                            e += d * d * a1[q];
                        }
                    const T t = s_g1[tid][c] * dexp(l1 - T(0.5) * e);
                    gsf += t;
#pragma unroll
                    for (int q = 0; q < QM; ++q)
                        if (q < Q) {
                            T d = m_[q] - Z[(int64_t)m * Q + q];
                            T dd = d * a1[q];
                            gmu[q] -= t * dd;
                            gS[q] += t * T(0.5) * (dd * dd - a1[q]);
                            gl[q] += t * (s_[q] * a1[q] / h.l[q] + h.l[q] * dd * dd);
                        }
                }
            }
        }
    }

    if (G2s && valid) {
        for (int m = range; m < M; m += rr) {
            T gsf_row = 0;  // sum over m' first, so long rows do not swamp the total
            for (int mp = m; mp < M; ++mp) {
                const T g = (m == mp ? T(1) : T(2)) * G2s[(int64_t)m * M + mp];
                T e = l2v;
#pragma unroll
                for (int q = 0; q < QM; ++q)
                    if (q < Q) {
                        T a = Z[(int64_t)m * Q + q], b = Z[(int64_t)mp * Q + q];
                        T d = m_[q] - T(0.5) * (a + b);
                        e -= (a - b) * (a - b) / (T(4) * h.l2[q]) + d * d * a2[q];
                    }
                const T t = g * dexp(e);
                gsf_row += T(2) * t;
#pragma unroll
                for (int q = 0; q < QM; ++q)
                    if (q < Q) {
                        T a = Z[(int64_t)m * Q + q], b = Z[(int64_t)mp * Q + q];
                        T d = m_[q] - T(0.5) * (a + b);
                        T dd = d * a2[q];
                        T del = a - b;
                        gmu[q] -= T(2) * t * dd;
                        gS[q] += t * (T(2) * dd * dd - a2[q]);
                        gl[q] += t * (T(2) * s_[q] * a2[q] / h.l[q] +
                                      del * del / (T(2) * h.l2[q] * h.l[q]) +
                                      T(2) * h.l[q] * dd * dd);
                    }
            }
            gsf += gsf_row;
        }
    }

    if (valid) {
        T *pm = rowg + ((int64_t)range * 2) * N * Q, *ps = pm + N * Q;
#pragma unroll
        for (int q = 0; q < QM; ++q)
            if (q < Q) {
                pm[n * Q + q] = gmu[q];
                ps[n * Q + q] = gS[q];
            }
    }
    // fixed-order block reduction of dl and dsf2 partials
    __syncthreads();
#pragma unroll
    for (int q = 0; q < QM; ++q) s_red[q][tid] = gl[q];
    s_red[QM][tid] = gsf / h.sf2;
    __syncthreads();
    for (int k = tid; k <= Q; k += kRowBlock) {
        const int row = k < Q ? k : QM;
        T s = 0;
        for (int i = 0; i < kRowBlock; ++i) s += s_red[row][i];
        rowpart[((int64_t)range * gridDim.x + blockIdx.x) * (Q + 1) + k] = s;
    }
}

// Psi2 and Psi1 gradients through per-(n, m) sums.  With W_n[m, m'] =
// G2s[m, m'] Psi2_n[m, m'], d = mu_n - z_m, w1 = 1/(l^2 + S_n), w2 = 1/(l^2 + 2 S_n),
//   r_nm = sum_m' W_n[m, m'],  V_nmq = sum_m' W_n[m, m'] d_nm'q,
//   t_nm = dL/dPsi1[n, m] Psi1[n, m],
// every gradient is a sum over (n, m) of (W is symmetric, so the double sum over
// ordered pairs folds onto the m index):
//   dmu_nq += -2 w2 d r - t d w1
//   dS_nq  += w2^2 (d^2 r + d V) - w2 r + t (d^2 w1^2 - w1) / 2
//   dZ_mq  += w2 (d r + V) - (V - d r) / l^2 + t d w1
//   dl_q   += (2 S w2 / l) r + (d^2 r - d V) / l^3 + l w2^2 (d^2 r + d V)
//             + t (S w1 / l + l d^2 w1^2)
//   dsf2   += (2 r + t) / sf2.
// One workgroup per (block of inducing inputs, row chunk), one thread per m, the
// Z table in LDS: dZ_m stays in the thread's registers over the chunk, and per
// row the dmu / dS contributions are summed over the block's m (wave
// butterflies, then the waves in order) into rowg[m-block][2][N][Q].
// Ordered form (SYM = false): thread m evaluates W for every (m, m').
// Symmetric form (SYM = true, the workgroup holds all M): each unordered pair
// is evaluated once.  Thread m takes the pairs (m, m + k mod M) for k = 0 ..
// M/2 (k = M/2 only for m < M/2 when M is even), so every thread has the same
// load; it adds W to its own r and V and leaves it in an LDS band, from which
// thread m + k adds it to its r and V.  The bands hold kBand offsets and are
// double buffered: one barrier per band.
template <typename T, int QM, bool SYM>
__global__ __launch_bounds__(256) void grad_pairs_kernel(const int *__restrict__ gate, 
    int64_t N, int M, int Q, int64_t rows_per_chunk, const T *__restrict__ mu,
    const T *__restrict__ S, const T *__restrict__ Z, const T *__restrict__ w1t,
    const T *__restrict__ w2t, const T *__restrict__ lp1, const T *__restrict__ lp2, Hyp<T> h,
    const T *__restrict__ G1, const T *__restrict__ G2s, const T *__restrict__ Gc,
    T *__restrict__ rowg, T *__restrict__ colpart, T *__restrict__ rowpart) {
    if (gate && gate[0] == 0) return;
    extern __shared__ double gp_smem[];
    T *sz = reinterpret_cast<T *>(gp_smem);  // [M][QM], zero beyond Q
    T *band = sz + M * QM;                    // [2][kBand][M] (symmetric form)
    __shared__ T red[2][4][2 * QM];           // per-wave row sums, double buffered by row
    const int tid = threadIdx.x, nthr = blockDim.x, nw = nthr >> 6, wv = tid >> 6;
    const int m = blockIdx.x * nthr + tid;
    const bool valid = m < M;
    for (int i = tid; i < M * QM; i += nthr) {
        const int mm = i / QM, q = i - mm * QM;
        sz[i] = q < Q ? Z[(int64_t)mm * Q + q] : T(0);
    }
    __syncthreads();
    T z[QM], c4[QM], il2[QM], gz[QM], gl[QM];
#pragma unroll
    for (int q = 0; q < QM; ++q) {
        z[q] = valid ? sz[m * QM + q] : T(0);
        c4[q] = q < Q ? T(0.25) / h.l2[q] : T(0);
        il2[q] = q < Q ? T(1) / h.l2[q] : T(0);
        gz[q] = gl[q] = 0;
    }
    T gsf = 0;
    const int K = M / 2;
    const bool even = (M & 1) == 0;
    const int Ku = even ? K - 1 : K;  // offsets taken by every thread
    int band_no = 0;
    const T gdiag = (SYM && valid) ? Gc[m] : T(0);  // G2s[m][m], the same for every row
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk, r1 = min(N, r0 + rows_per_chunk);
    for (int64_t n = r0; n < r1; ++n) {
        T x[QM], a1[QM], a2[QM], sv[QM], d[QM];
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            const bool in = q < Q;
            x[q] = in ? mu[n * Q + q] : T(0);
            a1[q] = in ? w1t[n * Q + q] : T(0);
            a2[q] = in ? w2t[n * Q + q] : T(0);
            sv[q] = in ? S[n * Q + q] : T(0);
            d[q] = x[q] - z[q];
        }
        T r = 0, V[QM];
#pragma unroll
        for (int q = 0; q < QM; ++q) V[q] = 0;
        // W_n[m, m'] = G2s[m, m'] Psi2_n[m, m'] for the partner m' (z row zr).
        // With v = z_m' - z_m and d = mu_n - z_m the exponent
        //   log Psi2 - log prefactor = -sum_q [c4 v^2 + (a2/4)(2 d - v)^2]
        // is a quadratic in v with per-(n, m) coefficients:
        //   e0 + sum_q v (a2 d - (c4 + a2/4) v),  e0 = lp2 - sum_q a2 d^2.
        // Where W is not negligible (exponent above about -30) each of its terms
        // is bounded by a few hundred, so the rounding stays near that of the
        // summed squares.
        T bq[QM], cq[QM], e0 = G2s ? lp2[n] : T(0);
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            bq[q] = a2[q] * d[q];
            cq[q] = c4[q] + T(0.25) * a2[q];
            e0 -= bq[q] * d[q];
        }
        auto pair_w = [&](const T *zr, T g, T e00) {
            T e = e00;
#pragma unroll
            for (int q = 0; q < QM; ++q) {
                const T v = zr[q] - z[q];
                e = fma(v, fma(-cq[q], v, bq[q]), e);
            }
            return g * dexp(e);
        };
        auto add_w = [&](T W, const T *zr) {
            r += W;
#pragma unroll
            for (int q = 0; q < QM; ++q) V[q] += W * (x[q] - zr[q]);
        };
        if (SYM) {
            if (G2s) {  // uniform: every thread reaches the band barriers
                if (valid) add_w(pair_w(sz + m * QM, gdiag, e0), sz + m * QM);
                // offsets every thread takes (1 .. Ku), in bands; then, for even
                // M, the offset M/2 of the first half
                for (int k0 = 1; k0 <= Ku; k0 += kBand, ++band_no) {
                    T *bs = band + (band_no & 1) * (kBand * M);
                    const int k1 = min(Ku, k0 + kBand - 1);
                    if (valid) {
                        int mp = m + k0;
                        if (mp >= M) mp -= M;
                        const T *gk = Gc + (int64_t)k0 * M + m;
#pragma unroll 2
                        for (int k = k0; k <= k1; ++k) {
                            const T W = pair_w(sz + mp * QM, *gk, e0);
                            add_w(W, sz + mp * QM);
                            bs[(k - k0) * M + m] = W;
                            gk += M;
                            mp = mp + 1 == M ? 0 : mp + 1;
                        }
                    }
                    __syncthreads();
                    if (valid) {
                        int sp = m - k0;
                        if (sp < 0) sp += M;
#pragma unroll 4
                        for (int k = k0; k <= k1; ++k) {
                            add_w(bs[(k - k0) * M + sp], sz + sp * QM);
                            sp = sp == 0 ? M - 1 : sp - 1;
                        }
                    }
                }
                if (even && K > 0) {
                    T *bs = band + (band_no & 1) * (kBand * M);
                    ++band_no;
                    if (valid && m < K) {
                        const T W = pair_w(sz + (m + K) * QM, Gc[(int64_t)K * M + m], e0);
                        add_w(W, sz + (m + K) * QM);
                        bs[m] = W;
                    }
                    __syncthreads();
                    if (valid && m >= K) add_w(bs[m - K], sz + (m - K) * QM);
                }
            }
        } else if (G2s && valid) {
            for (int mp = 0; mp < M; ++mp)  // G2s symmetric: G2s[mp][m] is a coalesced row
                add_w(pair_w(sz + mp * QM, G2s[(int64_t)mp * M + m], e0), sz + mp * QM);
        }
        T t = 0;
        if (G1 && valid) {
            T e1 = 0;
#pragma unroll
            for (int q = 0; q < QM; ++q) e1 += d[q] * d[q] * a1[q];
            t = G1[n * M + m] * dexp(lp1[n] - T(0.5) * e1);
        }
        T rv[2 * QM];
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            const T dq = d[q], d2 = dq * dq, dr = dq * r, dV = dq * V[q];
            rv[q] = -T(2) * a2[q] * dr - t * dq * a1[q];
            rv[QM + q] = a2[q] * a2[q] * (d2 * r + dV) - a2[q] * r +
                         T(0.5) * t * (d2 * a1[q] * a1[q] - a1[q]);
            gz[q] += a2[q] * (dr + V[q]) - (V[q] - dr) * il2[q] + t * dq * a1[q];
            if (q < Q) {
                const T l = h.l[q];
                gl[q] += (T(2) * sv[q] * a2[q] / l) * r + (d2 * r - dV) * il2[q] / l +
                         l * a2[q] * a2[q] * (d2 * r + dV) +
                         t * (sv[q] * a1[q] / l + l * d2 * a1[q] * a1[q]);
            }
        }
        gsf += T(2) * r + t;
        // sum of rv over the block's m: butterflies within each wave, then the
        // waves in order (double buffered by row parity: one barrier per row)
        const int b = (int)(n & 1);
#pragma unroll
        for (int k = 0; k < 2 * QM; ++k) {
            T v = rv[k];
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
            if ((tid & 63) == 0) red[b][wv][k] = v;
        }
        __syncthreads();
        if (tid < 2 * Q) {
            const int k = tid < Q ? tid : QM + (tid - Q);
            T v = 0;
            for (int w = 0; w < nw; ++w) v += red[b][w][k];
            const int part = tid < Q ? 0 : 1, q = tid < Q ? tid : tid - Q;
            rowg[(((int64_t)blockIdx.x * 2 + part) * N + n) * Q + q] = v;
        }
    }
    if (valid) {
#pragma unroll
        for (int q = 0; q < QM; ++q)
            if (q < Q) colpart[((int64_t)blockIdx.y * M + m) * Q + q] = gz[q];
    }
    // block sums of dl and dsf2 (fixed order, as above) -> rowpart[block][Q + 1]
    const int64_t blk = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
    __syncthreads();
#pragma unroll
    for (int k = 0; k <= QM; ++k) {
        if (k < Q || k == QM) {
            T v = k < QM ? gl[k] : gsf / h.sf2;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
            if ((tid & 63) == 0) red[0][wv][0] = v;
            __syncthreads();
            if (tid == 0) {
                T s = 0;
                for (int w = 0; w < nw; ++w) s += red[0][w][0];
                rowpart[blk * (Q + 1) + (k < QM ? k : Q)] = s;
            }
            __syncthreads();
        }
    }
}

// The band form with R = min(8, 512 / M) rows at a time, so that a workgroup
// of R M threads (rounded up to whole waves) leaves few lanes idle when M is
// not a multiple of 64.  Thread (slot, m) = (tid / M, tid % M) works on row
// r0 + it R + slot of pass it; each slot exchanges W through its own double
// buffered band of kSlotBand offsets.  Per row the dmu / dS terms are summed
// over m through LDS (32 lanes per output, each adding m = u, u + 32, ... in
// order, then a fixed butterfly); dZ_m adds the slots in order at the end.

template <typename T, int QM>
__global__ __launch_bounds__(512) void grad_pairs_slots_kernel(const int *__restrict__ gate, 
    int64_t N, int M, int Q, int R, int64_t rows_per_chunk, const T *__restrict__ mu,
    const T *__restrict__ S, const T *__restrict__ Z, const T *__restrict__ w1t,
    const T *__restrict__ w2t, const T *__restrict__ lp1, const T *__restrict__ lp2, Hyp<T> h,
    const T *__restrict__ G1, const T *__restrict__ G2s, const T *__restrict__ Gc,
    T *__restrict__ rowg, T *__restrict__ colpart, T *__restrict__ rowpart) {
    if (gate && gate[0] == 0) return;
    extern __shared__ double gs_smem[];
    T *sz = reinterpret_cast<T *>(gs_smem);        // [M][QM], zero beyond Q
    T *band = sz + M * QM;                          // [R][2][kSlotBand][M]
    T *rvs = band + (size_t)R * 2 * kSlotBand * M;  // [R M][2 QM]: row terms, then dZ by slot
    __shared__ T redw[8];
    const int tid = threadIdx.x, nthr = blockDim.x, nw = nthr >> 6, wv = tid >> 6;
    const int slot = tid / M, m = tid - slot * M;
    const bool valid = slot < R;
    for (int i = tid; i < M * QM; i += nthr) {
        const int mm = i / QM, q = i - mm * QM;
        sz[i] = q < Q ? Z[(int64_t)mm * Q + q] : T(0);
    }
    __syncthreads();
    T z[QM], c4[QM], il2[QM], gz[QM], gl[QM];
#pragma unroll
    for (int q = 0; q < QM; ++q) {
        z[q] = valid ? sz[m * QM + q] : T(0);
        c4[q] = q < Q ? T(0.25) / h.l2[q] : T(0);
        il2[q] = q < Q ? T(1) / h.l2[q] : T(0);
        gz[q] = gl[q] = 0;
    }
    T gsf = 0;
    const int K = M / 2;
    const bool even = (M & 1) == 0;
    const int Ku = even ? K - 1 : K;  // offsets taken by every thread
    int band_no = 0;
    const T gdiag = valid ? Gc[m] : T(0);
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk, r1 = min(N, r0 + rows_per_chunk);
    const int64_t iters = (r1 - r0 + R - 1) / R;
    for (int64_t it = 0; it < iters; ++it) {
        const int64_t n = r0 + it * R + slot;
        const bool rin = valid && n < r1;
        T x[QM], a1[QM], a2[QM], sv[QM], d[QM];
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            const bool in = rin && q < Q;
            x[q] = in ? mu[n * Q + q] : T(0);
            a1[q] = in ? w1t[n * Q + q] : T(0);
            a2[q] = in ? w2t[n * Q + q] : T(0);
            sv[q] = in ? S[n * Q + q] : T(0);
            d[q] = x[q] - z[q];
        }
        T r = 0, V[QM];
#pragma unroll
        for (int q = 0; q < QM; ++q) V[q] = 0;
        // the exponent as a quadratic in v = z_m' - z_m (as in grad_pairs_kernel)
        T bq[QM], cq[QM], e0 = (G2s && rin) ? lp2[n] : T(0);
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            bq[q] = a2[q] * d[q];
            cq[q] = c4[q] + T(0.25) * a2[q];
            e0 -= bq[q] * d[q];
        }
        auto pair_w = [&](const T *zr, T g) {
            T e = e0;
#pragma unroll
            for (int q = 0; q < QM; ++q) {
                const T v = zr[q] - z[q];
                e = fma(v, fma(-cq[q], v, bq[q]), e);
            }
            return g * dexp(e);
        };
        auto add_w = [&](T W, const T *zr) {
            r += W;
#pragma unroll
            for (int q = 0; q < QM; ++q) V[q] += W * (x[q] - zr[q]);
        };
        if (G2s) {  // uniform: every thread reaches the band barriers
            if (rin) add_w(pair_w(sz + m * QM, gdiag), sz + m * QM);
            for (int k0 = 1; k0 <= Ku; k0 += kSlotBand, ++band_no) {
                T *bs = band + ((size_t)slot * 2 + (band_no & 1)) * (kSlotBand * M);
                const int k1 = min(Ku, k0 + kSlotBand - 1);
                if (rin) {
                    int mp = m + k0;
                    if (mp >= M) mp -= M;
                    const T *gk = Gc + (int64_t)k0 * M + m;
#pragma unroll 2
                    for (int k = k0; k <= k1; ++k) {
                        const T W = pair_w(sz + mp * QM, *gk);
                        add_w(W, sz + mp * QM);
                        bs[(k - k0) * M + m] = W;
                        gk += M;
                        mp = mp + 1 == M ? 0 : mp + 1;
                    }
                }
                __syncthreads();
                if (rin) {
                    int sp = m - k0;
                    if (sp < 0) sp += M;
#pragma unroll 4
                    for (int k = k0; k <= k1; ++k) {
                        add_w(bs[(k - k0) * M + sp], sz + sp * QM);
                        sp = sp == 0 ? M - 1 : sp - 1;
                    }
                }
            }
            if (even && K > 0) {
                T *bs = band + ((size_t)slot * 2 + (band_no & 1)) * (kSlotBand * M);
                ++band_no;
                if (rin && m < K) {
                    const T W = pair_w(sz + (m + K) * QM, Gc[(int64_t)K * M + m]);
                    add_w(W, sz + (m + K) * QM);
                    bs[m] = W;
                }
                __syncthreads();
                if (rin && m >= K) add_w(bs[m - K], sz + (m - K) * QM);
            }
        }
        T rv[2 * QM];
#pragma unroll
        for (int k = 0; k < 2 * QM; ++k) rv[k] = 0;
        if (rin) {
            T t = 0;
            if (G1) {
                T e1 = 0;
#pragma unroll
                for (int q = 0; q < QM; ++q) e1 += d[q] * d[q] * a1[q];
                t = G1[n * M + m] * dexp(lp1[n] - T(0.5) * e1);
            }
#pragma unroll
            for (int q = 0; q < QM; ++q) {
                const T dq = d[q], d2 = dq * dq, dr = dq * r, dV = dq * V[q];
                rv[q] = -T(2) * a2[q] * dr - t * dq * a1[q];
                rv[QM + q] = a2[q] * a2[q] * (d2 * r + dV) - a2[q] * r +
                             T(0.5) * t * (d2 * a1[q] * a1[q] - a1[q]);
                gz[q] += a2[q] * (dr + V[q]) - (V[q] - dr) * il2[q] + t * dq * a1[q];
                if (q < Q) {
                    const T l = h.l[q];
                    gl[q] += (T(2) * sv[q] * a2[q] / l) * r + (d2 * r - dV) * il2[q] / l +
                             l * a2[q] * a2[q] * (d2 * r + dV) +
                             t * (sv[q] * a1[q] / l + l * d2 * a1[q] * a1[q]);
                }
            }
            gsf += T(2) * r + t;
        }
        if (valid) {
#pragma unroll
            for (int k = 0; k < 2 * QM; ++k) rvs[(size_t)tid * 2 * QM + k] = rv[k];
        }
        __syncthreads();
        {
            const int g = tid >> 5, u = tid & 31, outs = R * 2 * Q;
            for (int o = g; o < outs; o += nthr >> 5) {
                const int sl = o / (2 * Q), j = o - sl * 2 * Q;
                const int kk = j < Q ? j : QM + (j - Q);
                T v = 0;
                for (int mm = u; mm < M; mm += 32) v += rvs[((size_t)sl * M + mm) * 2 * QM + kk];
#pragma unroll
                for (int off = 16; off >= 1; off >>= 1) v += __shfl_xor(v, off);
                const int64_t nn = r0 + it * R + sl;
                if (u == 0 && nn < r1) {
                    const int part = j < Q ? 0 : 1, q = j < Q ? j : j - Q;
                    rowg[((int64_t)part * N + nn) * Q + q] = v;
                }
            }
        }
        __syncthreads();  // rvs is written again in the next pass
    }
    // dZ_m: the slots in order -> colpart[chunk][m][q]
    if (valid) {
#pragma unroll
        for (int q = 0; q < QM; ++q) rvs[((size_t)slot * M + m) * QM + q] = gz[q];
    }
    __syncthreads();
    if (tid < M) {
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            if (q < Q) {
                T v = 0;
                for (int sl = 0; sl < R; ++sl) v += rvs[((size_t)sl * M + tid) * QM + q];
                colpart[((int64_t)blockIdx.y * M + tid) * Q + q] = v;
            }
        }
    }
    // block sums of dl and dsf2 (wave butterflies, then the waves in order) ->
    // rowpart[chunk][Q + 1]
    const int64_t blk = blockIdx.y;
#pragma unroll
    for (int k = 0; k <= QM; ++k) {
        if (k < Q || k == QM) {
            T v = k < QM ? gl[k] : gsf / h.sf2;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
            __syncthreads();
            if ((tid & 63) == 0) redw[wv] = v;
            __syncthreads();
            if (tid == 0) {
                T s2 = 0;
                for (int w = 0; w < nw; ++w) s2 += redw[w];
                rowpart[blk * (Q + 1) + (k < QM ? k : Q)] = s2;
            }
        }
    }
}

// dmu, dS: the row kernel's range partials summed in range order.
template <typename T>
__global__ void grad_rows_reduce_kernel(const int *__restrict__ gate, int64_t NQ, int rr, const T *__restrict__ rowg,
                                        T *__restrict__ dmu, T *__restrict__ dS) {
    if (gate && gate[0] == 0) return;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < NQ;
         i += (int64_t)gridDim.x * blockDim.x) {
        T a = 0, b = 0;
        for (int r = 0; r < rr; ++r) {
            a += rowg[(int64_t)(2 * r) * NQ + i];
            b += rowg[(int64_t)(2 * r + 1) * NQ + i];
        }
        dmu[i] = a;
        dS[i] = b;
    }
}

// One thread per inducing input m, row chunk and range of partners (m' = r,
// r + cr, ...; the Psi1 term in range 0): partial dZ[m, :] per (chunk, range).
template <typename T, int QM>
__global__ __launch_bounds__(kColBlock) void grad_cols_kernel(const int *__restrict__ gate, 
    int64_t N, int M, int Q, int cr, int64_t rows_per_chunk, const T *__restrict__ mu,
    const T *__restrict__ Z, const T *__restrict__ w1, const T *__restrict__ w2,
    const T *__restrict__ lp1, const T *__restrict__ lp2, Hyp<T> h, const T *__restrict__ G1,
    const T *__restrict__ G2s, T *__restrict__ colpart) {
    if (gate && gate[0] == 0) return;
    __shared__ T s_mu[kRowTile][QM];
    __shared__ T s_w1[kRowTile][QM];
    __shared__ T s_w2[kRowTile][QM];
    __shared__ T s_lp1[kRowTile], s_lp2[kRowTile];
    const int m = blockIdx.x * kColBlock + threadIdx.x;
    const bool valid = m < M;
    T zm[QM], gz[QM];
#pragma unroll
    for (int q = 0; q < QM; ++q) {
        gz[q] = 0;
        zm[q] = (q < Q && valid) ? Z[(int64_t)m * Q + q] : T(0);
    }
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    for (int64_t base = r0; base < r1; base += kRowTile) {
        const int cnt = (int)min<int64_t>(kRowTile, r1 - base);
        __syncthreads();
        for (int i = threadIdx.x; i < cnt * Q; i += blockDim.x) {
            int r = i / Q, q = i - r * Q;
            s_mu[r][q] = mu[(base + r) * Q + q];
            s_w1[r][q] = w1[(base + r) * Q + q];
            s_w2[r][q] = w2[(base + r) * Q + q];
        }
        for (int r = threadIdx.x; r < cnt; r += blockDim.x) {
            s_lp1[r] = lp1[base + r];
            s_lp2[r] = lp2[base + r];
        }
        __syncthreads();
        if (!valid) continue;
        for (int r = 0; r < cnt; ++r) {
            if (G1 && blockIdx.z == 0) {
                T e = 0;
#pragma unroll
                for (int q = 0; q < QM; ++q)
                    if (q < Q) {
                        T d = s_mu[r][q] - zm[q];
                        e += d * d * s_w1[r][q];
                    }
                const T t = G1[(base + r) * M + m] * dexp(s_lp1[r] - T(0.5) * e);
#pragma unroll
                for (int q = 0; q < QM; ++q)
                    if (q < Q) gz[q] += t * (s_mu[r][q] - zm[q]) * s_w1[r][q];
            }
            if (G2s) {
                // two-level sum: the row's partners first, then into the chunk total
                // (the 64-wide variant, already short of registers, adds directly)
                constexpr bool kTwo = QM <= 32;
                T gzr_[kTwo ? QM : 1];
                T *gzr = kTwo ? gzr_ : gz;
                if constexpr (kTwo) {
#pragma unroll
                    for (int q = 0; q < QM; ++q) gzr[q] = 0;
                }
                for (int mp = blockIdx.z; mp < M; mp += cr) {
                    const T g = G2s[(int64_t)mp * M + m];
                    T e = s_lp2[r];
#pragma unroll
                    for (int q = 0; q < QM; ++q)
                        if (q < Q) {
                            T b = Z[(int64_t)mp * Q + q];
                            T d = s_mu[r][q] - T(0.5) * (zm[q] + b);
                            e -= (zm[q] - b) * (zm[q] - b) / (T(4) * h.l2[q]) +
                                 d * d * s_w2[r][q];
                        }
                    const T t = T(2) * g * dexp(e);
#pragma unroll
                    for (int q = 0; q < QM; ++q)
                        if (q < Q) {
                            T b = Z[(int64_t)mp * Q + q];
                            T d = s_mu[r][q] - T(0.5) * (zm[q] + b);
                            gzr[q] += t * (d * s_w2[r][q] - (zm[q] - b) / (T(2) * h.l2[q]));
                        }
                }
                if constexpr (kTwo) {
#pragma unroll
                    for (int q = 0; q < QM; ++q) gz[q] += gzr[q];
                }
            }
        }
    }
    if (valid) {
#pragma unroll
        for (int q = 0; q < QM; ++q)
            if (q < Q) colpart[(((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * M + m) * Q + q] = gz[q];
    }
}

// Fixed-order reduction of the gradient partials into dZ, dl, dsf2: one
// workgroup per output; thread t sums partials t, t + 256, ..., then a fixed
// tree combines the 256 sums.
template <typename T>
__global__ __launch_bounds__(256) void grad_reduce_kernel(const int *__restrict__ gate, int64_t N, int M, int Q, int64_t ncol,
                                                          int64_t nrow, const T *__restrict__ colpart,
                                                          const T *__restrict__ rowpart, T dL_dpsi0,
                                                          T *__restrict__ dZ, T *__restrict__ dsf2,
                                                          T *__restrict__ dl, int accumulate) {
    if (gate && gate[0] == 0) return;
    __shared__ T red[256];
    const int64_t MQ = (int64_t)M * Q;
    // outputs i = blockIdx.x, blockIdx.x + gridDim.x, ... (the grid is capped)
    for (int64_t i = blockIdx.x; i < MQ + Q + 1; i += gridDim.x) {
        T s = 0;
        if (i < MQ) {
            for (int64_t c = threadIdx.x; c < ncol; c += 256) s += colpart[c * MQ + i];
        } else {
            const int k = (int)(i - MQ);  // k < Q: dl_k; k == Q: dsf2
            for (int64_t b = threadIdx.x; b < nrow; b += 256) s += rowpart[b * (Q + 1) + k];
        }
        __syncthreads();
        red[threadIdx.x] = s;
        __syncthreads();
        for (int w = 128; w >= 1; w >>= 1) {
            if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
            __syncthreads();
        }
        if (threadIdx.x != 0) continue;
        s = red[0];
        if (i < MQ) {
            dZ[i] = (accumulate ? dZ[i] : T(0)) + s;
        } else if (i < MQ + Q) {
            dl[i - MQ] = (accumulate ? dl[i - MQ] : T(0)) + s;
        } else {
            s += dL_dpsi0 * T(N);
            dsf2[0] = (accumulate ? dsf2[0] : T(0)) + s;
        }
    }
}

// Wide form of the ordered pairs gradient, for Q past the pairs kernel's
// register budget (same outputs as grad_pairs_kernel with SYM = false: rowg,
// colpart, rowpart).  Two lanes of a wave share an inducing input m (lanes l
// and l + 32) and each holds QH of its dimensions (lane half hh takes
// q = hh QH .. hh QH + QH - 1), which halves the per-dimension registers (z,
// the exponent's coefficients, the V sums, the dZ and dl partials).  Per partner
// m' each lane forms its half of the exponent (the same quadratic in
// v = z_m' - z_m as the pairs kernel); the halves are exchanged across the lane
// pair and added in the same order on both lanes, so both evaluate the same
// W = G2s[m, m'] Psi2_n[m, m'] and update their own dimensions:
//   r += W,   Vd_q += W (z_m'q - z_mq)
// (the local differences, not W z_m'q, so that no sum of the size of |z| r
// cancels in the dZ and dl terms; V = d r - Vd).
// Row values are read from clamped addresses and masked, so that their loads
// issue together.  One workgroup per (block of 128 inducing inputs, row chunk).
template <typename T, int QH>
__global__ __launch_bounds__(256) void grad_wide_kernel(const int *__restrict__ gate,
    int64_t N, int M, int Q, int64_t rows_per_chunk, const T *__restrict__ mu,
    const T *__restrict__ S, const T *__restrict__ Z, const T *__restrict__ w1t,
    const T *__restrict__ w2t, const T *__restrict__ lp1, const T *__restrict__ lp2, Hyp<T> h,
    const T *__restrict__ G1, const T *__restrict__ G2s, T *__restrict__ rowg,
    T *__restrict__ colpart, T *__restrict__ rowpart) {
    if (gate && gate[0] == 0) return;
    constexpr int QM = 2 * QH;
    extern __shared__ double gw_smem[];
    T *sz = reinterpret_cast<T *>(gw_smem);  // [M][QM], zero beyond Q
    __shared__ T red[2][4][2 * QM];           // per-wave row sums, double buffered by row
    __shared__ T redf[4][QM + 1];             // per-wave dl and dsf2 sums
    __shared__ T sc4[QM], sil2[QM], sl[QM], sinvl[QM];  // 1/(4 l^2), 1/l^2, l, 1/l (zero
                                                        // beyond Q, except l = 1)
    __shared__ T srow[2][4][QM];              // staged row values (mu, w1, w2, S)
    __shared__ T sgl[4][QM];                  // per-wave dl sums over the chunk
    T *sgz = sz + M * QM;                     // [128][QM] the threads' dZ_m sums (dynamic LDS)
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, hh = lane >> 5;
    const int m = blockIdx.x * 128 + wv * 32 + (lane & 31);
    const bool valid = m < M;                 // the same on both lanes of a pair
    const int q0 = hh * QH;
    for (int i = tid; i < M * QM; i += 256) {
        const int mm = i / QM, q = i - mm * QM;
        sz[i] = q < Q ? Z[(int64_t)mm * Q + q] : T(0);
    }
    for (int q = tid; q < QM; q += 256) {
        sc4[q] = q < Q ? T(0.25) / h.l2[q] : T(0);
        sil2[q] = q < Q ? T(1) / h.l2[q] : T(0);
        sl[q] = q < Q ? h.l[q] : T(1);
        sinvl[q] = q < Q ? T(1) / h.l[q] : T(0);
    }
    __syncthreads();
    // the thread's dZ_m sums and each half-wave's dl sums live in LDS slots
    // that only they write (read-modify-write once per row and dimension)
    T z[QH];
    const int ml = m - blockIdx.x * 128;      // the thread's inducing input in the block
#pragma unroll
    for (int j = 0; j < QH; ++j) {
        z[j] = valid ? sz[m * QM + q0 + j] : T(0);
        sgz[ml * QM + q0 + j] = 0;
    }
    if ((lane & 31) == 0)
        for (int j = 0; j < QH; ++j) sgl[wv][q0 + j] = 0;
    T gsf = 0;
    // Each row's values (mu, w1, w2, S at every dimension, zero beyond Q) are
    // staged in LDS, double buffered by row parity: the next row's are written
    // before the barrier that ends the current row.
    auto stage_row = [&](int64_t n, int buf) {
        for (int i = tid; i < 4 * QM; i += 256) {
            const int k = i / QM, q = i - k * QM;
            const T *src = k == 0 ? mu : k == 1 ? w1t : k == 2 ? w2t : S;
            srow[buf][k][q] = (q < Q ? T(1) : T(0)) * src[n * Q + min(q, Q - 1)];
        }
    };
    // the two halves of a per-lane-pair sum, added in the same order on both lanes
    auto pair_sum = [&](T own) {
        const T other = __shfl_xor(own, 32);
        return hh == 0 ? own + other : other + own;
    };
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk, r1 = min(N, r0 + rows_per_chunk);
    if (r0 < r1) stage_row(r0, (int)(r0 & 1));
    __syncthreads();
    for (int64_t n = r0; n < r1; ++n) {
        const int b = (int)(n & 1);   // the row's buffer (its first row may be odd)
        const T *xs = srow[b][0] + q0, *a1s = srow[b][1] + q0, *a2s = srow[b][2] + q0,
                *svs = srow[b][3] + q0;
        T bq[QH], cq[QH], Vd[QH];
        T r = 0, e0 = 0;
        {
            T part = 0;
#pragma unroll
            for (int j = 0; j < QH; ++j) {
                const T a2 = a2s[j], d = xs[j] - z[j];
                bq[j] = a2 * d;
                cq[j] = sc4[q0 + j] + T(0.25) * a2;
                part -= bq[j] * d;
                Vd[j] = 0;
            }
            e0 = (G2s ? lp2[n] : T(0)) + pair_sum(part);
        }
        if (G2s && valid) {
            // G2s is symmetric: G2s[m'][m] is a coalesced row over the wave's m;
            // its entries are loaded kAhead partners ahead
            constexpr int kAhead = 2;
            const T *g2 = G2s + m;
            T gb[kAhead];
#pragma unroll
            for (int u = 0; u < kAhead; ++u) gb[u] = u < M ? g2[(int64_t)u * M] : T(0);
            for (int mp0 = 0; mp0 < M; mp0 += kAhead) {
#pragma unroll
                for (int u = 0; u < kAhead; ++u) {
                    const int mp = mp0 + u;
                    if (mp >= M) break;  // uniform
                    const T g = gb[u];
                    if (mp + kAhead < M) gb[u] = g2[(int64_t)(mp + kAhead) * M];
                    const T *zr = sz + mp * QM + q0;
                    T v[QH];
#pragma unroll
                    for (int j = 0; j < QH; ++j) v[j] = zr[j] - z[j];
                    T ep = 0;
#pragma unroll
                    for (int j = 0; j < QH; ++j) ep = fma(v[j], fma(-cq[j], v[j], bq[j]), ep);
                    const T W = g * dexp(e0 + pair_sum(ep));
                    r += W;
#pragma unroll
                    for (int j = 0; j < QH; ++j) Vd[j] = fma(W, v[j], Vd[j]);
                }
            }
        }
        T t = 0;
        if (G1 && valid) {
            T e1 = 0;
#pragma unroll
            for (int j = 0; j < QH; ++j) {
                const T d = xs[j] - z[j];
                e1 += d * d * a1s[j];
            }
            t = G1[n * M + m] * dexp(lp1[n] - T(0.5) * pair_sum(e1));
        }
        // per dimension: the dmu / dS terms summed over the block's m (butterflies
        // within each half-wave, whose lanes hold the same dimensions; then the
        // waves in order), the thread's dZ_m and dl terms.  The scheduling
        // barrier keeps each dimension's reads in its own step, so that the
        // epilogue does not hold every dimension's values at once.
        gsf += hh == 0 ? T(2) * r + t : T(0);  // dsf2 term, counted once per m
#pragma unroll
        for (int j = 0; j < QH; ++j) {
            const int q = q0 + j;
            const T x = xs[j], a1 = a1s[j], a2 = a2s[j], sv = svs[j];
            // with V = d r - Vd: d r + V = 2 d r - Vd, V - d r = -Vd,
            // d^2 r + d V = d (d r + V), d^2 r - d V = d Vd
            const T dq = x - z[j], d2 = dq * dq, dr = dq * r;
            const T s1 = T(2) * dr - Vd[j];
            const T il2 = sil2[q], l = sl[q], il = sinvl[q];
            T v0 = -T(2) * a2 * dr - t * dq * a1;
            T v1 = a2 * a2 * (dq * s1) - a2 * r + T(0.5) * t * (d2 * a1 * a1 - a1);
            sgz[ml * QM + q] += a2 * s1 + Vd[j] * il2 + t * dq * a1;
            T v2 = (T(2) * sv * a2 * il) * r + dq * Vd[j] * il2 * il + l * a2 * a2 * (dq * s1) +
                   t * (sv * a1 * il + l * d2 * a1 * a1);
#pragma unroll
            for (int off = 16; off >= 1; off >>= 1) {
                v0 += __shfl_xor(v0, off);
                v1 += __shfl_xor(v1, off);
                v2 += __shfl_xor(v2, off);
            }
            if ((lane & 31) == 0) {
                red[b][wv][q] = v0;
                red[b][wv][QM + q] = v1;
                sgl[wv][q] += v2;
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if (n + 1 < r1) stage_row(n + 1, b ^ 1);
        __syncthreads();
        if (tid < 2 * Q) {
            const int part = tid < Q ? 0 : 1, q = tid < Q ? tid : tid - Q;
            T v = 0;
            for (int w = 0; w < 4; ++w) v += red[b][w][part * QM + q];
            rowg[(((int64_t)blockIdx.x * 2 + part) * N + n) * Q + q] = v;
        }
    }
    if (valid) {
#pragma unroll
        for (int j = 0; j < QH; ++j)
            if (q0 + j < Q)
                colpart[((int64_t)blockIdx.y * M + m) * Q + q0 + j] = sgz[ml * QM + q0 + j];
    }
    // block sums of dl and dsf2 (fixed order) -> rowpart[block][Q + 1]
    if ((lane & 31) == 0)
        for (int j = 0; j < QH; ++j) redf[wv][q0 + j] = sgl[wv][q0 + j];
    {
        T v = gsf;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
        if (lane == 0) redf[wv][QM] = v;
    }
    __syncthreads();
    const int64_t blk = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
    if (tid <= Q) {
        const int k = tid < Q ? tid : QM;
        T v = 0;
        for (int w = 0; w < 4; ++w) v += redf[w][k];
        rowpart[blk * (Q + 1) + tid] = tid < Q ? v : v / h.sf2;
    }
}

template <typename T, int QM>
void launch_psi2_partial(const Shape &s, const Plan &p, const T *mu, const T *Z, const T *w2,
                         const T *lp2, const Hyp<T> &h, T *partial, const int *gate,
                         hipStream_t st) {
    dim3 grid((unsigned)p.pblocks, (unsigned)p.nc2);
    TimedScope ts(st, "generic_psi2_partial");
    if (fwd_ppt(s.Q, sizeof(T)) == 2)
        psi2_partial_kernel<T, QM, 2><<<grid, 256, 0, st>>>(gate, s.N, (int)s.M, (int)s.Q, s.P,
                                                            p.rows2, mu, Z, w2, lp2, h, partial);
    else
        psi2_partial_kernel<T, QM, 1><<<grid, 256, 0, st>>>(gate, s.N, (int)s.M, (int)s.Q, s.P,
                                                            p.rows2, mu, Z, w2, lp2, h, partial);
}

template <typename T, int QM>
void launch_grads(const Shape &s, const Plan &p, const T *mu, const T *S, const T *Z,
                  const T *w1, const T *w2, const T *lp1, const T *lp2, const Hyp<T> &h,
                  const T *G1, const T *G2s, T *rowg, T *colpart, T *rowpart, const int *gate,
                  hipStream_t st) {
    {
        TimedScope ts(st, "generic_grad_rows");
        grad_rows_kernel<T, QM><<<dim3((unsigned)p.row_blocks, (unsigned)p.rr), kRowBlock, 0, st>>>(gate, 
            s.N, (int)s.M, (int)s.Q, (int)p.rr, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s, rowg,
            rowpart);
    }
    dim3 grid((unsigned)p.col_blocks, (unsigned)p.ncc, (unsigned)p.cr);
    TimedScope ts(st, "generic_grad_cols");
    grad_cols_kernel<T, QM><<<grid, kColBlock, 0, st>>>(gate, s.N, (int)s.M, (int)s.Q, (int)p.cr,
                                                         p.rowsc, mu, Z, w1, w2, lp1, lp2, h, G1,
                                                         G2s, colpart);
}

template <typename T>
void rows_pre(const Shape &s, const Plan &p, const T *S, const Hyp<T> &h, void *ws,
              const int *gate, hipStream_t st) {
    TimedScope ts(st, "generic_rows_pre");
    rows_pre_kernel<T><<<(unsigned)cdiv(s.N, 256), 256, 0, st>>>(gate, 
        s.N, (int)s.Q, S, h, at<T>(ws, p.off_w1), at<T>(ws, p.off_w2), at<T>(ws, p.off_lp1),
        at<T>(ws, p.off_lp2));
}

}  // namespace

size_t generic_workspace_bytes(const Shape &s, size_t elem) { return make_plan(s, elem).total; }

template <typename T>
hipError_t generic_psi_stats(const Shape &s, const T *mu, const T *S, const T *Z,
                             const Hyp<T> &h, T *psi0, T *Psi1, T *Psi2, int accumulate,
                             void *ws, const int *gate, hipStream_t st) {
    const Plan p = make_plan(s, sizeof(T));
    rows_pre<T>(s, p, S, h, ws, gate, st);
    const T *w1 = at<T>(ws, p.off_w1), *w2 = at<T>(ws, p.off_w2);
    const T *lp1 = at<T>(ws, p.off_lp1), *lp2 = at<T>(ws, p.off_lp2);
    if (Psi1) {
        TimedScope ts(st, "generic_psi1");
        psi1_kernel<T><<<(unsigned)std::min<int64_t>(cdiv(s.N * s.M, 256), kGridCap), 256, 0, st>>>(gate, s.N, (int)s.M, (int)s.Q,
                                                                       mu, Z, w1, lp1, Psi1);
    }
    T *partial = at<T>(ws, p.off_p2);
    switch (fwd_qm(s.Q)) {
#define GPPS_FWD(QMV) \
    case QMV: launch_psi2_partial<T, QMV>(s, p, mu, Z, w2, lp2, h, partial, gate, st); break
        GPPS_FWD(1); GPPS_FWD(2); GPPS_FWD(4); GPPS_FWD(8); GPPS_FWD(12); GPPS_FWD(16);
        GPPS_FWD(20); GPPS_FWD(24); GPPS_FWD(32); GPPS_FWD(48);
        default: launch_psi2_partial<T, 64>(s, p, mu, Z, w2, lp2, h, partial, gate, st); break;
#undef GPPS_FWD
    }
    dim3 g((unsigned)p.tiles_edge, (unsigned)p.tiles_edge);
    TimedScope ts(st, "generic_psi2_reduce");
    psi2_reduce_kernel<T><<<g, kPairTile * kPairTile, 0, st>>>(gate, s.N, (int)s.M, s.P, p.nc2,
                                                               partial, h, psi0, Psi2,
                                                               accumulate);
    return hipGetLastError();
}

template <typename T>
hipError_t generic_psi_grads(const Shape &s, const T *mu, const T *S, const T *Z,
                             const Hyp<T> &h, T dL_dpsi0, const T *G1, const T *G2, T *dmu,
                             T *dS, T *dZ, T *dsf2, T *dl, int accumulate, void *ws,
                             const int *gate, hipStream_t st) {
    const Plan p = make_plan(s, sizeof(T));
    rows_pre<T>(s, p, S, h, ws, gate, st);
    const T *w1 = at<T>(ws, p.off_w1), *w2 = at<T>(ws, p.off_w2);
    const T *lp1 = at<T>(ws, p.off_lp1), *lp2 = at<T>(ws, p.off_lp2);
    T *G2s = nullptr;
    if (G2) {
        G2s = at<T>(ws, p.off_g2s);
        TimedScope ts(st, "generic_sym");
        sym_kernel<T><<<(unsigned)cdiv(s.M * s.M, 256), 256, 0, st>>>(gate, (int)s.M, G2, G2s);
    }
    T *colpart = at<T>(ws, p.off_colp), *rowpart = at<T>(ws, p.off_rowp);
    T *rowg = at<T>(ws, p.off_rowg);
    if (p.pairs) {
        const bool sym = p.psym && G2s;
        T *Gc = at<T>(ws, p.off_gc);
        if (sym) {
            TimedScope ts(st, "generic_circ");
            circ_kernel<T><<<(unsigned)cdiv((s.M / 2 + 1) * s.M, 256), 256, 0, st>>>(gate, (int)s.M, G2s, Gc);
        }
        const size_t lds = sizeof(T) * s.M * (pairs_qm(s.Q) + (sym ? 2 * kBand : 0));
        const size_t lds_slots =
            sizeof(T) * s.M * (pairs_qm(s.Q) + p.prs * 2 * kSlotBand + p.prs * 2 * pairs_qm(s.Q));
        dim3 grid((unsigned)p.pmb, (unsigned)p.pchunks);
        {
            TimedScope ts(st, "generic_grad_pairs");
#define GPPS_PAIRS(QMV)                                                                            \
    do {                                                                                           \
        if (sym && p.pslots)                                                                       \
            grad_pairs_slots_kernel<T, QMV><<<grid, p.psthreads, lds_slots, st>>>(gate,                  \
                s.N, (int)s.M, (int)s.Q, p.prs, p.prows, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s,   \
                Gc, rowg, colpart, rowpart);                                                       \
        else if (sym)                                                                              \
            grad_pairs_kernel<T, QMV, true><<<grid, p.pthreads, lds, st>>>(gate,                         \
                s.N, (int)s.M, (int)s.Q, p.prows, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s, Gc,      \
                rowg, colpart, rowpart);                                                           \
        else                                                                                       \
            grad_pairs_kernel<T, QMV, false><<<grid, p.pthreads, lds, st>>>(gate,                        \
                s.N, (int)s.M, (int)s.Q, p.prows, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s, Gc,      \
                rowg, colpart, rowpart);                                                           \
    } while (0)
            switch (pairs_qm(s.Q)) {
                case 1: GPPS_PAIRS(1); break;
                case 2: GPPS_PAIRS(2); break;
                case 4: GPPS_PAIRS(4); break;
                default:
                    if (sizeof(T) == 4) GPPS_PAIRS(8);
                    break;
            }
#undef GPPS_PAIRS
        }
        const int64_t total = s.M * s.Q + s.Q + 1;
        TimedScope ts(st, "generic_grad_reduce");
        grad_rows_reduce_kernel<T><<<(unsigned)std::min<int64_t>(cdiv(s.N * s.Q, 256), kGridCap), 256, 0, st>>>(gate, 
            s.N * s.Q, (int)p.pmb, rowg, dmu, dS);
        grad_reduce_kernel<T><<<(unsigned)std::min<int64_t>(total, kGridCap), 256, 0, st>>>(gate, 
            s.N, (int)s.M, (int)s.Q, p.pchunks, p.pmb * p.pchunks, colpart, rowpart, dL_dpsi0, dZ,
            dsf2, dl, accumulate);
        return hipGetLastError();
    }
    if (p.wide) {
        const size_t lds = sizeof(T) * (s.M + 128) * 2 * p.wqh;
        dim3 grid((unsigned)p.wmb, (unsigned)p.wchunks);
        {
            TimedScope ts(st, "generic_grad_wide");
#define GPPS_WIDE(QHV)                                                                             \
    case QHV:                                                                                      \
        grad_wide_kernel<T, QHV><<<grid, 256, lds, st>>>(gate, s.N, (int)s.M, (int)s.Q, p.wrows,  \
                                                          mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s,  \
                                                          rowg, colpart, rowpart);                 \
        break
            switch (p.wqh) {
                GPPS_WIDE(4);
                GPPS_WIDE(6);
                GPPS_WIDE(8);
                GPPS_WIDE(10);
                GPPS_WIDE(12);
                GPPS_WIDE(16);
                default:
                    if constexpr (sizeof(T) == 4) {
                        switch (p.wqh) {
                            GPPS_WIDE(24);
                            GPPS_WIDE(32);
                            default: break;
                        }
                    }
                    break;
            }
#undef GPPS_WIDE
        }
        const int64_t total = s.M * s.Q + s.Q + 1;
        TimedScope ts(st, "generic_grad_reduce");
        grad_rows_reduce_kernel<T><<<(unsigned)std::min<int64_t>(cdiv(s.N * s.Q, 256), kGridCap), 256, 0, st>>>(gate,
            s.N * s.Q, (int)p.wmb, rowg, dmu, dS);
        grad_reduce_kernel<T><<<(unsigned)std::min<int64_t>(total, kGridCap), 256, 0, st>>>(gate,
            s.N, (int)s.M, (int)s.Q, p.wchunks, p.wmb * p.wchunks, colpart, rowpart, dL_dpsi0, dZ,
            dsf2, dl, accumulate);
        return hipGetLastError();
    }
    if (s.Q <= 4)
        launch_grads<T, 4>(s, p, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s, rowg, colpart, rowpart, gate, st);
    else if (s.Q <= 8)
        launch_grads<T, 8>(s, p, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s, rowg, colpart, rowpart, gate, st);
    else if (s.Q <= 16)
        launch_grads<T, 16>(s, p, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s, rowg, colpart, rowpart, gate, st);
    else if (s.Q <= 32)
        launch_grads<T, 32>(s, p, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s, rowg, colpart, rowpart, gate, st);
    else
        launch_grads<T, 64>(s, p, mu, S, Z, w1, w2, lp1, lp2, h, G1, G2s, rowg, colpart, rowpart, gate, st);
    const int64_t total = s.M * s.Q + s.Q + 1;
    TimedScope ts(st, "generic_grad_reduce");
    grad_rows_reduce_kernel<T><<<(unsigned)std::min<int64_t>(cdiv(s.N * s.Q, 256), kGridCap), 256, 0, st>>>(gate, s.N * s.Q, (int)p.rr,
                                                                              rowg, dmu, dS);
    grad_reduce_kernel<T><<<(unsigned)std::min<int64_t>(total, kGridCap), 256, 0, st>>>(gate, 
        s.N, (int)s.M, (int)s.Q, p.ncc * p.cr, p.rr * p.row_blocks, colpart, rowpart, dL_dpsi0,
        dZ, dsf2, dl, accumulate);
    return hipGetLastError();
}

template hipError_t generic_psi_stats<float>(const Shape &, const float *, const float *,
                                             const float *, const Hyp<float> &, float *,
                                             float *, float *, int, void *, const int *,
                                             hipStream_t);
template hipError_t generic_psi_stats<double>(const Shape &, const double *, const double *,
                                              const double *, const Hyp<double> &, double *,
                                              double *, double *, int, void *, const int *,
                                              hipStream_t);
template hipError_t generic_psi_grads<float>(const Shape &, const float *, const float *,
                                             const float *, const Hyp<float> &, float,
                                             const float *, const float *, float *, float *,
                                             float *, float *, float *, int, void *,
                                             const int *, hipStream_t);
template hipError_t generic_psi_grads<double>(const Shape &, const double *, const double *,
                                              const double *, const Hyp<double> &, double,
                                              const double *, const double *, double *,
                                              double *, double *, double *, double *, int,
                                              void *, const int *, hipStream_t);

}  // namespace gpps
