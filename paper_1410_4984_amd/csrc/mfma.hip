// Matrix-core path (F32, gfx950): the O(N M^2 Q) Psi2 statistic and its
// gradient on v_mfma_f32_32x32x2_f32, with exp2 and the dL/dPsi2 weighting on
// the vector ALU.
//
// Per datapoint n the Psi2 summand is a Gram matrix pushed through exp
// (section 2, eq. (4): Phi turned into an expectation under q(x_n); Alg. 1
// computes it per pair of inducing inputs and sums over datapoints).  With
// d_m = mu_n - z_m (per dimension q), w2 = 1/(l^2 + 2 S_nq) and
// kappa = S_nq / (l^2 (l^2 + 2 S_nq)) >= 0, the exponent of
//   Psi2_n[m, m'] = sf2^2 prod_q (1 + 2S/l^2)^(-1/2)
//                   exp(-sum_q [(z_m - z_m')^2/(4 l^2) + (mu - (z_m + z_m')/2)^2 w2])
// splits exactly into a row term, a column term and a Gram term:
//   log2 Psi2_n[m, m'] = b_m + b_m' + sum_q a_mq a_m'q,
//   a_mq = d_mq sqrt(log2(e) kappa_q),
//   b_m  = log2(e) (log sf2 - 1/4 sum_q log(1 + 2S/l^2) - 1/4 sum_q (1/l^2 + w2) d_mq^2).
// The Gram term is a K = Q contraction per 32 x 32 tile of pairs (MFMA); the
// row and column terms enter through the MFMA's C input; exp2 is one
// v_exp_f32.  Inputs are centred (Z and mu shifted by the mean inducing
// input), which changes no result (every quantity depends on mu - z only).
//
// Gradient (Alg. 2): with W_n = G2s o Psi2_n (G2s the symmetric part of
// dL/dPsi2), r_n = W_n 1 and V_n = W_n D_n (D_n[m, q] = d_mq), every derivative
// is linear in r_n and V_n:
//   dmu_nq   = -2 w2 sum_m d r
//   dS_nq    = w2^2 (X + Y) - w2 R,        X = sum_m d^2 r, Y = sum_m d V, R = sum_m r
//   dZ_mq   += V (w2 - 1/l^2) + d r (w2 + 1/l^2)
//   dl_q    += (2 S w2 / l) R + l w2^2 (X + Y) + (X - Y) / l^3
//   dsf2    += 2 R / sf2
// Since D_n = 1 mu_n^T - Z, V_n = r_n mu_n^T - W_n Z: the second MFMA product
// is W_n [Z | 1], whose B operand is the constant Z table and whose ones
// column yields r_n.  Its A operand is the W tile exactly as the first MFMA
// left it in registers.
//
// Work split.  Z (centred, plus the ones column) is staged in LDS once per
// workgroup.  Rows are processed in batches: the batch's per-row values and
// its row terms b (exact d-form, one thread per inducing input) are staged in
// LDS, then every wave runs its rows with no further barrier.  Forward: a
// workgroup owns a group of upper-triangular 32 x 32 pair tiles and a chunk of
// rows; each wave keeps its tiles' running sums in registers; partial tiles
// are reduced over chunks in a fixed order.  Gradient: every term above is
// linear in (r_n, V_n), so the full M x M tile grid is split into wave tasks
// (one row block of W, up to four column blocks) whose dL/dPsi2 tiles stay in
// registers; each task adds its share of dZ (registers) and of the per-row
// sums X, Y, P, R (LDS, then global), which a finalize kernel combines.  No
// atomics; every cross-wave or cross-workgroup sum runs in a fixed order, so
// results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace gpps {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kTile = 32;
constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kRowStride = 64;         // stride of per-row tables padded to 64 dimensions
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kPadBias = -1.0e30f;   // row term of a padded inducing input: exp2 -> 0
constexpr int kMaxTilesPerWave = 4;    // forward
constexpr int kRBF = 16;               // forward rows per batch
constexpr int kRBG = 8;                // gradient rows per batch
constexpr int64_t kFwdTargetWGs = 1024;
constexpr int64_t kGradTargetWGs = 512;
constexpr int kFinRows = 64;           // rows per block of the gradient finalize kernel

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Row of the 32x32 C/D register layout: lane l holds column l % 32 and, in
// register t, row 8 (t / 4) + 4 (l / 32) + t % 4.
__device__ __forceinline__ int crow(int t, int g) { return 8 * (t >> 2) + 4 * g + (t & 3); }

struct MPlan {
    int64_t Mp;            // M rounded up to the tile edge
    int nb;                // tiles per edge
    int nqb;               // 32-column blocks of [Z | 1] (Q + 1 columns)
    int DS;                // LDS row stride of the Z table (odd: conflict-free column reads)
    int ks;                // MFMA k-steps (2 latent dimensions each), instantiated value
    int jpw, njr, ntasks;  // gradient: column blocks per wave task, ranges, tasks (nb * njr)
    int64_t ggroups;       // gradient: workgroups (4 tasks each) per row chunk
    int64_t T;             // upper-triangular tiles
    int64_t tpg, groups;   // forward: tiles per group, groups
    int64_t frows, fchunks;
    int64_t grows, gchunks;
    size_t lds_fwd, lds_grad;
    int64_t fin_blocks;    // finalize: blocks of kFinRows rows
    size_t off_sq, off_hq, off_w2, off_hl, off_zc, off_g2, off_fp, off_rs, off_dz, off_dl, total;
};

int round_ks(int ks, int nqb) {
    static const int one[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 15, 16};
    static const int two[] = {16, 24, 32};
    if (nqb == 1) {
        for (int v : one)
            if (ks <= v) return v;
    } else {
        for (int v : two)
            if (ks <= v) return v;
    }
    return -1;
}

// LDS layout (floats), shared by both kernels:
//   Zx  [Mp][DS]        centred z, column Q = 1 for real rows, zero padding
//   bb  [RB][Mp]        row terms of the batch
//   mub [RB][64]        centred mu of the batch (zero beyond Q)
//   sqb [RB][64]        sqrt(log2e kappa) of the batch (zero beyond Q)
//   hqb [RB][Q]         -log2e/4 (1/l^2 + w2)
//   hlb [RB]            log-prefactor
// gradient only:
//   w2b [RB][Q], red [RB][kWaves][3Q + 1]
struct Lds {
    int zx, bb, mub, sqb, hqb, hlb, w2b, red, total;
};

__host__ __device__ inline Lds lds_layout(int Mp, int DS, int Q, int RB, bool grad) {
    Lds L{};
    int o = 0;
    L.zx = o; o += Mp * DS;
    L.bb = o; o += RB * Mp;
    L.mub = o; o += RB * kRowStride;
    L.sqb = o; o += RB * kRowStride;
    L.hqb = o; o += RB * Q;
    L.hlb = o; o += (RB + 3) / 4 * 4;
    L.w2b = L.red = o;
    if (grad) {
        L.w2b = o; o += RB * Q;
        L.red = o; o += RB * kWaves * (3 * Q + 1);
    }
    L.total = o;
    return L;
}

MPlan make_mplan(const Shape &s) {
    MPlan p{};
    p.Mp = cdiv(s.M, kTile) * kTile;
    p.nb = (int)(p.Mp / kTile);
    p.nqb = s.Q + 1 <= 32 ? 1 : 2;
    p.DS = 32 * p.nqb + 1;
    p.ks = round_ks((int)cdiv(s.Q, 2), p.nqb);
    p.jpw = p.nb >= 2 ? 2 : 1;   // 2: the task fits 2 waves per SIMD
    p.njr = (int)cdiv(p.nb, p.jpw);
    p.ntasks = p.nb * p.njr;
    p.ggroups = cdiv(p.ntasks, kWaves);
    p.T = (int64_t)p.nb * (p.nb + 1) / 2;
    p.groups = cdiv(p.T, kWaves * kMaxTilesPerWave);
    p.tpg = cdiv(p.T, p.groups);
    p.fchunks = std::max<int64_t>(1, std::min(cdiv(kFwdTargetWGs, p.groups), cdiv(s.N, 32)));
    p.frows = cdiv(s.N, p.fchunks);
    p.fchunks = cdiv(s.N, p.frows);
    p.gchunks = std::max<int64_t>(1, std::min(cdiv(kGradTargetWGs, p.ggroups), cdiv(s.N, 16)));
    p.grows = cdiv(s.N, p.gchunks);
    p.gchunks = cdiv(s.N, p.grows);
    p.lds_fwd = sizeof(float) * lds_layout((int)p.Mp, p.DS, (int)s.Q, kRBF, false).total;
    p.lds_grad = sizeof(float) * lds_layout((int)p.Mp, p.DS, (int)s.Q, kRBG, true).total;
    size_t o = generic_workspace_bytes(s, sizeof(float));   // Psi1 pieces live first
    auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
    p.off_sq = take(sizeof(float) * s.N * kRowStride);
    p.off_hq = take(sizeof(float) * s.N * s.Q);
    p.off_w2 = take(sizeof(float) * s.N * s.Q);
    p.off_hl = take(sizeof(float) * s.N);
    p.off_zc = take(sizeof(float) * s.Q);
    p.off_g2 = take(sizeof(float) * p.Mp * p.Mp);
    p.off_fp = take(sizeof(float) * p.fchunks * p.T * kTile * kTile);
    p.fin_blocks = cdiv(s.N, kFinRows);
    p.off_rs = take(sizeof(float) * p.ggroups * s.N * (3 * s.Q + 1));
    p.off_dz = take(sizeof(float) * p.gchunks * p.njr * s.M * s.Q);
    p.off_dl = take(sizeof(float) * p.fin_blocks * (s.Q + 1));
    p.total = o;
    return p;
}

float *fat(void *ws, size_t off) { return reinterpret_cast<float *>(static_cast<char *>(ws) + off); }

// ---------------------------------------------------------------- small kernels
// sq[n][q] = sqrt(log2e * kappa_nq) (zero for q >= Q up to the stride),
// hq[n][q] = -log2e/4 (1/l^2 + w2), w2[n][q], hl[n] = log2e (log sf2 - 1/4 sum_q log(1 + 2S/l^2)).
__global__ void mfma_rows_kernel(int64_t N, int Q, const float *__restrict__ S, Hyp<float> h,
                                 float *__restrict__ sq, float *__restrict__ hq,
                                 float *__restrict__ w2t, float *__restrict__ hl) {
    const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= N) return;
    float lsum = 0.f;
    for (int q = 0; q < kRowStride; ++q) {
        if (q < Q) {
            const float s = S[n * Q + q];
            const float l2 = h.l2[q];
            const float w2 = 1.f / (l2 + 2.f * s);
            const float kap = s * w2 / l2;
            sq[n * kRowStride + q] = sqrtf(kLog2e * kap);
            hq[n * Q + q] = -0.25f * kLog2e * (1.f / l2 + w2);
            w2t[n * Q + q] = w2;
            lsum += log1pf(2.f * s / l2);
        } else {
            sq[n * kRowStride + q] = 0.f;
        }
    }
    hl[n] = kLog2e * (h.log_sf2 - 0.25f * lsum);
}

// Mean inducing input per dimension (fixed-order sum): the centring shift.
__global__ void mfma_centre_kernel(int M, int Q, const float *__restrict__ Z,
                                   float *__restrict__ zc) {
    const int q = threadIdx.x;
    if (q >= Q) return;
    float s = 0.f;
    for (int m = 0; m < M; ++m) s += Z[(int64_t)m * Q + q];
    zc[q] = s / (float)M;
}

// Symmetric part of dL/dPsi2, zero-padded to Mp x Mp.
__global__ void mfma_sym_kernel(int M, int Mp, const float *__restrict__ G2,
                                float *__restrict__ G2p) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)Mp * Mp) return;
    const int m = (int)(i / Mp), mp = (int)(i - (int64_t)m * Mp);
    G2p[i] = (m < M && mp < M) ? 0.5f * (G2[(int64_t)m * M + mp] + G2[(int64_t)mp * M + m]) : 0.f;
}

// ---------------------------------------------------------------- LDS staging
__device__ void stage_z(float *lds, const Lds &L, int M, int Mp, int Q, int DS,
                        const float *__restrict__ Z, const float *__restrict__ zc) {
    for (int i = threadIdx.x; i < Mp * DS; i += kThreads) {
        const int m = i / DS, q = i - m * DS;
        float v = 0.f;
        if (m < M) {
            if (q < Q) v = Z[(int64_t)m * Q + q] - zc[q];
            else if (q == Q) v = 1.f;
        }
        lds[L.zx + i] = v;
    }
}

// Per-row values of rows [n0, n0 + cb) into the batch arrays, then (after a
// barrier) the row terms b of every inducing input.  Rows >= cb are zero.
template <int RB, bool GRAD>
__device__ void stage_batch(float *lds, const Lds &L, int64_t n0, int cb, int M, int Mp, int Q,
                            int DS, const float *__restrict__ mu, const float *__restrict__ zc,
                            const float *__restrict__ sq, const float *__restrict__ hq,
                            const float *__restrict__ hl, const float *__restrict__ w2t) {
    for (int i = threadIdx.x; i < RB * kRowStride; i += kThreads) {
        const int r = i / kRowStride, q = i - r * kRowStride;
        const bool ok = r < cb && q < Q;
        const int64_t n = n0 + r;
        lds[L.mub + i] = ok ? mu[n * Q + q] - zc[q] : 0.f;
        lds[L.sqb + i] = ok ? sq[n * kRowStride + q] : 0.f;
    }
    for (int i = threadIdx.x; i < RB * Q; i += kThreads) {
        const int r = i / Q;
        const bool ok = r < cb;
        lds[L.hqb + i] = ok ? hq[n0 * Q + i] : 0.f;
        if (GRAD) lds[L.w2b + i] = ok ? w2t[n0 * Q + i] : 0.f;
    }
    for (int r = threadIdx.x; r < RB; r += kThreads) lds[L.hlb + r] = r < cb ? hl[n0 + r] : 0.f;
    __syncthreads();
    for (int m = threadIdx.x; m < Mp; m += kThreads) {
        float acc[RB];
#pragma unroll
        for (int r = 0; r < RB; ++r) acc[r] = lds[L.hlb + r];
        if (m < M) {
            for (int q = 0; q < Q; ++q) {
                const float z = lds[L.zx + m * DS + q];
#pragma unroll
                for (int r = 0; r < RB; ++r) {
                    const float d = lds[L.mub + r * kRowStride + q] - z;
                    acc[r] = fmaf(lds[L.hqb + r * Q + q] * d, d, acc[r]);
                }
            }
        }
#pragma unroll
        for (int r = 0; r < RB; ++r) lds[L.bb + r * Mp + m] = (m < M && r < cb) ? acc[r] : kPadBias;
    }
}

// MFMA operand values a_{m, 2s+g} for the 32 rows of block `blk` (lane supplies row c).
template <int KS>
__device__ __forceinline__ void operands(const float *zx, int DS, int blk, int c, int g,
                                         const float (&muk)[KS], const float (&sk)[KS],
                                         float (&out)[KS]) {
    const float *zr = zx + (blk * kTile + c) * DS + g;
#pragma unroll
    for (int s = 0; s < KS; ++s) out[s] = (muk[s] - zr[2 * s]) * sk[s];
}

// ---------------------------------------------------------------- Psi2 forward
template <int KS>
__global__ __launch_bounds__(kThreads) void psi2_fwd_kernel(
    int64_t N, int M, int Q, int Mp, int nb, int DS, int64_t T, int64_t tpg,
    int64_t rows_per_chunk, const float *__restrict__ mu, const float *__restrict__ Z,
    const float *__restrict__ zc, const float *__restrict__ sq, const float *__restrict__ hq,
    const float *__restrict__ hl, float *__restrict__ partial) {
    extern __shared__ float lds[];
    const Lds L = lds_layout(Mp, DS, Q, kRBF, false);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c = lane & 31, g = lane >> 5;

    // this wave's tiles: a contiguous run of the group, so neighbours share their row block
    const int64_t t0 = (int64_t)blockIdx.x * tpg, t1 = min(T, t0 + tpg);
    const int64_t tpw = (tpg + kWaves - 1) / kWaves;
    int ti[kMaxTilesPerWave], tj[kMaxTilesPerWave];
    bool tv[kMaxTilesPerWave];
#pragma unroll
    for (int k = 0; k < kMaxTilesPerWave; ++k) {
        const int64_t t = t0 + wave * tpw + k;
        tv[k] = k < tpw && t < t1;
        int64_t r = 0, u = tv[k] ? t : 0;
        while (u >= nb - r) { u -= nb - r; ++r; }
        ti[k] = (int)r;
        tj[k] = (int)(r + u);
    }
    v16f acc[kMaxTilesPerWave];
#pragma unroll
    for (int k = 0; k < kMaxTilesPerWave; ++k)
#pragma unroll
        for (int t = 0; t < 16; ++t) acc[k][t] = 0.f;

    stage_z(lds, L, M, Mp, Q, DS, Z, zc);
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    for (int64_t n0 = r0; n0 < r1; n0 += kRBF) {
        const int cb = (int)min<int64_t>(kRBF, r1 - n0);
        __syncthreads();
        stage_batch<kRBF, false>(lds, L, n0, cb, M, Mp, Q, DS, mu, zc, sq, hq, hl, nullptr);
        __syncthreads();
        for (int r = 0; r < cb; ++r) {
            float muk[KS], sk[KS];
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                muk[s] = lds[L.mub + r * kRowStride + 2 * s + g];
                sk[s] = lds[L.sqb + r * kRowStride + 2 * s + g];
            }
            const float *bb = lds + L.bb + r * Mp;
            float aop[KS];
            int cur = -1;
#pragma unroll
            for (int k = 0; k < kMaxTilesPerWave; ++k) {
                if (!tv[k]) continue;
                if (ti[k] != cur) {
                    operands<KS>(lds + L.zx, DS, ti[k], c, g, muk, sk, aop);
                    cur = ti[k];
                }
                float bop[KS];
                operands<KS>(lds + L.zx, DS, tj[k], c, g, muk, sk, bop);
                const float bcol = bb[tj[k] * kTile + c];
                v16f e;
#pragma unroll
                for (int t = 0; t < 16; ++t) e[t] = bb[ti[k] * kTile + crow(t, g)] + bcol;
#pragma unroll
                for (int s = 0; s < KS; ++s)
                    e = __builtin_amdgcn_mfma_f32_32x32x2f32(aop[s], bop[s], e, 0, 0, 0);
#pragma unroll
                for (int t = 0; t < 16; ++t) acc[k][t] += __builtin_amdgcn_exp2f(e[t]);
            }
        }
    }
    // partial tiles, row-major inside the tile
#pragma unroll
    for (int k = 0; k < kMaxTilesPerWave; ++k) {
        if (!tv[k]) continue;
        const int64_t t = t0 + wave * tpw + k;
        float *dst = partial + ((int64_t)blockIdx.y * T + t) * (kTile * kTile);
#pragma unroll
        for (int r = 0; r < 16; ++r) dst[crow(r, g) * kTile + c] = acc[k][r];
    }
}

// Fixed-order sum over chunks; both triangles written from the same value.
__global__ void psi2_reduce_kernel(int64_t N, int M, int nb, int64_t T, int64_t chunks,
                                   const float *__restrict__ partial, float sf2,
                                   float *__restrict__ psi0, float *__restrict__ Psi2,
                                   int accumulate) {
    const int mp = blockIdx.x * 16 + (threadIdx.x & 15);
    const int m = blockIdx.y * 16 + (threadIdx.x >> 4);
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
        psi0[0] = (accumulate ? psi0[0] : 0.f) + (float)N * sf2;
    if (m >= M || mp >= M || m > mp) return;
    const int ti = m / kTile, tj = mp / kTile;
    const int64_t t = (int64_t)ti * nb - (int64_t)ti * (ti - 1) / 2 + (tj - ti);
    const int64_t off = t * (kTile * kTile) + (m % kTile) * kTile + (mp % kTile);
    float s = 0.f;
    for (int64_t ch = 0; ch < chunks; ++ch) s += partial[ch * T * (kTile * kTile) + off];
    const float v = (accumulate ? Psi2[(int64_t)m * M + mp] : 0.f) + s;
    Psi2[(int64_t)m * M + mp] = v;
    Psi2[(int64_t)mp * M + m] = v;
}

// ---------------------------------------------------------------- Psi2 gradient
// Every gradient term is linear in (r_n, V_n), so the M x M tile grid may be
// split freely: a wave task is one row block i (the m index of W) and up to
// JPW column blocks j (the m' index).  The task's dL/dPsi2 tiles stay in
// registers for the whole kernel; V' = W [Z | 1] accumulates over the task's
// tiles; the epilogue turns it into the task's share of dZ (registers) and of
// the per-row sums X, Y, P, R, which the workgroup combines in LDS and writes
// per (group, row) for psi2_finalize_kernel.
template <int KS, int JPW, int NQB>
__global__ __launch_bounds__(kThreads) void psi2_grad_kernel(
    int64_t N, int M, int Q, int Mp, int nb, int DS, int njr, int ntasks,
    int64_t rows_per_chunk, const float *__restrict__ mu, const float *__restrict__ Z,
    const float *__restrict__ zc, const float *__restrict__ sq, const float *__restrict__ hq,
    const float *__restrict__ hl, const float *__restrict__ w2t, const float *__restrict__ G2p,
    Hyp<float> h, float *__restrict__ rowsum, float *__restrict__ part_dz) {
    extern __shared__ float lds[];
    const Lds L = lds_layout(Mp, DS, Q, kRBG, true);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c = lane & 31, g = lane >> 5;
    const int ones_src = 32 * g + (Q & 31);    // lane holding column Q (the row sums r)
    const int ones_qb = Q >> 5;
    const int RED = 3 * Q + 1;
    const int group = blockIdx.x;
    const int task = group * kWaves + wave;
    const bool active = task < ntasks;         // wave-uniform
    const int i = active ? task / njr : 0;     // row block of W (m)
    const int jr = active ? task % njr : 0;    // range of column blocks of W (m')

    float g2r[JPW][16];
    bool jv[JPW];
#pragma unroll
    for (int k = 0; k < JPW; ++k) {
        const int j = jr * JPW + k;
        jv[k] = active && j < nb;
        const float *g2 = G2p + (int64_t)(jv[k] ? j : 0) * kTile * Mp + i * kTile + c;
#pragma unroll
        for (int t = 0; t < 16; ++t) g2r[k][t] = jv[k] ? g2[(int64_t)crow(t, g) * Mp] : 0.f;
    }
    v16f dz[NQB];
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
        for (int t = 0; t < 16; ++t) dz[qb][t] = 0.f;
    float il2[NQB];
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
        const int q = qb * 32 + c;
        il2[qb] = q < Q ? 1.f / h.l2[q] : 0.f;
    }

    stage_z(lds, L, M, Mp, Q, DS, Z, zc);
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    for (int64_t n0 = r0; n0 < r1; n0 += kRBG) {
        const int cb = (int)min<int64_t>(kRBG, r1 - n0);
        __syncthreads();
        stage_batch<kRBG, true>(lds, L, n0, cb, M, Mp, Q, DS, mu, zc, sq, hq, hl, w2t);
        __syncthreads();
        for (int r = 0; r < cb; ++r) {
            float *rs = lds + L.red + (r * kWaves + wave) * RED;
            if (!active) {
                for (int k = lane; k < RED; k += 64) rs[k] = 0.f;
                continue;
            }
            float muk[KS], sk[KS];
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                muk[s] = lds[L.mub + r * kRowStride + 2 * s + g];
                sk[s] = lds[L.sqb + r * kRowStride + 2 * s + g];
            }
            const float *bb = lds + L.bb + r * Mp;
            // Gram B operand: column block i (the m index of W)
            float bop[KS];
            operands<KS>(lds + L.zx, DS, i, c, g, muk, sk, bop);
            const float bcol = bb[i * kTile + c];
            v16f V[NQB];
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
                for (int t = 0; t < 16; ++t) V[qb][t] = 0.f;
#pragma unroll
            for (int k = 0; k < JPW; ++k) {
                if (!jv[k]) continue;
                const int j = jr * JPW + k;
                // rows m' in block j (A operand), columns m in block i (B operand)
                float aop[KS];
                operands<KS>(lds + L.zx, DS, j, c, g, muk, sk, aop);
                v16f e;
#pragma unroll
                for (int t = 0; t < 16; ++t) e[t] = bb[j * kTile + crow(t, g)] + bcol;
#pragma unroll
                for (int s = 0; s < KS; ++s)
                    e = __builtin_amdgcn_mfma_f32_32x32x2f32(aop[s], bop[s], e, 0, 0, 0);
                const float *zrow = lds + L.zx + j * kTile * DS + c;
#pragma unroll
                for (int t = 0; t < 16; ++t) {
                    const float w = g2r[k][t] * __builtin_amdgcn_exp2f(e[t]);
#pragma unroll
                    for (int qb = 0; qb < NQB; ++qb)
                        V[qb] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            w, zrow[crow(t, g) * DS + qb * 32], V[qb], 0, 0, 0);
                }
            }
            // epilogue for rows m = i*32 + crow(t, g); V' = W [Z | 1] -> V = r mu^T - V'
            float muq[NQB], alpha[NQB], beta[NQB];
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) {
                const int q = qb * 32 + c;
                muq[qb] = lds[L.mub + r * kRowStride + q];
                const float w2 = q < Q ? lds[L.w2b + r * Q + q] : 0.f;
                alpha[qb] = w2 - il2[qb];
                beta[qb] = w2 + il2[qb];
            }
            float X[NQB], Y[NQB], P[NQB], R = 0.f;
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) X[qb] = Y[qb] = P[qb] = 0.f;
            const float *zblk = lds + L.zx + i * kTile * DS;
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int rr = crow(t, g);
                const float rt = __int_as_float(__builtin_amdgcn_ds_bpermute(
                    ones_src * 4, __float_as_int(ones_qb == 0 ? V[0][t] : V[NQB - 1][t])));
                R += rt;
#pragma unroll
                for (int qb = 0; qb < NQB; ++qb) {
                    const float d = muq[qb] - zblk[rr * DS + qb * 32 + c];
                    const float v = fmaf(rt, muq[qb], -V[qb][t]);
                    const float dr = d * rt;
                    dz[qb][t] = fmaf(alpha[qb], v, fmaf(beta[qb], dr, dz[qb][t]));
                    X[qb] = fmaf(dr, d, X[qb]);
                    P[qb] += dr;
                    Y[qb] = fmaf(d, v, Y[qb]);
                }
            }
            // combine the two lane halves, publish this wave's sums for row r
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) {
                const float x2 = __shfl_xor(X[qb], 32), y2 = __shfl_xor(Y[qb], 32),
                            p2 = __shfl_xor(P[qb], 32);
                const int q = qb * 32 + c;
                if (g == 0 && q < Q) {
                    rs[q] = X[qb] + x2;
                    rs[Q + q] = Y[qb] + y2;
                    rs[2 * Q + q] = P[qb] + p2;
                }
            }
            const float R2 = __shfl_xor(R, 32);
            if (lane == 0) rs[3 * Q] = R + R2;
        }
        __syncthreads();
        // per-(group, row) sums over the four waves, fixed order
        for (int k = threadIdx.x; k < cb * RED; k += kThreads) {
            const int r = k / RED, e = k - r * RED;
            const float *rs = lds + L.red + r * kWaves * RED + e;
            float v = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) v += rs[w * RED];
            rowsum[((int64_t)group * N + n0 + r) * RED + e] = v;
        }
    }

    // this task's share of dZ for the rows of block i: slab [chunk][jr][M][Q]
    if (active) {
        float *pdz = part_dz + ((int64_t)blockIdx.y * njr + jr) * M * Q;
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) {
            const int q = qb * 32 + c;
            if (q >= Q) continue;
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int m = i * kTile + crow(t, g);
                if (m < M) pdz[(int64_t)m * Q + q] = dz[qb][t];
            }
        }
    }
}

// Per row: X, Y, P, R summed over the task groups (fixed order), then
//   dmu += -2 w2 P,  dS += w2^2 (X + Y) - w2 R,
// and per block of kFinRows rows the partial sums of dl and dsf2.
__global__ __launch_bounds__(256) void psi2_finalize_kernel(
    int64_t N, int Q, int groups, const float *__restrict__ rowsum,
    const float *__restrict__ w2t, const float *__restrict__ S, Hyp<float> h,
    float *__restrict__ dmu, float *__restrict__ dS, float *__restrict__ part_dl) {
    __shared__ float red[4][65];
    const int q = threadIdx.x & 63, rl = threadIdx.x >> 6;
    const int RED = 3 * Q + 1;
    const int64_t n0 = (int64_t)blockIdx.x * kFinRows;
    float dl = 0.f, dsf = 0.f;
    if (q < Q) {
        const float l = h.l[q], l2 = h.l2[q];
        for (int k = rl; k < kFinRows; k += 4) {
            const int64_t n = n0 + k;
            if (n >= N) break;
            float X = 0.f, Y = 0.f, P = 0.f, R = 0.f;
            for (int gi = 0; gi < groups; ++gi) {
                const float *rs = rowsum + ((int64_t)gi * N + n) * RED;
                X += rs[q];
                Y += rs[Q + q];
                P += rs[2 * Q + q];
                R += rs[3 * Q];
            }
            const float w2 = w2t[n * Q + q];
            const float s = S[n * Q + q];
            dmu[n * Q + q] += -2.f * w2 * P;
            dS[n * Q + q] += w2 * w2 * (X + Y) - w2 * R;
            dl += (2.f * s * w2 / l) * R + l * w2 * w2 * (X + Y) + (X - Y) / (l2 * l);
            dsf += 2.f * R;
        }
    }
    red[rl][q] = dl;
    if (q == 0) red[rl][64] = dsf;
    __syncthreads();
    if (rl == 0 && q < Q) {
        part_dl[(int64_t)blockIdx.x * (Q + 1) + q] = red[0][q] + red[1][q] + red[2][q] + red[3][q];
        if (q == 0)
            part_dl[(int64_t)blockIdx.x * (Q + 1) + Q] =
                (red[0][64] + red[1][64] + red[2][64] + red[3][64]) / h.sf2;
    }
}

// dZ, dl, dsf2 from the Psi1 partials (generic kernels) and the Psi2 partials.
__global__ void grad_reduce_kernel(int64_t N, int M, int Q, Psi1GradParts<float> p1,
                                   const float *__restrict__ pdz, int64_t dz_slabs,
                                   const float *__restrict__ pdl, int64_t dl_parts,
                                   float dL_dpsi0, float *__restrict__ dZ,
                                   float *__restrict__ dsf2, float *__restrict__ dl,
                                   int accumulate) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t MQ = (int64_t)M * Q;
    if (i < MQ) {
        float s1 = 0.f, s2 = 0.f;
        for (int64_t ch = 0; ch < p1.ncc; ++ch) s1 += p1.colpart[ch * MQ + i];
        for (int64_t sl = 0; sl < dz_slabs; ++sl) s2 += pdz[sl * MQ + i];
        dZ[i] = (accumulate ? dZ[i] : 0.f) + (s1 + s2);
    } else if (i < MQ + Q + 1) {
        const int k = (int)(i - MQ);
        float s1 = 0.f, s2 = 0.f;
        for (int64_t b = 0; b < p1.row_blocks; ++b) s1 += p1.rowpart[b * (Q + 1) + k];
        for (int64_t b = 0; b < dl_parts; ++b) s2 += pdl[b * (Q + 1) + k];
        float s = s1 + s2;
        if (k < Q) {
            dl[k] = (accumulate ? dl[k] : 0.f) + s;
        } else {
            s += dL_dpsi0 * (float)N;
            dsf2[0] = (accumulate ? dsf2[0] : 0.f) + s;
        }
    }
}

// ---------------------------------------------------------------- dispatch
template <int KS>
hipError_t launch_fwd(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                      const float *zc, const float *sq, const float *hq, const float *hl,
                      float *part, hipStream_t st) {
    auto k = psi2_fwd_kernel<KS>;
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_fwd);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)p.groups, (unsigned)p.fchunks);
    TimedScope ts(st, "mfma_psi2_fwd");
    k<<<grid, kThreads, p.lds_fwd, st>>>(s.N, (int)s.M, (int)s.Q, (int)p.Mp, p.nb, p.DS, p.T,
                                         p.tpg, p.frows, mu, Z, zc, sq, hq, hl, part);
    return hipGetLastError();
}

template <int KS, int JPW, int NQB>
hipError_t launch_grad(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                       const float *zc, const float *sq, const float *hq, const float *hl,
                       const float *w2, const float *G2p, const Hyp<float> &h, float *rowsum,
                       float *pdz, hipStream_t st) {
    auto k = psi2_grad_kernel<KS, JPW, NQB>;
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_grad);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)p.ggroups, (unsigned)p.gchunks);
    TimedScope ts(st, "mfma_psi2_grad");
    k<<<grid, kThreads, p.lds_grad, st>>>(s.N, (int)s.M, (int)s.Q, (int)p.Mp, p.nb, p.DS, p.njr,
                                          p.ntasks, p.grows, mu, Z, zc, sq, hq, hl, w2, G2p, h,
                                          rowsum, pdz);
    return hipGetLastError();
}

hipError_t dispatch_fwd(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                        const float *zc, const float *sq, const float *hq, const float *hl,
                        float *part, hipStream_t st) {
    switch (p.ks) {
#define GPPS_F(K) \
    case K: return launch_fwd<K>(p, s, mu, Z, zc, sq, hq, hl, part, st);
        GPPS_F(1) GPPS_F(2) GPPS_F(3) GPPS_F(4) GPPS_F(5) GPPS_F(6) GPPS_F(8) GPPS_F(10)
        GPPS_F(12) GPPS_F(15) GPPS_F(16) GPPS_F(24) GPPS_F(32)
#undef GPPS_F
    }
    return hipErrorInvalidValue;
}

hipError_t dispatch_grad(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                         const float *zc, const float *sq, const float *hq, const float *hl,
                         const float *w2, const float *G2p, const Hyp<float> &h, float *rowsum,
                         float *pdz, hipStream_t st) {
#define GPPS_G(K, J, Q)                                                                      \
    if (p.ks == K && p.jpw == J && p.nqb == Q)                                               \
        return launch_grad<K, J, Q>(p, s, mu, Z, zc, sq, hq, hl, w2, G2p, h, rowsum, pdz, st);
#define GPPS_G3(K, Q) GPPS_G(K, 1, Q) GPPS_G(K, 2, Q) GPPS_G(K, 4, Q)
    GPPS_G3(1, 1) GPPS_G3(2, 1) GPPS_G3(3, 1) GPPS_G3(4, 1) GPPS_G3(5, 1) GPPS_G3(6, 1)
    GPPS_G3(8, 1) GPPS_G3(10, 1) GPPS_G3(12, 1) GPPS_G3(15, 1) GPPS_G3(16, 1)
    GPPS_G3(16, 2) GPPS_G3(24, 2) GPPS_G3(32, 2)
#undef GPPS_G3
#undef GPPS_G
    return hipErrorInvalidValue;
}

hipError_t row_tables(const MPlan &p, const Shape &s, const float *S, const float *Z,
                      const Hyp<float> &h, void *ws, hipStream_t st) {
    {
        TimedScope ts(st, "mfma_rows");
        mfma_rows_kernel<<<(unsigned)cdiv(s.N, 256), 256, 0, st>>>(
            s.N, (int)s.Q, S, h, fat(ws, p.off_sq), fat(ws, p.off_hq), fat(ws, p.off_w2),
            fat(ws, p.off_hl));
    }
    TimedScope ts(st, "mfma_centre");
    mfma_centre_kernel<<<1, 64, 0, st>>>((int)s.M, (int)s.Q, Z, fat(ws, p.off_zc));
    return hipGetLastError();
}

}  // namespace

bool mfma_supports(const Shape &s) {
    const int64_t Mp = cdiv(s.M, kTile) * kTile;
    if (!((Mp <= 512 && s.Q <= 31) || (Mp <= 256 && s.Q <= GPPS_MAX_Q_MFMA))) return false;
    const MPlan p = make_mplan(s);
    return p.ks > 0 && p.lds_grad <= 160 * 1024 && p.lds_fwd <= 160 * 1024;
}

size_t mfma_workspace_bytes(const Shape &s) { return make_mplan(s).total; }

hipError_t mfma_psi_stats(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float *psi0, float *Psi1, float *Psi2,
                          int accumulate, void *ws, hipStream_t st) {
    const MPlan p = make_mplan(s);
    if (Psi1) generic_psi1_fwd<float>(s, mu, S, Z, h, Psi1, ws, st);
    hipError_t e = row_tables(p, s, S, Z, h, ws, st);
    if (e != hipSuccess) return e;
    float *part = fat(ws, p.off_fp);
    e = dispatch_fwd(p, s, mu, Z, fat(ws, p.off_zc), fat(ws, p.off_sq), fat(ws, p.off_hq),
                     fat(ws, p.off_hl), part, st);
    if (e != hipSuccess) return e;
    dim3 g((unsigned)cdiv(s.M, 16), (unsigned)cdiv(s.M, 16));
    TimedScope ts(st, "mfma_psi2_reduce");
    psi2_reduce_kernel<<<g, 256, 0, st>>>(s.N, (int)s.M, p.nb, p.T, p.fchunks, part, h.sf2, psi0,
                                          Psi2, accumulate);
    return hipGetLastError();
}

hipError_t mfma_psi_grads(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float dL_dpsi0, const float *G1,
                          const float *G2, float *dmu, float *dS, float *dZ, float *dsf2,
                          float *dl, int accumulate, void *ws, hipStream_t st) {
    const MPlan p = make_mplan(s);
    // Psi1 terms first: they overwrite dmu and dS, the Psi2 kernel adds to them.
    const Psi1GradParts<float> p1 = generic_psi1_grads<float>(s, mu, S, Z, h, G1, dmu, dS, ws, st);
    float *pdz = fat(ws, p.off_dz), *pdl = fat(ws, p.off_dl);
    if (G2) {
        hipError_t e = row_tables(p, s, S, Z, h, ws, st);
        if (e != hipSuccess) return e;
        float *G2p = fat(ws, p.off_g2);
        {
            TimedScope ts(st, "mfma_sym");
            mfma_sym_kernel<<<(unsigned)cdiv(p.Mp * p.Mp, 256), 256, 0, st>>>((int)s.M, (int)p.Mp,
                                                                              G2, G2p);
        }
        float *rowsum = fat(ws, p.off_rs);
        e = dispatch_grad(p, s, mu, Z, fat(ws, p.off_zc), fat(ws, p.off_sq), fat(ws, p.off_hq),
                          fat(ws, p.off_hl), fat(ws, p.off_w2), G2p, h, rowsum, pdz, st);
        if (e != hipSuccess) return e;
        TimedScope ts(st, "mfma_psi2_finalize");
        psi2_finalize_kernel<<<(unsigned)p.fin_blocks, 256, 0, st>>>(
            s.N, (int)s.Q, (int)p.ggroups, rowsum, fat(ws, p.off_w2), S, h, dmu, dS, pdl);
    }
    const int64_t total = s.M * s.Q + s.Q + 1;
    TimedScope ts(st, "mfma_grad_reduce");
    grad_reduce_kernel<<<(unsigned)cdiv(total, 256), 256, 0, st>>>(
        s.N, (int)s.M, (int)s.Q, p1, pdz, G2 ? p.gchunks * p.njr : 0, pdl,
        G2 ? p.fin_blocks : 0, dL_dpsi0, dZ, dsf2, dl, accumulate);
    return hipGetLastError();
}

}  // namespace gpps
