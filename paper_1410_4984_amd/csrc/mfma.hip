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
// row and column terms are added to the MFMA's C input; exp2 is one v_exp_f32.
//
// Gradient (Alg. 2): with W_n = G2s o Psi2_n (G2s the symmetric part of
// dL/dPsi2), r_n = W_n 1 and V_n = W_n D_n (D_n[m, q] = d_mq), every derivative
// is linear in r_n and V_n:
//   dmu_nq   = -2 w2 sum_m d r
//   dS_nq    = w2^2 (X + Y) - w2 R,        X = sum_m d^2 r, Y = sum_m d V, R = sum_m r
//   dZ_mq   += V (w2 - 1/l^2) + d r (w2 + 1/l^2)
//   dl_q    += (2 S w2 / l) R + l w2^2 (X + Y) + (X - Y) / l^3
//   dsf2    += 2 R / sf2
// V_n is a second MFMA product whose A operand is the W tile exactly as the
// first MFMA left it in registers (no data movement); r_n is the ones column
// appended to D_n.
//
// Work split.  Forward: a workgroup owns a group of upper-triangular 32 x 32
// pair tiles and a chunk of datapoints; each wave keeps its tiles' running
// sums in registers; per-chunk partial tiles are reduced in a fixed order.
// Gradient: a workgroup owns every tile of a chunk of datapoints (the full
// M x M W_n is needed to complete r_n and V_n), each wave owns whole row
// blocks of V_n.  Per-datapoint tables (d, b) are staged in LDS, double
// buffered, one barrier per datapoint.  No atomics: every cross-wave or
// cross-workgroup sum runs in a fixed order, so results are bitwise
// reproducible.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace gpps {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kTile = 32;
constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kSqStride = 64;          // per-row stride of the sqrt(log2e kappa) table
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kPadBias = -1.0e30f;   // b of a padded inducing row: exp2 -> 0
constexpr int kMaxTilesPerWave = 4;    // forward
constexpr int64_t kFwdTargetWGs = 1024;
constexpr int64_t kGradTargetWGs = 512;

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Row of the 32x32 C/D register layout: lane l holds column l % 32 and, in
// register t, row 8 (t / 4) + 4 (l / 32) + t % 4.
__device__ __forceinline__ int crow(int t, int g) { return 8 * (t >> 2) + 4 * g + (t & 3); }

struct MPlan {
    int64_t Mp;            // M rounded up to the tile edge
    int nb;                // tiles per edge
    int nqb;               // 32-column blocks of D (Q + 1 columns incl. the ones column)
    int DS;                // LDS row stride of D (odd: conflict-free column reads)
    int ks;                // MFMA k-steps (2 latent dimensions each), instantiated value
    int bpw;               // gradient: row blocks per wave
    int64_t T;             // upper-triangular tiles
    int64_t tpg, groups;   // forward: tiles per group, groups
    int64_t frows, fchunks;
    int64_t grows, gchunks;
    size_t lds_fwd, lds_grad;
    size_t off_sq, off_hq, off_w2, off_hl, off_g2, off_fp, off_dz, off_dl, total;
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

MPlan make_mplan(const Shape &s) {
    MPlan p{};
    p.Mp = cdiv(s.M, kTile) * kTile;
    p.nb = (int)(p.Mp / kTile);
    p.nqb = s.Q + 1 <= 32 ? 1 : 2;
    p.DS = 32 * p.nqb + 1;
    p.ks = round_ks((int)cdiv(s.Q, 2), p.nqb);
    p.bpw = (int)cdiv(p.nb, kWaves);
    if (p.bpw == 3) p.bpw = 4;
    p.T = (int64_t)p.nb * (p.nb + 1) / 2;
    p.groups = cdiv(p.T, kWaves * kMaxTilesPerWave);
    p.tpg = cdiv(p.T, p.groups);
    p.fchunks = std::max<int64_t>(1, std::min(cdiv(kFwdTargetWGs, p.groups), cdiv(s.N, 32)));
    p.frows = cdiv(s.N, p.fchunks);
    p.fchunks = cdiv(s.N, p.frows);
    p.gchunks = std::max<int64_t>(1, std::min(kGradTargetWGs, cdiv(s.N, 16)));
    p.grows = cdiv(s.N, p.gchunks);
    p.gchunks = cdiv(s.N, p.grows);
    const size_t buf = (size_t)p.Mp * p.DS + p.Mp;           // floats per LDS buffer
    p.lds_fwd = 2 * buf * sizeof(float);
    p.lds_grad = p.lds_fwd + 2 * kWaves * (3 * 32 * p.nqb + 1) * sizeof(float);
    size_t o = generic_workspace_bytes(s, sizeof(float));   // Psi1 pieces live first
    auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
    p.off_sq = take(sizeof(float) * s.N * kSqStride);
    p.off_hq = take(sizeof(float) * s.N * s.Q);
    p.off_w2 = take(sizeof(float) * s.N * s.Q);
    p.off_hl = take(sizeof(float) * s.N);
    p.off_g2 = take(sizeof(float) * p.Mp * p.Mp);
    p.off_fp = take(sizeof(float) * p.fchunks * p.T * kTile * kTile);
    p.off_dz = take(sizeof(float) * p.gchunks * s.M * s.Q);
    p.off_dl = take(sizeof(float) * p.gchunks * (s.Q + 1));
    p.total = o;
    return p;
}

float *fat(void *ws, size_t off) { return reinterpret_cast<float *>(static_cast<char *>(ws) + off); }

// ---------------------------------------------------------------- per-row tables
// sq[n][q] = sqrt(log2e * kappa_nq) (zero for q >= Q up to the stride),
// hq[n][q] = -log2e/4 (1/l^2 + w2), w2[n][q], hl[n] = log2e (log sf2 - 1/4 sum_q log(1 + 2S/l^2)).
__global__ void mfma_rows_kernel(int64_t N, int Q, const float *__restrict__ S, Hyp<float> h,
                                 float *__restrict__ sq, float *__restrict__ hq,
                                 float *__restrict__ w2t, float *__restrict__ hl) {
    const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= N) return;
    float lsum = 0.f;
    for (int q = 0; q < kSqStride; ++q) {
        if (q < Q) {
            const float s = S[n * Q + q];
            const float l2 = h.l2[q];
            const float w2 = 1.f / (l2 + 2.f * s);
            const float kap = s * w2 / l2;
            sq[n * kSqStride + q] = sqrtf(kLog2e * kap);
            hq[n * Q + q] = -0.25f * kLog2e * (1.f / l2 + w2);
            w2t[n * Q + q] = w2;
            lsum += log1pf(2.f * s / l2);
        } else {
            sq[n * kSqStride + q] = 0.f;
        }
    }
    hl[n] = kLog2e * (h.log_sf2 - 0.25f * lsum);
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
// One buffer: D [Mp][DS] (d_mq for q < Q, 1 in column Q for real rows, 0
// elsewhere) followed by b [Mp].  Constant parts are written once per kernel.
__device__ void stage_init(float *buf, int M, int Mp, int Q, int DS) {
    for (int i = threadIdx.x; i < Mp * DS; i += kThreads) {
        const int m = i / DS, c = i - m * DS;
        buf[i] = (c == Q && m < M) ? 1.f : 0.f;
    }
    for (int m = threadIdx.x; m < Mp; m += kThreads) buf[Mp * DS + m] = m < M ? 0.f : kPadBias;
}

__device__ void stage_row(float *buf, int64_t n, int M, int Q, int DS,
                          const float *__restrict__ mu, const float *__restrict__ Z,
                          const float *__restrict__ hq, const float *__restrict__ hl, int Mp) {
    const float *mun = mu + n * Q;
    const float *hqn = hq + n * Q;
    const float hln = hl[n];
    for (int m = threadIdx.x; m < M; m += kThreads) {
        float *row = buf + m * DS;
        const float *zm = Z + (int64_t)m * Q;
        float b = hln;
        for (int q = 0; q < Q; ++q) {
            const float d = mun[q] - zm[q];
            row[q] = d;
            b = fmaf(hqn[q] * d, d, b);
        }
        buf[Mp * DS + m] = b;
    }
}

// Gram tile (rows from block `rb`, columns from block `cb`) plus the row and
// column terms, in log2 units, for the datapoint staged in `buf`.
template <int KS>
__device__ __forceinline__ v16f gram_tile(const float *buf, int Mp, int DS, int rb, int cb,
                                          const float (&mult)[KS], const float (&bop)[KS],
                                          float bcol, int c, int g) {
    const float *bv = buf + Mp * DS;
    v16f acc;
#pragma unroll
    for (int t = 0; t < 16; ++t) acc[t] = bv[rb * kTile + crow(t, g)] + bcol;
    const float *arow = buf + (rb * kTile + c) * DS + g;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const float a = arow[2 * s] * mult[s];
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bop[s], acc, 0, 0, 0);
    }
    (void)cb;
    return acc;
}

// ---------------------------------------------------------------- Psi2 forward
template <int KS>
__global__ __launch_bounds__(kThreads) void psi2_fwd_kernel(
    int64_t N, int M, int Q, int Mp, int nb, int DS, int64_t T, int64_t tpg,
    int64_t rows_per_chunk, const float *__restrict__ mu, const float *__restrict__ Z,
    const float *__restrict__ sq, const float *__restrict__ hq, const float *__restrict__ hl,
    float *__restrict__ partial) {
    extern __shared__ float lds[];
    const int bufsz = Mp * DS + Mp;
    float *bufs[2] = {lds, lds + bufsz};
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c = lane & 31, g = lane >> 5;

    // this wave's tiles: t = t0 + wave + 4 k
    const int64_t t0 = (int64_t)blockIdx.x * tpg, t1 = min(T, t0 + tpg);
    int ti[kMaxTilesPerWave], tj[kMaxTilesPerWave];
    bool tv[kMaxTilesPerWave];
#pragma unroll
    for (int k = 0; k < kMaxTilesPerWave; ++k) {
        int64_t t = t0 + wave + kWaves * k;
        tv[k] = t < t1;
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

    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    const int cnt = (int)(r1 - r0);
    stage_init(bufs[0], M, Mp, Q, DS);
    stage_init(bufs[1], M, Mp, Q, DS);
    __syncthreads();
    stage_row(bufs[0], r0, M, Q, DS, mu, Z, hq, hl, Mp);
    __syncthreads();
    for (int it = 0; it < cnt; ++it) {
        const int64_t n = r0 + it;
        const float *buf = bufs[it & 1];
        if (it + 1 < cnt) stage_row(bufs[(it + 1) & 1], n + 1, M, Q, DS, mu, Z, hq, hl, Mp);
        float mult[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) mult[s] = sq[n * kSqStride + 2 * s + g];
#pragma unroll
        for (int k = 0; k < kMaxTilesPerWave; ++k) {
            if (!tv[k]) continue;
            // B operand: column block tj
            float bop[KS];
            const float *brow = buf + (tj[k] * kTile + c) * DS + g;
#pragma unroll
            for (int s = 0; s < KS; ++s) bop[s] = brow[2 * s] * mult[s];
            const float bcol = buf[Mp * DS + tj[k] * kTile + c];
            v16f e = gram_tile<KS>(buf, Mp, DS, ti[k], tj[k], mult, bop, bcol, c, g);
#pragma unroll
            for (int t = 0; t < 16; ++t) acc[k][t] += __builtin_amdgcn_exp2f(e[t]);
        }
        __syncthreads();
    }
    // partial tiles, row-major inside the tile
#pragma unroll
    for (int k = 0; k < kMaxTilesPerWave; ++k) {
        if (!tv[k]) continue;
        const int64_t t = t0 + wave + kWaves * k;
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
template <int KS, int BPW, int NQB>
__global__ __launch_bounds__(kThreads) void psi2_grad_kernel(
    int64_t N, int M, int Q, int Mp, int nb, int DS, int64_t rows_per_chunk,
    const float *__restrict__ mu, const float *__restrict__ S, const float *__restrict__ Z,
    const float *__restrict__ sq, const float *__restrict__ hq, const float *__restrict__ hl,
    const float *__restrict__ w2t, const float *__restrict__ G2p, Hyp<float> h,
    float *__restrict__ dmu, float *__restrict__ dS, float *__restrict__ part_dz,
    float *__restrict__ part_dl) {
    extern __shared__ float lds[];
    const int bufsz = Mp * DS + Mp;
    float *bufs[2] = {lds, lds + bufsz};
    constexpr int QV = 32 * NQB;
    constexpr int RED = 3 * QV + 1;            // X, Y, P per latent dimension, then R
    float *red = lds + 2 * bufsz;              // [2 slots][kWaves][RED]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c = lane & 31, g = lane >> 5;
    const int ones_src = 32 * g + (Q & 31);    // lane holding column Q (the row sums)
    const int ones_qb = Q >> 5;

    v16f dz[BPW][NQB];
#pragma unroll
    for (int ib = 0; ib < BPW; ++ib)
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
            for (int t = 0; t < 16; ++t) dz[ib][qb][t] = 0.f;
    // per-lane constants for the latent dimensions this lane finalises (wave 0)
    float dl_acc[NQB], dsf_acc = 0.f;
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) dl_acc[qb] = 0.f;

    const int64_t r0 = (int64_t)blockIdx.x * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    const int cnt = (int)(r1 - r0);

    // finalise datapoint n from the per-wave sums in red slot `slot` (wave 0, lanes q < Q)
    auto finalise = [&](int64_t n, int slot) {
        if (wave != 0 || g != 0) return;
        const float *rs = red + slot * kWaves * RED;
        float R = 0.f;
        for (int w = 0; w < kWaves; ++w) R += rs[w * RED + 3 * QV];
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) {
            const int q = qb * 32 + c;
            if (q >= Q) continue;
            float X = 0.f, Y = 0.f, P = 0.f;
            for (int w = 0; w < kWaves; ++w) {
                X += rs[w * RED + q];
                Y += rs[w * RED + QV + q];
                P += rs[w * RED + 2 * QV + q];
            }
            const float w2 = w2t[n * Q + q];
            const float s = S[n * Q + q];
            const float l = h.l[q];
            dmu[n * Q + q] += -2.f * w2 * P;
            dS[n * Q + q] += w2 * w2 * (X + Y) - w2 * R;
            dl_acc[qb] += (2.f * s * w2 / l) * R + l * w2 * w2 * (X + Y) + (X - Y) / (h.l2[q] * l);
        }
        if (c == 0) dsf_acc += 2.f * R;
    };

    stage_init(bufs[0], M, Mp, Q, DS);
    stage_init(bufs[1], M, Mp, Q, DS);
    __syncthreads();
    if (cnt > 0) stage_row(bufs[0], r0, M, Q, DS, mu, Z, hq, hl, Mp);
    __syncthreads();
    for (int it = 0; it < cnt; ++it) {
        const int64_t n = r0 + it;
        const float *buf = bufs[it & 1];
        if (it + 1 < cnt) stage_row(bufs[(it + 1) & 1], n + 1, M, Q, DS, mu, Z, hq, hl, Mp);
        if (it > 0) finalise(n - 1, (it - 1) & 1);

        float mult[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) mult[s] = sq[n * kSqStride + 2 * s + g];
        float alpha[NQB], beta[NQB];
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) {
            const int q = qb * 32 + c;
            const float w2 = q < Q ? w2t[n * Q + q] : 0.f;
            const float il2 = q < Q ? 1.f / h.l2[q] : 0.f;
            alpha[qb] = w2 - il2;
            beta[qb] = w2 + il2;
        }
        float X[NQB], Y[NQB], P[NQB], R = 0.f;
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) X[qb] = Y[qb] = P[qb] = 0.f;

#pragma unroll
        for (int ib = 0; ib < BPW; ++ib) {
            const int i = wave + kWaves * ib;
            if (i >= nb) continue;
            // Gram B operand: column block i (the m index of W)
            float bop[KS];
            const float *brow = buf + (i * kTile + c) * DS + g;
#pragma unroll
            for (int s = 0; s < KS; ++s) bop[s] = brow[2 * s] * mult[s];
            const float bcol = buf[Mp * DS + i * kTile + c];
            v16f V[NQB];
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
                for (int t = 0; t < 16; ++t) V[qb][t] = 0.f;
            for (int j = 0; j < nb; ++j) {
                // rows m' in block j, columns m in block i
                v16f e = gram_tile<KS>(buf, Mp, DS, j, i, mult, bop, bcol, c, g);
                const float *g2 = G2p + (int64_t)(j * kTile) * Mp + i * kTile + c;
                const float *drow = buf + j * kTile * DS + c;
#pragma unroll
                for (int t = 0; t < 16; ++t) {
                    const int rr = crow(t, g);
                    const float w = g2[(int64_t)rr * Mp] * __builtin_amdgcn_exp2f(e[t]);
#pragma unroll
                    for (int qb = 0; qb < NQB; ++qb)
                        V[qb] = __builtin_amdgcn_mfma_f32_32x32x2f32(w, drow[rr * DS + qb * 32],
                                                                     V[qb], 0, 0, 0);
                }
            }
            // epilogue for rows m = i*32 + crow(t, g): r from the ones column
            const float *dblk = buf + i * kTile * DS;
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int rr = crow(t, g);
                const float r = __int_as_float(__builtin_amdgcn_ds_bpermute(
                    ones_src * 4, __float_as_int(ones_qb == 0 ? V[0][t] : V[NQB - 1][t])));
                R += r;
#pragma unroll
                for (int qb = 0; qb < NQB; ++qb) {
                    const float d = dblk[rr * DS + qb * 32 + c];
                    const float dr = d * r;
                    const float v = V[qb][t];
                    dz[ib][qb][t] = fmaf(alpha[qb], v, fmaf(beta[qb], dr, dz[ib][qb][t]));
                    X[qb] = fmaf(dr, d, X[qb]);
                    P[qb] += dr;
                    Y[qb] = fmaf(d, v, Y[qb]);
                }
            }
        }
        // combine the two lane halves, then publish this wave's sums
        float *rs = red + (it & 1) * kWaves * RED + wave * RED;
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) {
            const float x2 = __shfl_xor(X[qb], 32), y2 = __shfl_xor(Y[qb], 32),
                        p2 = __shfl_xor(P[qb], 32);
            if (g == 0) {
                rs[qb * 32 + c] = X[qb] + x2;
                rs[QV + qb * 32 + c] = Y[qb] + y2;
                rs[2 * QV + qb * 32 + c] = P[qb] + p2;
            }
        }
        const float R2 = __shfl_xor(R, 32);
        if (lane == 0) rs[3 * QV] = R + R2;
        __syncthreads();
    }
    if (cnt > 0) finalise(r1 - 1, (cnt - 1) & 1);

    // per-chunk partials: dZ rows owned by this wave, dl / dsf2 from wave 0
    float *pdz = part_dz + (int64_t)blockIdx.x * M * Q;
#pragma unroll
    for (int ib = 0; ib < BPW; ++ib) {
        const int i = wave + kWaves * ib;
        if (i >= nb) continue;
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) {
            const int q = qb * 32 + c;
            if (q >= Q) continue;
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int m = i * kTile + crow(t, g);
                if (m < M) pdz[(int64_t)m * Q + q] = dz[ib][qb][t];
            }
        }
    }
    if (wave == 0 && g == 0) {
        float *pdl = part_dl + (int64_t)blockIdx.x * (Q + 1);
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) {
            const int q = qb * 32 + c;
            if (q < Q) pdl[q] = dl_acc[qb];
        }
        if (c == 0) pdl[Q] = dsf_acc / h.sf2;
    }
}

// dZ, dl, dsf2 from the Psi1 partials (generic kernels) and the Psi2 partials.
__global__ void grad_reduce_kernel(int64_t N, int M, int Q, Psi1GradParts<float> p1,
                                   const float *__restrict__ pdz, const float *__restrict__ pdl,
                                   int64_t gchunks, bool has_psi2, float dL_dpsi0,
                                   float *__restrict__ dZ, float *__restrict__ dsf2,
                                   float *__restrict__ dl, int accumulate) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t MQ = (int64_t)M * Q;
    if (i < MQ) {
        float s1 = 0.f, s2 = 0.f;
        for (int64_t ch = 0; ch < p1.ncc; ++ch) s1 += p1.colpart[ch * MQ + i];
        if (has_psi2)
            for (int64_t ch = 0; ch < gchunks; ++ch) s2 += pdz[ch * MQ + i];
        dZ[i] = (accumulate ? dZ[i] : 0.f) + (s1 + s2);
    } else if (i < MQ + Q + 1) {
        const int k = (int)(i - MQ);
        float s1 = 0.f, s2 = 0.f;
        for (int64_t b = 0; b < p1.row_blocks; ++b) s1 += p1.rowpart[b * (Q + 1) + k];
        if (has_psi2)
            for (int64_t ch = 0; ch < gchunks; ++ch) s2 += pdl[ch * (Q + 1) + k];
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
                      const float *sq, const float *hq, const float *hl, float *part,
                      hipStream_t st) {
    auto k = psi2_fwd_kernel<KS>;
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_fwd);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)p.groups, (unsigned)p.fchunks);
    TimedScope ts(st, "mfma_psi2_fwd");
    k<<<grid, kThreads, p.lds_fwd, st>>>(s.N, (int)s.M, (int)s.Q, (int)p.Mp, p.nb, p.DS, p.T,
                                         p.tpg, p.frows, mu, Z, sq, hq, hl, part);
    return hipGetLastError();
}

template <int KS, int BPW, int NQB>
hipError_t launch_grad(const MPlan &p, const Shape &s, const float *mu, const float *S,
                       const float *Z, const float *sq, const float *hq, const float *hl,
                       const float *w2, const float *G2p, const Hyp<float> &h, float *dmu,
                       float *dS, float *pdz, float *pdl, hipStream_t st) {
    auto k = psi2_grad_kernel<KS, BPW, NQB>;
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_grad);
    if (e != hipSuccess) return e;
    TimedScope ts(st, "mfma_psi2_grad");
    k<<<(unsigned)p.gchunks, kThreads, p.lds_grad, st>>>(s.N, (int)s.M, (int)s.Q, (int)p.Mp, p.nb,
                                                        p.DS, p.grows, mu, S, Z, sq, hq, hl, w2,
                                                        G2p, h, dmu, dS, pdz, pdl);
    return hipGetLastError();
}

hipError_t dispatch_fwd(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                        const float *sq, const float *hq, const float *hl, float *part,
                        hipStream_t st) {
    switch (p.ks) {
#define GPPS_F(K) \
    case K: return launch_fwd<K>(p, s, mu, Z, sq, hq, hl, part, st);
        GPPS_F(1) GPPS_F(2) GPPS_F(3) GPPS_F(4) GPPS_F(5) GPPS_F(6) GPPS_F(8) GPPS_F(10)
        GPPS_F(12) GPPS_F(15) GPPS_F(16) GPPS_F(24) GPPS_F(32)
#undef GPPS_F
    }
    return hipErrorInvalidValue;
}

hipError_t dispatch_grad(const MPlan &p, const Shape &s, const float *mu, const float *S,
                         const float *Z, const float *sq, const float *hq, const float *hl,
                         const float *w2, const float *G2p, const Hyp<float> &h, float *dmu,
                         float *dS, float *pdz, float *pdl, hipStream_t st) {
#define GPPS_G(K, B, Q)                                                                      \
    if (p.ks == K && p.bpw == B && p.nqb == Q)                                               \
        return launch_grad<K, B, Q>(p, s, mu, S, Z, sq, hq, hl, w2, G2p, h, dmu, dS, pdz, pdl, st);
#define GPPS_G3(K) GPPS_G(K, 1, 1) GPPS_G(K, 2, 1) GPPS_G(K, 4, 1)
    GPPS_G3(1) GPPS_G3(2) GPPS_G3(3) GPPS_G3(4) GPPS_G3(5) GPPS_G3(6) GPPS_G3(8) GPPS_G3(10)
    GPPS_G3(12) GPPS_G3(15) GPPS_G3(16)
    GPPS_G(16, 1, 2) GPPS_G(16, 2, 2) GPPS_G(24, 1, 2) GPPS_G(24, 2, 2) GPPS_G(32, 1, 2)
    GPPS_G(32, 2, 2)
#undef GPPS_G3
#undef GPPS_G
    return hipErrorInvalidValue;
}

hipError_t rows_tables(const MPlan &p, const Shape &s, const float *S, const Hyp<float> &h,
                       void *ws, hipStream_t st) {
    TimedScope ts(st, "mfma_rows");
    mfma_rows_kernel<<<(unsigned)cdiv(s.N, 256), 256, 0, st>>>(
        s.N, (int)s.Q, S, h, fat(ws, p.off_sq), fat(ws, p.off_hq), fat(ws, p.off_w2),
        fat(ws, p.off_hl));
    return hipGetLastError();
}

}  // namespace

bool mfma_supports(const Shape &s) {
    const int64_t Mp = cdiv(s.M, kTile) * kTile;
    if (!((Mp <= 512 && s.Q <= 31) || (Mp <= 256 && s.Q <= GPPS_MAX_Q_MFMA))) return false;
    const MPlan p = make_mplan(s);
    return p.ks > 0 && p.lds_grad <= 160 * 1024;
}

size_t mfma_workspace_bytes(const Shape &s) { return make_mplan(s).total; }

hipError_t mfma_psi_stats(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float *psi0, float *Psi1, float *Psi2,
                          int accumulate, void *ws, hipStream_t st) {
    const MPlan p = make_mplan(s);
    if (Psi1) generic_psi1_fwd<float>(s, mu, S, Z, h, Psi1, ws, st);
    hipError_t e = rows_tables(p, s, S, h, ws, st);
    if (e != hipSuccess) return e;
    float *part = fat(ws, p.off_fp);
    e = dispatch_fwd(p, s, mu, Z, fat(ws, p.off_sq), fat(ws, p.off_hq), fat(ws, p.off_hl), part, st);
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
        hipError_t e = rows_tables(p, s, S, h, ws, st);
        if (e != hipSuccess) return e;
        float *G2p = fat(ws, p.off_g2);
        {
            TimedScope ts(st, "mfma_sym");
            mfma_sym_kernel<<<(unsigned)cdiv(p.Mp * p.Mp, 256), 256, 0, st>>>((int)s.M, (int)p.Mp,
                                                                              G2, G2p);
        }
        e = dispatch_grad(p, s, mu, S, Z, fat(ws, p.off_sq), fat(ws, p.off_hq), fat(ws, p.off_hl),
                          fat(ws, p.off_w2), G2p, h, dmu, dS, pdz, pdl, st);
        if (e != hipSuccess) return e;
    }
    const int64_t total = s.M * s.Q + s.Q + 1;
    TimedScope ts(st, "mfma_grad_reduce");
    grad_reduce_kernel<<<(unsigned)cdiv(total, 256), 256, 0, st>>>(
        s.N, (int)s.M, (int)s.Q, p1, pdz, pdl, p.gchunks, G2 != nullptr, dL_dpsi0, dZ, dsf2, dl,
        accumulate);
    return hipGetLastError();
}

}  // namespace gpps
