// Matrix-core path (F32, gfx950): the O(N M^2 Q) Psi2 statistic and its
// gradient on the matrix cores, with exp2 and the dL/dPsi2 weighting on the
// vector ALU.
//
// Precision.  Both contractions run on v_mfma_f32_32x32x16_f16 with both
// operands split into two fp16 parts rounded to nearest, x = x_hi + x_lo
// (22 significant bits); three of the four cross products are kept (the dropped
// one is below 2^-22 |a||b|) and all products accumulate in fp32.  In the Gram
// product the three cross products share one K range: each dimension takes three
// k slots (hi*hi, hi*lo, lo*hi) and the column bias two, so Q = 20 needs 62
// slots, four 16-slot instructions instead of six.  The f16 MFMA does 16 times
// the work per cycle of v_mfma_f32_32x32x2_f32 and, unlike it, lets the vector
// ALU issue while it runs, which is where exp2, the weighting and the splits
// execute.
//
// Per datapoint n the Psi2 summand is a Gram matrix pushed through exp
// (section 2, eq. (4): Phi turned into an expectation under q(x_n); Alg. 1
// computes it per pair of inducing inputs and sums over datapoints).  With
// d_m = mu_n - z_m (per dimension q) and w2 = 1/(l^2 + 2 S_nq), the closed form
//   Psi2_n[m, m'] = sf2^2 prod_q (1 + 2S/l^2)^(-1/2)
//                   exp(-sum_q [(z_m - z_m')^2/(4 l^2) + (mu - (z_m + z_m')/2)^2 w2])
// has an n-independent factor 2^C_mm', C_mm' = -log2(e) sum_q (z_m - z_m')^2/(4 l^2),
// which is taken out of the sum over n: Psi2 = 2^C o sum_n 2^E'_n.  The rest,
// E'_n = 2 hl_n - log2(e) sum_q w2 (d_m + d_m')^2 / 4 <= 2 hl_n, splits exactly into
// a row term, a column term and a Gram term:
//   E'_n[m, m'] = b_m + b_m' + sum_q K_q d_mq d_m'q,     K = -log2(e) w2 / 2,
//   b_m = hl_n - log2(e)/4 sum_q w2 d_mq^2,   hl_n = log2(e) (log sf2 - 1/4 sum_q log(1 + 2S/l^2)).
// The Gram term is written with one side independent of n:
//   sum_q K d_mq d_m'q = c_m + sum_q (z_m'q s_q) (-K_q d_mq / s_q),  c_m = sum_q K_q d_mq mu_q,
// so one MFMA operand is the (centred) z table scaled per dimension by the power
// of two s_q that brings max_m |z_mq| into (1/2, 1], and the other, -K d / s, is
// formed once per datapoint and row block.  b and b + c come from a per-call
// table (mfma_rowterm_kernel); exp2 is one v_exp_f32.  Inputs are centred (Z and
// mu shifted by the mean inducing input), which changes no result: every
// quantity depends on mu - z only.
//
// Range.  Every fp16 operand is bounded before the kernels run: per datapoint,
// |-K d / s| <= log2(e)/2 w2 (|mu| + R_q) / s_q and |b + c| <= |hl| + log2(e)/4
// sum_q w2 (|mu| + R_q)(3 |mu| + R_q), with R_q = max_m |z_mq| (centred).  A guard
// kernel evaluates these bounds over all rows (O(N Q)) and writes a route word:
// when a bound reaches kOperandLimit (or R_q reaches kZLimit, the range of the
// unscaled z table of the gradient's second product) the matrix-core kernels of
// the call return at once and the generic kernels, enqueued after them on the
// same stream, compute the call instead.  Nothing is clamped.  Taking C out of the
// sum keeps the split terms of the summands that matter small: for those, w2 d_m^2,
// w2 d_m'^2 and the Gram term are bounded by a few times |E'| whatever the
// lengthscales (w2 <= 1/l^2), so the exponent error stays a few 2^-22 of the
// exponent's own size, and the per-dimension scale makes the operands invariant
// under a common scaling of mu, Z and l.  The guard also sends calls whose
// inducing inputs spread over more than kSpreadLimit lengthscales (R_q / l_q) to
// the generic kernels, for the accuracy of the gradient (mfma_guard_kernel).  W in the gradient's second product is scaled per
// datapoint by a power of two that bounds it by 2^14, and the product is scaled
// back exactly.
//
// Gradient (Alg. 2): with W_n = G2s o Psi2_n (G2s the symmetric part of
// dL/dPsi2), r_n = W_n 1 and V_n = W_n D_n (D_n[m, q] = d_mq), every derivative
// is linear in r_n and V_n (and W_n = G2c o 2^E'_n, where G2c = G2s o 2^C is
// formed once per call):
//   dmu_nq   = -2 w2 sum_m d r
//   dS_nq    = w2^2 (X + Y) - w2 R,        X = sum_m d^2 r, Y = sum_m d V, R = sum_m r
//   dZ_mq   += V (w2 - 1/l^2) + d r (w2 + 1/l^2)
//   dl_q    += (2 S w2 / l) R + l w2^2 (X + Y) + (X - Y) / l^3
//   dsf2    += 2 R / sf2
// Since D_n = 1 mu_n^T - Z, V_n = r_n mu_n^T - W_n Z: the second MFMA product
// is W_n [Z | 1], whose B operand is the constant z table and whose ones
// column yields r_n.  Its A operand is the W tile exactly as the first MFMA
// left it in registers.  The Psi1 terms (t = dL/dPsi1 * Psi1) join the same
// epilogue: dmu -= w1 sum_m t d, dS += 1/2 w1^2 sum_m t d^2 - 1/2 w1 sum_m t,
// dZ += t d w1, with w1 = 1/(l^2 + S).
//
// Work split.  The split z tables are staged in LDS once per workgroup.  Rows
// are processed in batches whose per-row values and row terms are copied into
// LDS (the forward prefetches the next batch into registers); then every wave
// runs its rows with no further barrier.  Forward: a wave task is a run of
// upper-triangular 32 x 32 pair tiles in one row block; its running sums stay
// in registers; partial tiles are reduced over row chunks in a fixed order.
// Gradient: every term above is linear in (r_n, V_n), so the full M x M tile
// grid is split into wave tasks (one row block of W, four column blocks) whose
// dL/dPsi2 tiles stay in registers; each task adds its share of dZ (registers)
// and of the per-row sums (LDS, then global), which a finalize kernel
// combines.  No atomics;
// every cross-wave or cross-workgroup sum runs in a fixed order, so results
// are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <type_traits>

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
constexpr float kPadBias = -1.0e30f;   // row term (fp32) of a padded inducing input: exp2 -> 0
// column bias of a padded inducing input, exact in fp16: its z is 0, so the range
// guard's bound on |b + c| (>= its Gram term plus |hl| + 128) keeps its exponent
// below -128 + the gradient's row scale (<= 120): exp2 is finite and tiny, and
// dL/dPsi2 is zero there
constexpr float kPadBiasCol = -6.0e4f;
constexpr float kOperandLimit = 6.0e4f; // guard: largest fp16 Gram operand or bias (fp16 max 65504)
constexpr float kZLimit = 3.0e4f;       // guard: largest centred |z| (unscaled fp16 z table)
constexpr float kSpreadLimit = 64.f;    // guard: largest R_q / l_q (gradient conditioning)
constexpr int kRB = 8;                 // gradient: rows per batch
constexpr int kFRB = 4;                // forward: rows per batch (prefetched a batch ahead)
constexpr int kGPF = 4;                // gradient: per-thread load slots of a staged row table
static_assert(kGPF * 64 >= kRB * 32, "kGPF slots cover the [kRB][32 wpg] row tables of any workgroup");
static_assert(kFRB * kRowStride == kThreads, "one mu / kappa value per forward thread");
constexpr int64_t kCUs = 256;          // compute units of one MI355X
constexpr int64_t kLdsBytes = 160 * 1024;
constexpr int kFinRows = 64;           // rows per block of the gradient finalize kernel
constexpr int kRTRows = 32;            // rows per block of the row-term kernel
// gradient: column blocks per wave task (the dL/dPsi2 tiles it holds in registers)
constexpr int grad_jpw(int nqb) { return nqb == 1 ? 4 : 2; }
// gradient: most waves per workgroup (one row block each); with two q-blocks
// a wave needs more than 256 registers, so only one wave per SIMD
constexpr int grad_waves(int nqb) { return nqb == 1 ? 8 : 4; }

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Row of the 32x32 C/D register layout: lane l holds column l % 32 and, in
// register t, row 8 (t / 4) + 4 (l / 32) + t % 4.
__device__ __forceinline__ int crow(int t, int g) { return 8 * (t >> 2) + 4 * g + (t & 3); }

// Forward wave tasks: row block ti, tiles tj = tj0 .. tj0 + TPW - 1 (clamped to
// the last block; clamped tiles are computed but never written).
__host__ __device__ inline int fwd_tasks(int nb, int tpw) {
    int n = 0;
    for (int ti = 0; ti < nb; ++ti) n += (nb - ti + tpw - 1) / tpw;
    return n;
}

__device__ inline void fwd_task(int task, int nb, int tpw, int &ti, int &tj0) {
    for (ti = 0; ti < nb; ++ti) {
        const int k = (nb - ti + tpw - 1) / tpw;
        if (task < k) break;
        task -= k;
    }
    tj0 = ti + task * tpw;
}

// Packed Gram layout over NK 16-slot f16 MFMA instructions.  The per-datapoint
// operand (B, column m) holds the fp16 parts hi + lo of x_q = (z_mq - mu_q) K_q,
// the constant one (A, row m') those of the centred z_m'q; the three kept cross
// products share one K range.  Each lane group (g = lane / 32) holds 8 k slots
// per instruction, 4 NK packed f16 pairs (dwords) in all, and takes the
// T = gram_t(NK) dimensions q = g T .. g T + T - 1, in pairs (a, b):
//   dwords [0, NP)       B (x_hi,a, x_hi,b)   A (z_hi,a, z_hi,b)
//          [NP, 2NP)     B (x_lo,a, x_lo,b)   A (z_hi,a, z_hi,b)
//          [2NP, 3NP)    B (x_hi,a, x_hi,b)   A (z_lo,a, z_lo,b)
//          an odd dimension s, if any: B (x_hi, x_lo), (x_hi, 0); A (z_hi, z_hi), (z_lo, 0)
//          the bias b + c: B (hi, lo) in lane group 1, zero in group 0; A (1, 1)
//          zero beyond.
// Dimensions past Q have zero z, mu and K, so their slots contribute nothing.
constexpr int gram_np(int nk) { return (4 * nk - 1) / 3; }
constexpr int gram_odd(int nk) { return (4 * nk - 1) - 3 * gram_np(nk) >= 2 ? 1 : 0; }
constexpr int gram_t(int nk) { return 2 * gram_np(nk) + gram_odd(nk); }
// instructions for Q dimensions (instantiated counts only): Q <= 4, 8, 14, 20,
// 30, 40, 52, 62
inline int gram_nk(int64_t Q) {
    for (int nk : {1, 2, 3, 4, 6, 8, 10, 12})
        if (2 * gram_t(nk) >= Q) return nk;
    return -1;
}

// Widest forward task (tiles per wave) whose registers fit two waves per SIMD
// without spilling, for nk Gram instructions.
constexpr int fwd_tpw_max(int nk) { return nk <= 2 ? 4 : (nk <= 6 ? 2 : 1); }

// Upper-triangular tile index of (ti, tj), row-major.
__host__ __device__ inline int64_t tile_index(int ti, int tj, int nb) {
    return (int64_t)ti * nb - (int64_t)ti * (ti - 1) / 2 + (tj - ti);
}

struct MPlan {
    int64_t Mp;            // M rounded up to the tile edge
    int nb;                // tiles per edge
    int nqb;               // 32-column blocks of [Z | 1] (Q + 1 columns)
    int DSFs;              // symmetric gradient: the same stride, >= 2 gram_t(nk) and >= Q
    int grb;               // symmetric gradient: rows per staged batch (0: not used)
    bool gsplit;           // 13 <= nb <= 16: symmetric kernel on each half, tile kernel across
    int64_t sgrows, sgchunks;  // ... the halves' row chunks
    size_t lds_sym;        // ... the first half's LDS
    int64_t dzslabs;       // dZ slabs of M x Q summed by the final reduction
                           // (odd; lanes past Q read the next row, see lds_sym_layout)
    int DSF;               // gradient: LDS row stride of the fp32 z table (odd, >= 2
                           // gram_t(nk) and >= 32 nqb, so that no read needs a bounds test)
    int nk;                // Gram: 16-slot f16 MFMA instructions (packed layout)
    int64_t T;             // upper-triangular tiles
    bool fsym;             // forward: symmetric kernel (Mp <= 512, NK <= 6)
    int tpw, ftasks;       // forward: tiles per wave task, tasks
    int64_t fgroups;       // forward: workgroups (4 tasks each) per row chunk
    int64_t frows, fchunks;
    bool gsym;             // gradient: symmetric kernel (one workgroup covers every pair)
    int jpw, njr;          // gradient: column blocks per wave task, column-block ranges
    int wpg, igroups;      // gradient: waves per workgroup (one row block each), row-block groups
    int64_t ggroups;       // gradient: workgroups per row chunk (njr * igroups)
    int64_t grows, gchunks;
    int64_t fin_blocks;    // finalize: blocks of kFinRows rows
    size_t lds_fwd, lds_grad;
    size_t off_K, off_hq, off_w2, off_hl, off_w1, off_l1, off_zc, off_bt, off_bc, off_t1, off_g2,
        off_fp, off_rs, off_dz, off_dl, off_gmax, off_gpart, off_bmax, off_smax, total;
};

// Forward LDS layout (floats):
//   za  [waves][tpw][nk][2][32][8] f16   [centred z | 1] of each wave's row blocks
//                       (tj0 .. tj0 + tpw - 1, clamped) in the packed Gram layout
//                       (fp16 parts of z and the bias multiplier 1), as A operands
//                       of the 32x32x16 f16 MFMA: wave, block, instruction, lane
//                       group, row, 8 consecutive k (only the blocks the wave reads,
//                       so that more workgroups fit per CU at large M)
//   rt  [FRB][waves][32 (1 + tpw)]   per wave, the batch's b + c of its column block
//                       ti, then the row terms b of its tpw row blocks (log2 units):
//                       only what the wave reads
//   mub [FRB][64]       centred mu of the batch (zero beyond Q)
//   kb  [FRB][64]       log2e kappa of the batch (zero beyond Q)
struct LdsF {
    int za, rt, mub, kb, total;
};

__host__ __device__ inline LdsF lds_fwd_layout(int Mp, int nk, int tpw) {
    LdsF L{};
    int o = 0;
    L.za = o; o += kWaves * tpw * nk * 2 * 32 * 8 / 2;
    L.rt = o; o += kFRB * kWaves * kTile * (1 + tpw);
    L.mub = o; o += kFRB * kRowStride;
    L.kb = o; o += kFRB * kRowStride;
    L.total = o;
    return L;
}

// Symmetric forward: tile assignment.  Wave w (column block w) takes the tiles
// j = w + k (mod nb) for k = 0 .. kx = (nb - 1) / 2 and, nb even, k = nb / 2 where
// w < nb / 2 (every unordered tile once).  Where that is more than kFSymSlots
// tiles (nb >= 10), the list is split into two ranges of k, the first
// ceil(nt / 2) tiles and the rest, computed by workgroups of their own.  A
// workgroup (four consecutive column blocks, one range) stages a window of at
// most kFSymWindow consecutive blocks (mod nb) that holds every row block its
// waves read.
constexpr int kFSymSlots = 5;
constexpr int kFSymWindow = 8;
constexpr int kFSRB = 8;    // rows per batch (prefetched a batch ahead)
__host__ __device__ inline int fsym_tiles(int nb, int w) {
    return 1 + (nb - 1) / 2 + ((nb > 1 && (nb & 1) == 0 && w < nb / 2) ? 1 : 0);
}
__host__ __device__ inline int fsym_ranges(int nb) { return fsym_tiles(nb, 0) <= kFSymSlots ? 1 : 2; }
__host__ __device__ inline int fsym_window(int nb) { return nb < kFSymWindow ? nb : kFSymWindow; }
// Even nb with one range: workgroup g holds the partner pairs (p, p + nb / 2) for
// p = 2 g, 2 g + 1 (wave slots 0, 1: p; slots 2, 3: p + nb / 2), and the two
// partners split their shared tile (k = nb / 2) by row parity, so that every wave
// takes kx + 1.5 tiles per row instead of kx + 2 for one and kx + 1 for the other.
__host__ __device__ inline bool fsym_pairs(int nb) {
    return nb > 1 && (nb & 1) == 0 && fsym_ranges(nb) == 1;
}
__host__ __device__ inline int fsym_groups(int nb) {
    return fsym_pairs(nb) ? (nb / 2 + 1) / 2 : (nb + kWaves - 1) / kWaves * fsym_ranges(nb);
}

// Symmetric forward LDS layout (floats): za [nzb][nk][2][32][8] f16 (the window's
// [centred z | 1] as Gram A operands), bb [FRB][32 nzb] (row terms b of the
// window's blocks), bcb [FRB][waves 32] (b + c of the workgroup's column blocks),
// mub, kb [FRB][64].
struct LdsFS {
    int za, bb, bcb, mub, kb, total;
};

__host__ __device__ inline LdsFS lds_fsym_layout(int nzb, int nk) {
    LdsFS L{};
    int o = 0;
    L.za = o; o += nzb * nk * 2 * 32 * 8 / 2;
    L.bb = o; o += kFSRB * nzb * kTile;
    L.bcb = o; o += kFSRB * kWaves * kTile;
    L.mub = o; o += kFSRB * kRowStride;
    L.kb = o; o += kFSRB * kRowStride;
    L.total = o > 2 * 32 * 33 ? o : 2 * 32 * 33;   // also the shared tiles' hand-over
    return L;
}

// Gradient LDS layout (floats):
//   zx  [wpg 32][DSF]   centred z (fp32) of the workgroup's row blocks (rows m of W),
//                       zero past Q up to the odd stride DSF (>= 2 gram_t(nk), >= 32 nqb)
//   zh  [jpw][2][2][2][32 nqb][8] f16    the workgroup's column blocks of [Z | 1] split
//                       into two fp16 parts, laid out as the B operands of the
//                       32x32x16 f16 MFMA (8 consecutive k per lane and instruction)
//   za  [jpw][nk][2][32][8] f16           the same rows of [centred z | 1] as Gram A
//                       operands in the packed layout (row m' per lane, 8 consecutive
//                       slots per lane group and instruction)
//   bb  [RB][32 jpw]   row terms b of the workgroup's column blocks of W (m')
//   bcb [RB][32 wpg]   b + c of its row blocks (m), one block per wave
//   mub, kb, w1b, w2b [RB][64] (zero past Q)
//   t1  [RB][32 wpg]   dL/dPsi1 * Psi1 of its row blocks
//   sc [RB] (log2 of the per-row scale of W), red [RB][wpg][5Q + 2]
// (only the blocks the workgroup reads are staged, so that the widest workgroup
// fits in LDS at Mp = 512 too)
struct LdsG {
    int zx, zb, za, bb, bcb, mub, kb, w1b, w2b, t1, sc, red, total;
};

__host__ __device__ inline LdsG lds_grad_layout(int Mp, int DSF, int Q, int nqb, int nk, int wpg) {
    const int jpw = grad_jpw(nqb);
    LdsG L{};
    int o = 0;
    L.zx = o; o += (wpg * kTile * DSF + 3) / 4 * 4;
    L.zb = o; o += jpw * 2 * 2 * 2 * 32 * nqb * 8 / 2;
    L.za = o; o += jpw * nk * 2 * 32 * 8 / 2;
    L.bb = o; o += kRB * jpw * kTile;
    L.bcb = o; o += kRB * wpg * kTile;
    L.mub = o; o += kRB * kRowStride;
    L.kb = o; o += kRB * kRowStride;
    L.w1b = o; o += kRB * kRowStride;
    L.w2b = o; o += kRB * kRowStride;
    L.t1 = o; o += kRB * wpg * kTile;
    L.sc = o; o += kRB;
    L.red = o; o += kRB * wpg * (5 * Q + 2);
    L.total = o;
    return L;
}

// Symmetric gradient LDS layout (floats), one workgroup of nb waves:
//   zx  [nb 32][DSF]   centred z (fp32) of every block, zero past Q, then 32 zeros: the
//                       stride is only >= Q, so the epilogue's lanes q >= Q read the
//                       next row's values (finite; their results are never stored)
//   zh  [nb][2][2][2][32][8] f16   [Z | 1] of every block as V-product B operands
//   za  [nb][nk][2][32][8] f16     [centred z | 1] of every block as Gram A operands
//   xw  [nb][2][32][kXS] f16       per wave, its exchanged W tile as two fp16 parts:
//                       row m of the writer's block, the 32 m' of the reader's block
//                       contiguous (kXS > 32 spreads the rows over the LDS banks)
//   bb, bcb, t1 [RB][Mp]   b, b + c and dL/dPsi1 * Psi1 of the batch, every column
//   mub, kb, w1b, w2b [RB][64] (zero past Q), sc [RB] (padded to 4), red [RB][nb][5Q + 2]
// RB, the rows per staged batch, is 8 where the tables fit and nb >= 5, 4 otherwise.
constexpr int kSymRBMax = 8;
constexpr int kXS = 36;     // halves per row of an exchanged tile
struct LdsS {
    int zx, zb, za, xw, bb, bcb, t1, mub, kb, w1b, w2b, sc, red, total;
};

__host__ __device__ inline LdsS lds_sym_layout(int nb, int DSF, int Q, int nk, int rb) {
    LdsS L{};
    int o = 0;
    const int Mp = nb * kTile;
    L.zx = o; o += (nb * kTile * DSF + 32 + 3) / 4 * 4;
    L.zb = o; o += nb * 2 * 2 * 2 * 32 * 8 / 2;
    L.za = o; o += nb * nk * 2 * 32 * 8 / 2;
    L.xw = o; o += nb * 2 * 32 * kXS / 2;
    L.bb = o; o += rb * Mp;
    L.bcb = o; o += rb * Mp;
    L.t1 = o; o += rb * Mp;
    L.mub = o; o += rb * kRowStride;
    L.kb = o; o += rb * kRowStride;
    L.w1b = o; o += rb * kRowStride;
    L.w2b = o; o += rb * kRowStride;
    L.sc = o; o += (rb + 3) / 4 * 4;
    L.red = o; o += rb * nb * (5 * Q + 2);
    L.total = o;
    return L;
}

MPlan make_mplan(const Shape &s) {
    MPlan p{};
    p.Mp = cdiv(s.M, kTile) * kTile;
    p.nb = (int)(p.Mp / kTile);
    p.nqb = s.Q + 1 <= 32 ? 1 : 2;
    p.nk = gram_nk(s.Q);
    p.DSF = std::max<int>(2 * gram_t(std::max(p.nk, 1)), 32 * p.nqb) | 1;
    p.DSFs = std::max<int>(2 * gram_t(std::max(p.nk, 1)), (int)s.Q) | 1;
    p.T = (int64_t)p.nb * (p.nb + 1) / 2;
    // forward tasks: tiles per task by a cost model in cycles: each task splits its
    // n-dependent operand once per row (about 60 vector instructions per Gram
    // instruction), each tile slot costs about 400 (MFMA, exp2, sum)
    p.tpw = 1;
    int64_t best = -1;
    for (int t = 1; t <= fwd_tpw_max(p.nk); ++t) {
        const int64_t groups = cdiv(fwd_tasks(p.nb, t), kWaves);
        const int64_t cost = groups * kWaves * (60 * p.nk + 400 * t);
        if (best < 0 || cost < best) { best = cost; p.tpw = t; }
    }
    p.ftasks = fwd_tasks(p.nb, p.tpw);
    p.fgroups = cdiv(p.ftasks, kWaves);
    p.lds_fwd = sizeof(float) * lds_fwd_layout((int)p.Mp, p.nk, p.tpw).total;
    // symmetric forward (wave w owns column block w, one operand split per row)
    p.fsym = p.nb <= 16 && p.nk > 0 && p.nk <= 6;
    if (p.fsym) {
        p.fgroups = fsym_groups(p.nb);
        p.lds_fwd = sizeof(float) * lds_fsym_layout(fsym_window(p.nb), p.nk).total;
    }
    // whole rounds of the chip's workgroup slots, so that no partly filled last
    // round idles most CUs: 6 per CU is two rounds at three workgroups per CU and
    // three at two (the register counts of the instances allow two or three)
    // (the symmetric forward's register count allows two per CU: one round)
    // (two rounds when its tiles are split into two ranges, whose workgroups differ
    // in length: 4.95 -> 4.85 ms per stress chunk; one round is faster at large)
    const int64_t fslots = p.fsym ? (fsym_ranges(p.nb) > 1 ? 2 : 1) * kCUs *
                                        std::min<int64_t>(2, std::max<int64_t>(1, kLdsBytes / p.lds_fwd))
                                  : kCUs * std::min<int64_t>(6, 2 * std::max<int64_t>(1, kLdsBytes / p.lds_fwd));
    p.fchunks = std::max<int64_t>(1, std::min(fslots / p.fgroups, cdiv(s.N, 32)));
    p.frows = cdiv(s.N, p.fchunks);
    p.fchunks = cdiv(s.N, p.frows);
    // symmetric gradient kernel (one workgroup of nb waves per row chunk) where
    // [Z | 1] is one column block, Mp <= 256 and its tables fit in LDS
    // (batches of 8 rows where those tables fit and nb >= 5, else 4: measured on
    // the gradient call at N = 100000, eight rows take 1-6% off at nb = 5 to 8
    // where they fit (Q = 20 up to nb = 7, Q <= 10 at nb = 8; at nb = 8 and Q = 20
    // they do not) and add 40% at nb = 4, at M = 128 and at 50000 x 100 x 10)
    p.grb = 0;
    for (int rb : {kSymRBMax, kSymRBMax / 2})
        if (p.grb == 0 && (rb < kSymRBMax || p.nb >= 5) && p.nqb == 1 && p.nb <= 8 && p.nk > 0 &&
            sizeof(float) * lds_sym_layout(p.nb, p.DSFs, (int)s.Q, std::max(p.nk, 1), rb).total <=
                (size_t)kLdsBytes)
            p.grb = rb;
    p.gsym = p.grb > 0;
    if (p.gsym) {
        p.jpw = p.nb;
        p.njr = 1;
        p.wpg = p.nb;
    } else {
        p.jpw = grad_jpw(p.nqb);
        p.njr = (int)cdiv(p.nb, p.jpw);
        // widest workgroup whose LDS fits
        p.wpg = std::min(p.nb, grad_waves(p.nqb));
        while (p.wpg > 1 && sizeof(float) * lds_grad_layout((int)p.Mp, p.DSF, (int)s.Q, p.nqb,
                                                            p.nk, p.wpg).total > 160 * 1024)
            p.wpg /= 2;
    }
    p.igroups = (int)cdiv(p.nb, p.wpg);
    p.ggroups = (int64_t)p.njr * p.igroups;
    // 13 <= nb <= 16 with [Z | 1] one column block: the symmetric kernel on blocks
    // 0 .. 7 and on 8 .. nb - 1 (one workgroup each per row chunk, every unordered
    // tile within a half once) and the tile kernel on the tiles between the
    // halves only (row blocks of one half against the column ranges of the
    // other: four workgroups of eight waves); 208 tiles per row at nb = 16
    // instead of 256.  Row sums: the halves in groups 0, 1, the tile kernel's in
    // 2 .. 5; dZ slabs: one per half-chunk, then two per tile-kernel chunk.
    // Measured on the gradient call at N = 100000 against the tile kernel alone:
    // 13-17% faster at nb = 13 to 16 (M = 416 .. 512, Q = 8 .. 20), 2-4% slower
    // at nb = 10 and 12, whose second half's workgroup has only 2 or 4 waves; at
    // Q = 30 the halves' tables do not fit.
    p.gsplit = false;
    if (!p.gsym && p.nqb == 1 && p.nb >= 13 && p.nb <= 16 && p.nk > 0 && p.jpw == 4 &&
        p.wpg == 8 && p.njr == (int)cdiv(p.nb, 4)) {
        int rb = 0;
        for (int r : {kSymRBMax, kSymRBMax / 2})
            if (rb == 0 && sizeof(float) * lds_sym_layout(8, p.DSFs, (int)s.Q, p.nk, r).total <=
                               (size_t)kLdsBytes)
                rb = r;
        if (rb > 0) {
            p.gsplit = true;
            p.grb = rb;
            p.lds_sym = sizeof(float) * lds_sym_layout(8, p.DSFs, (int)s.Q, p.nk, rb).total;
        }
    }
    p.lds_grad = sizeof(float) *
                 (p.gsym ? lds_sym_layout(p.nb, p.DSFs, (int)s.Q, std::max(p.nk, 1), p.grb).total
                         : lds_grad_layout((int)p.Mp, p.DSF, (int)s.Q, p.nqb, p.nk, p.wpg).total);
    // full rounds of workgroups (per CU: limited by LDS and by the waves per CU
    // the kernel's register count allows, two per SIMD; one per SIMD for the
    // wide [Z | 1] of psi2_grad_kernel): one round for the symmetric kernel and
    // for eight-wave workgroups (which fill a CU alone), else two
    const int64_t gwaves = p.gsym ? 8 : grad_waves(p.nqb);
    const int64_t gslots = kCUs * std::max<int64_t>(
                                      1, std::min<int64_t>(kLdsBytes / p.lds_grad,
                                                           gwaves / p.wpg));
    const int64_t tgroups = p.gsplit ? 4 : p.ggroups;   // tile-kernel workgroups per chunk
    p.gchunks = std::max<int64_t>(1, std::min((p.gsym || p.wpg >= 8 ? 1 : 2) * gslots / tgroups, cdiv(s.N, 16)));
    p.grows = cdiv(s.N, p.gchunks);
    p.gchunks = cdiv(s.N, p.grows);
    p.dzslabs = p.gchunks * p.njr;
    if (p.gsplit) {
        // each half: one round of one-workgroup-per-CU chunks
        p.sgchunks = std::max<int64_t>(1, std::min<int64_t>(kCUs, cdiv(s.N, 16)));
        p.sgrows = cdiv(s.N, p.sgchunks);
        p.sgchunks = cdiv(s.N, p.sgrows);
        p.ggroups = 6;
        p.dzslabs = p.sgchunks + 2 * p.gchunks;
    }
    p.fin_blocks = cdiv(s.N, kFinRows);
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
    p.off_K = take(sizeof(float) * s.N * s.Q);
    p.off_hq = take(sizeof(float) * s.N * s.Q);
    p.off_w2 = take(sizeof(float) * s.N * s.Q);
    p.off_hl = take(sizeof(float) * s.N);
    p.off_w1 = take(sizeof(float) * s.N * s.Q);
    p.off_l1 = take(sizeof(float) * s.N);
    p.off_zc = take(sizeof(float) * 4 * s.Q);  // zc, 1/s_q, s_q, R_q
    p.off_bt = take(sizeof(float) * s.N * p.Mp);
    p.off_bc = take(sizeof(float) * s.N * p.Mp);
    p.off_t1 = take(sizeof(float) * s.N * p.Mp);
    p.off_g2 = take(sizeof(float) * p.Mp * p.Mp);
    p.off_fp = take(sizeof(float) * p.fchunks * p.T * kTile * kTile);
    p.off_rs = take(sizeof(float) * p.ggroups * s.N * (5 * s.Q + 2));
    p.off_dz = take(sizeof(float) * p.dzslabs * s.M * s.Q);
    p.off_dl = take(sizeof(float) * p.fin_blocks * (s.Q + 1));
    p.off_gmax = take(sizeof(float) * 2);
    p.off_gpart = take(sizeof(float) * cdiv(s.N, 64));
    p.off_bmax = take(sizeof(float) * cdiv(p.Mp, 256) * s.N);
    p.off_smax = take(sizeof(float) * 2 * cdiv(p.Mp * p.Mp, 256));
    p.total = o;
    return p;
}

float *fat(void *ws, size_t off) { return reinterpret_cast<float *>(static_cast<char *>(ws) + off); }

// ---------------------------------------------------------------- small kernels
// Centring table of the call, [4][Q] floats: the mean inducing input zc_q, the
// per-dimension scale of the Gram operands as 1/s_q = 2^e_q and s_q = 2^-e_q
// (e_q the exponent of R_q, so that R_q s_q lies in (1/2, 1]; e_q = 0 when
// R_q = 0), and R_q = max_m |z_mq - zc_q|.  G = 256 / Q groups of Q threads take
// rows m = g, g + G, ... (coalesced); the G partial sums (then maxima) of each
// dimension are combined in group order.
__global__ __launch_bounds__(256) void mfma_centre_kernel(int M, int Q,
                                                          const float *__restrict__ Z,
                                                          float *__restrict__ zt) {
    __shared__ float part[256];
    __shared__ float s_zc[GPPS_MAX_Q];
    const int t = threadIdx.x, G = 256 / Q;
    const bool act = t < G * Q;
    const int g = t / Q, q = t - g * Q;
    if (act) {
        float s = 0.f;
#pragma unroll 8
        for (int m = g; m < M; m += G) s += Z[(int64_t)m * Q + q];
        part[t] = s;
    }
    __syncthreads();
    if (t < Q) {
        float s = 0.f;
        for (int k = 0; k < G; ++k) s += part[k * Q + t];
        s_zc[t] = s / (float)M;
    }
    __syncthreads();
    if (act) {
        const float c = s_zc[q];
        float r = 0.f;
        for (int m = g; m < M; m += G) r = fmaxf(r, fabsf(Z[(int64_t)m * Q + q] - c));
        part[t] = r;
    }
    __syncthreads();
    if (t < Q) {
        float r = 0.f;
        for (int k = 0; k < G; ++k) r = fmaxf(r, part[k * Q + t]);
        int e = 0;
        if (r > 0.f && r <= 3.0e38f) frexpf(r, &e);
        zt[t] = s_zc[t];
        zt[Q + t] = ldexpf(1.f, e);
        zt[2 * Q + t] = ldexpf(1.f, -e);
        zt[3 * Q + t] = r;
    }
}

// Per-row tables, 64 datapoints per workgroup.  For every (n, q), with
// w2 = 1/(l^2 + 2S):
//   K[n][q]  = -log2e/2 w2 / s_q
//   hq[n][q] = -log2e/4 w2,  w2[n][q],  w1[n][q] = 1/(l^2 + S)
// (one pass over the workgroup's (row, dimension) pairs, coalesced), then per row
//   hl[n]    = log2e (log sf2 - 1/4 sum_q log(1 + 2S/l^2))   (Psi2 prefactor, half of it)
//   l1[n]    = log2e (log sf2 - 1/2 sum_q log(1 + S/l^2))    (Psi1 prefactor)
// with the sums over q taken in order from LDS.  The range guard's bound for the
// row (the larger of its column bias bound |hl| + log2e/4 sum_q w2 (|mu| + R_q)
// (3 |mu| + R_q) + 128, the 128 covering the gradient's row scale, and its
// largest Gram operand bound log2e/2 w2 (|mu| + R_q) / s_q; mu centred) goes to
// gpart, as the maximum over the workgroup's rows.
constexpr int kRowsPerBlock = 64;
__global__ __launch_bounds__(256) void mfma_rows_kernel(
    int64_t N, int Q, const float *__restrict__ mu, const float *__restrict__ S,
    const float *__restrict__ zt, Hyp<float> h, float *__restrict__ Kt, float *__restrict__ hq,
    float *__restrict__ w2t, float *__restrict__ hl, float *__restrict__ w1t,
    float *__restrict__ l1, float *__restrict__ gpart) {
    __shared__ float la2[kRowsPerBlock][GPPS_MAX_Q + 1], la1[kRowsPerBlock][GPPS_MAX_Q + 1];
    __shared__ float lb[kRowsPerBlock][GPPS_MAX_Q + 1], lx[kRowsPerBlock][GPPS_MAX_Q + 1];
    __shared__ float red[kRowsPerBlock];
    const int64_t n0 = (int64_t)blockIdx.x * kRowsPerBlock;
    const int rows = (int)min<int64_t>(kRowsPerBlock, N - n0);
    for (int i = threadIdx.x; i < rows * Q; i += 256) {
        const int r = i / Q, q = i - r * Q;
        const int64_t k = n0 * Q + i;  // = (n0 + r) * Q + q
        const float sv = S[k];
        const float am = fabsf(mu[k] - zt[q]), R = zt[3 * Q + q];
        const float l2 = h.l2[q];
        const float w2 = 1.f / (l2 + 2.f * sv);
        Kt[k] = -0.5f * kLog2e * w2 * zt[Q + q];
        hq[k] = -0.25f * kLog2e * w2;
        w2t[k] = w2;
        w1t[k] = 1.f / (l2 + sv);
        la2[r][q] = log1pf(2.f * sv / l2);
        la1[r][q] = log1pf(sv / l2);
        lb[r][q] = w2 * (am + R) * (3.f * am + R);
        lx[r][q] = 0.5f * kLog2e * w2 * (am + R) * zt[Q + q];
    }
    __syncthreads();
    const int r = threadIdx.x;
    if (r < kRowsPerBlock) {
        float bound = 0.f;
        if (r < rows) {
            float a2 = 0.f, a1 = 0.f, b = 0.f, x = 0.f;
            for (int q = 0; q < Q; ++q) {
                a2 += la2[r][q];
                a1 += la1[r][q];
                b += lb[r][q];
                x = fmaxf(x, lx[r][q]);
            }
            const float hlr = kLog2e * (h.log_sf2 - 0.25f * a2);
            hl[n0 + r] = hlr;
            l1[n0 + r] = kLog2e * (h.log_sf2 - 0.5f * a1);
            // NaN anywhere makes the bound NaN, which the guard treats as out of range
            const float bb = fabsf(hlr) + 0.25f * kLog2e * b + 128.f;
            bound = (bb != bb || x != x) ? __builtin_nanf("") : fmaxf(bb, x);
        }
        red[r] = bound;
    }
    __syncthreads();
    if (r == 0) {
        float m = 0.f;
        bool nan = false;
        for (int k = 0; k < rows; ++k) {
            nan |= red[k] != red[k];
            m = fmaxf(m, red[k]);
        }
        gpart[blockIdx.x] = nan ? __builtin_nanf("") : m;
    }
}

// Range guard of the matrix-core path: route[0] = 0 when every row bound and
// every R_q is inside the fp16 limits and every R_q / l_q is at most
// kSpreadLimit (the matrix-core kernels compute the call), 1 otherwise (they
// return at once and the generic kernels compute it).  The last condition is
// one of accuracy, not range: the gradient forms dZ from V' - z_m r = sum_m'
// W (z_m' - z_m), two terms of size |z| r whose difference is of the size of the
// pair spacings that matter, about l, so fp32-class rounding of V' is amplified
// by about R / l, and by more when pairs on both sides of z_m cancel (a CPU model
// of these kernels' arithmetic: dZ error 2e-6 at R / l = 70 and 1e-3 at 440).
// One workgroup; the maximum is order-independent.
__global__ __launch_bounds__(256) void mfma_guard_kernel(int64_t nparts, int Q,
                                                         const float *__restrict__ gpart,
                                                         const float *__restrict__ zt,
                                                         Hyp<float> h, int *__restrict__ route) {
    __shared__ int bad[256];
    int b = 0;
    for (int64_t i = threadIdx.x; i < nparts; i += 256) b |= !(gpart[i] < kOperandLimit);
    for (int q = threadIdx.x; q < Q; q += 256)
        b |= !(zt[3 * Q + q] < kZLimit) | !(zt[3 * Q + q] <= kSpreadLimit * h.l[q]);
    bad[threadIdx.x] = b;
    __syncthreads();
    if (threadIdx.x == 0) {
        int v = 0;
        for (int k = 0; k < 256; ++k) v |= bad[k];
        route[0] = v;
    }
}

// Pair constant of the exponent, C_mm' = -log2e sum_q (z_mq - z_m'q)^2 / (4 l_q^2)
// (the n-independent factor 2^C of every summand; symmetric in (m, m') bit for bit).
__device__ __forceinline__ float pair_const(int m, int mp, int Q, const float *__restrict__ Z,
                                            const Hyp<float> &h) {
    float c = 0.f;
    for (int q = 0; q < Q; ++q) {
        const float d = Z[(int64_t)m * Q + q] - Z[(int64_t)mp * Q + q];
        c = fmaf(d * d, 0.25f / h.l2[q], c);
    }
    return -kLog2e * c;
}

// G2c = G2s o 2^C: the symmetric part of dL/dPsi2 times the pair factor,
// zero-padded to Mp x Mp (all zero when G2 is NULL); per workgroup, the largest
// |G2c| and |G2s| of its entries go to smax[2 block], smax[2 block + 1].
__global__ __launch_bounds__(256) void mfma_sym_kernel(int M, int Mp, int Q,
                                                       const float *__restrict__ G2,
                                                       const float *__restrict__ Z, Hyp<float> h,
                                                       const int *__restrict__ route,
                                                       float *__restrict__ G2p,
                                                       float *__restrict__ smax) {
    __shared__ float red[2][4];
    if (route[0]) return;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    float gc = 0.f, gs = 0.f;
    if (i < (int64_t)Mp * Mp) {
        const int m = (int)(i / Mp), mp = (int)(i - (int64_t)m * Mp);
        if (G2 && m < M && mp < M) {
            gs = 0.5f * (G2[(int64_t)m * M + mp] + G2[(int64_t)mp * M + m]);
            gc = gs * __builtin_amdgcn_exp2f(pair_const(m, mp, Q, Z, h));
        }
        G2p[i] = gc;
    }
    float a = fabsf(gc), b = fabsf(gs);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        a = fmaxf(a, __shfl_xor(a, off));
        b = fmaxf(b, __shfl_xor(b, off));
    }
    if ((threadIdx.x & 63) == 0) {
        red[0][threadIdx.x >> 6] = a;
        red[1][threadIdx.x >> 6] = b;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        float v = 0.f;
        for (int w = 0; w < 4; ++w) v = fmaxf(v, red[threadIdx.x][w]);
        smax[2 * blockIdx.x + threadIdx.x] = v;
    }
}

// Maximum of v over the 64 lanes of the wave, in lane 63 (other lanes hold
// partial maxima): prefix maxima inside each 16-lane row by DPP row shifts
// (a lane shifted in from outside the row keeps its own value), then the rows
// joined by the row broadcasts of lane 15 and lane 31.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_max(float x) {
    const int y = __builtin_amdgcn_update_dpp(__float_as_int(x), __float_as_int(x), CTRL, ROW_MASK,
                                              0xf, false);
    return fmaxf(x, __int_as_float(y));
}

__device__ __forceinline__ float wave_max_lane63(float v) {
    v = dpp_max<0x111, 0xf>(v);   // row_shr:1
    v = dpp_max<0x112, 0xf>(v);   // row_shr:2
    v = dpp_max<0x114, 0xf>(v);   // row_shr:4
    v = dpp_max<0x118, 0xf>(v);   // row_shr:8
    v = dpp_max<0x142, 0xa>(v);   // row_bcast:15 into rows 1 and 3
    v = dpp_max<0x143, 0xc>(v);   // row_bcast:31 into rows 2 and 3
    return v;
}

// Row terms and Psi1 for every (n, m), once per call (d = mu - z, centred):
//   bt[n][m] = hl_n + sum_q hq_nq d^2,   bc[n][m] = bt[n][m] + sum_q 2 hq_nq d mu_nq
// (2 hq = -log2e w2 / 2 is the Gram weight K of the exponent split)
//   Psi1     = exp2(l1_n - log2e/2 sum_q w1_nq d^2)
// (kPadBias in bt and kPadBiasCol in bc for m >= M).  The forward writes Psi1
// (NULL: skipped); the gradient writes t1[n][m] = dL/dPsi1[n][m] * Psi1 with
// row stride Mp (zero where G1 is NULL or m >= M) and, per row and range of 256
// inducing inputs (blockIdx.y), bmax[y][n] = max over the range's real m of
// bt[n][m] (the gradient's scale of W: max_m E'_n[m, m] = 4 max_m bt - 2 hl_n).
// A wave takes whole rows of the range: lane l holds the four inducing inputs
// m0 = y 256 + 4 l .. m0 + 3 (their z in registers up to 32 dimensions, read
// from LDS per dimension above that), so each table row is one 16-byte
// store per lane and the row maximum is a wave reduction; the workgroup's four
// waves take the batch's rows wave, wave + 4, ...  Rows are staged in LDS as one
// (mu, hq, w1, K mu) vector per dimension: one broadcast read serves four
// inducing inputs, five vector instructions each.
template <int QM, bool GRAD>
__global__ __launch_bounds__(256) void mfma_rowterm_kernel(
    int64_t N, int M, int Q, int Mp, const float *__restrict__ mu, const float *__restrict__ Z,
    const float *__restrict__ zc, const float *__restrict__ hq, const float *__restrict__ hl,
    const float *__restrict__ w1t, const float *__restrict__ l1, const float *__restrict__ G1,
    const int *__restrict__ route, float *__restrict__ bt, float *__restrict__ bc,
    float *__restrict__ psi1, float *__restrict__ t1, float *__restrict__ bmax) {
    typedef float v4f __attribute__((ext_vector_type(4)));
    // z of the range's 256 inducing inputs, dimension-major, centred and zero
    // outside the real (m, q): lane l reads its four with one 16-byte load
    constexpr bool kZReg = QM <= 32;   // z held in registers (4 QM of them)
    __shared__ v4f s_row[kRTRows][QM];
    __shared__ v4f s_zt[QM][64];
    __shared__ float s_hl[kRTRows], s_l1[kRTRows];
    if (route[0]) return;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m0 = blockIdx.y * 256 + 4 * lane;
    const int64_t n0 = (int64_t)blockIdx.x * kRTRows;
    const int cnt = (int)min<int64_t>(kRTRows, N - n0);
    // The loads below read clamped (always valid) addresses and are masked by
    // a multiplication by 0 or 1 afterwards, so that they issue back to back
    // (a select lets the compiler branch around each load and wait for it).
    // Every value read is finite here: the range guard, which sends inputs with
    // an infinite or NaN bound to the generic kernels, has passed.
    for (int i = threadIdx.x; i < kRTRows * QM; i += 256) {
        const int r = i / QM, q = i - r * QM;
        const float ok = (r < cnt && q < Q) ? 1.f : 0.f;
        const int qc = min(q, Q - 1);
        const int64_t k = (n0 + min(r, cnt - 1)) * Q + qc;
        v4f v;
        v.x = ok * (mu[k] - zc[qc]);
        v.y = ok * hq[k];
        v.z = ok * w1t[k];
        v.w = 2.f * v.y * v.x;
        s_row[r][q] = v;
    }
    for (int r = threadIdx.x; r < kRTRows; r += 256) {
        const int64_t n = n0 + min(r, cnt - 1);
        const float hv = hl[n], lv = l1[n];
        s_hl[r] = r < cnt ? hv : 0.f;
        s_l1[r] = r < cnt ? lv : 0.f;
    }
    {
        // thread t stages inducing input y 256 + t (consecutive threads write
        // consecutive words of a dimension's row)
        const int m = blockIdx.y * 256 + threadIdx.x;
        const int mc = min(m, M - 1);
        const float okm = m < M ? 1.f : 0.f;
        float *zt = reinterpret_cast<float *>(&s_zt[0][0]);
#pragma unroll 8
        for (int q = 0; q < QM; ++q) {
            const int qc = min(q, Q - 1);
            zt[q * 256 + threadIdx.x] = (q < Q ? okm : 0.f) * (Z[(int64_t)mc * Q + qc] - zc[qc]);
        }
    }
    // every lane runs the row loop (the wave reductions below read all 64 lanes);
    // lanes past Mp store nothing (Mp is a multiple of 32: the lane's four m are
    // all below it or all past it)
    const bool inb = m0 < Mp;
    const bool p1vec = (M & 3) == 0 && (reinterpret_cast<uintptr_t>(psi1) & 15) == 0;
    float realf[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) realf[u] = m0 + u < M ? 1.f : 0.f;
    // dL/dPsi1 of the wave's rows, loaded one row ahead of its use (padded
    // columns: the product of column M - 1's value and 0)
    // (one 16-byte load per lane where M is a multiple of 4 and G1 16-byte
    // aligned: the lane's four m are then all real or all padding)
    float g1c[4] = {0.f, 0.f, 0.f, 0.f};
    const bool g1vec = (M & 3) == 0 && (reinterpret_cast<uintptr_t>(G1) & 15) == 0;
    auto load_g1 = [&](int r, float *g) {
        const int64_t row = (n0 + min(r, cnt - 1)) * M;
        if (g1vec) {
            const v4f v = *reinterpret_cast<const v4f *>(G1 + row + (m0 < M ? m0 : 0));
#pragma unroll
            for (int u = 0; u < 4; ++u) g[u] = realf[u] * v[u];
        } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) g[u] = realf[u] * G1[row + min(m0 + u, M - 1)];
        }
    };
    if constexpr (GRAD)
        if (G1) load_g1(wave, g1c);
    __syncthreads();
    v4f z[kZReg ? QM : 1];
    if constexpr (kZReg) {
#pragma unroll
        for (int q = 0; q < QM; ++q) z[q] = s_zt[q][lane];
    }
#pragma unroll 1
    for (int r = wave; r < cnt; r += 4) {
        float g1n[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (GRAD)
            if (G1) load_g1(r + 4, g1n);
        float b[4], cc[4], e[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            b[u] = s_hl[r];
            cc[u] = e[u] = 0.f;
        }
#pragma unroll
        for (int q = 0; q < QM; ++q) {
            const v4f v = s_row[r][q];
            v4f zq;
            if constexpr (kZReg)
                zq = z[q];
            else
                zq = s_zt[q][lane];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const float d = v.x - zq[u];
                const float d2 = d * d;
                b[u] = fmaf(v.y, d2, b[u]);
                e[u] = fmaf(v.z, d2, e[u]);
                cc[u] = fmaf(v.w, d, cc[u]);
            }
        }
        // the sums are complete here: without this the compiler sinks the e
        // and cc chains into the store branch below and keeps every d and d^2
        // of the row live until then
#pragma unroll
        for (int u = 0; u < 4; ++u) asm volatile("" : "+v"(b[u]), "+v"(e[u]), "+v"(cc[u]));
        const int64_t n = n0 + r;
        v4f vb, vc, p1;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const bool real = realf[u] != 0.f;
            vb[u] = real ? b[u] : kPadBias;
            vc[u] = real ? b[u] + cc[u] : kPadBiasCol;
            p1[u] = __builtin_amdgcn_exp2f(fmaf(-0.5f * kLog2e, e[u], s_l1[r]));
        }
        if (inb) {
            *reinterpret_cast<v4f *>(bt + n * Mp + m0) = vb;
            *reinterpret_cast<v4f *>(bc + n * Mp + m0) = vc;
        }
        if constexpr (GRAD) {
            if (inb) {
                v4f tv;
#pragma unroll
                for (int u = 0; u < 4; ++u) tv[u] = g1c[u] * p1[u];
                *reinterpret_cast<v4f *>(t1 + n * Mp + m0) = tv;
            }
            float w = -INFINITY;
#pragma unroll
            for (int u = 0; u < 4; ++u) w = fmaxf(w, realf[u] != 0.f ? b[u] : -INFINITY);
            w = wave_max_lane63(w);
            if (lane == 63) bmax[(int64_t)blockIdx.y * N + n] = w;
        } else if (psi1) {
            // Psi1 has row stride M: one 16-byte store where M is a multiple
            // of 4 and the array 16-byte aligned (then the lane's four m are
            // all real or all padding), else one store per real m
            if (p1vec) {
                if (m0 < M) *reinterpret_cast<v4f *>(psi1 + n * M + m0) = p1;
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (m0 + u < M) psi1[n * M + m0 + u] = p1[u];
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) g1c[u] = g1n[u];
    }
}

// gmax[0] = max |G2c|, gmax[1] = max |G2s| from the sym kernel's per-workgroup
// maxima (one workgroup; max is order-independent, so the result is
// deterministic).
__global__ __launch_bounds__(1024) void mfma_absmax_kernel(int64_t nblocks,
                                                           const float *__restrict__ smax,
                                                           const int *__restrict__ route,
                                                           float *__restrict__ gmax) {
    __shared__ float part[2][16];
    if (route[0]) return;
    float a = 0.f, b = 0.f;
    for (int64_t i = threadIdx.x; i < nblocks; i += 1024) {
        a = fmaxf(a, smax[2 * i]);
        b = fmaxf(b, smax[2 * i + 1]);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        a = fmaxf(a, __shfl_xor(a, off));
        b = fmaxf(b, __shfl_xor(b, off));
    }
    if ((threadIdx.x & 63) == 0) {
        part[0][threadIdx.x >> 6] = a;
        part[1][threadIdx.x >> 6] = b;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        float r = 0.f;
        for (int w = 0; w < 16; ++w) r = fmaxf(r, part[threadIdx.x][w]);
        gmax[threadIdx.x] = r;
    }
}

// ---------------------------------------------------------------- shared helpers
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));

// fp16 residuals of exact products, by v_fma_mix: given the packed high parts
// f16(a b) of two products, v_fma_mixlo / v_fma_mixhi write f16(fma(a, b, -hi))
// into one half of a register each, reading the high part straight from the
// packed register (op_sel).  These half-register writes are inline assembly:
// written in C the compiler recomputes each fp16 high part first (two more
// vector instructions per pair).  The compiler cannot see that an asm block
// writes half registers, so it would not keep the wait states the hardware needs
// between such a write and an instruction that reads the register (an MFMA one
// instruction later may see the old value): each block ends with them.
//
// lo_pair: one pair, (a0 b0) in the low half, (a1 b1) in the high half.
__device__ __forceinline__ unsigned lo_pair(float a0, float b0, float a1, float b1, unsigned hi) {
    unsigned lo;
    asm("v_fma_mixlo_f16 %0, %1, %2, -%5 op_sel_hi:[0,0,1]\n\t"
        "s_nop 0\n\t"
        "v_fma_mixhi_f16 %0, %3, %4, -%5 op_sel:[0,0,1] op_sel_hi:[0,0,1]\n\t"
        "s_nop 1"
        : "=&v"(lo) : "v"(a0), "v"(b0), "v"(a1), "v"(b1), "v"(hi));
    return lo;
}

// lo_quad: four pairs at once, pair p from (a[2p], b[2p]) and (a[2p+1], b[2p+1])
// with high parts hi[p]; the four low-half writes come first, so that each
// register's two writes are three instructions apart, and one wait at the end.
__device__ __forceinline__ void lo_quad(const float (&a)[8], const float (&b)[8],
                                        const unsigned (&hi)[4], unsigned (&lo)[4]) {
    asm("v_fma_mixlo_f16 %0, %4, %5, -%20 op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixlo_f16 %1, %8, %9, -%21 op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixlo_f16 %2, %12, %13, -%22 op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixlo_f16 %3, %16, %17, -%23 op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixhi_f16 %0, %6, %7, -%20 op_sel:[0,0,1] op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixhi_f16 %1, %10, %11, -%21 op_sel:[0,0,1] op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixhi_f16 %2, %14, %15, -%22 op_sel:[0,0,1] op_sel_hi:[0,0,1]\n\t"
        "v_fma_mixhi_f16 %3, %18, %19, -%23 op_sel:[0,0,1] op_sel_hi:[0,0,1]\n\t"
        "s_nop 1"
        : "=&v"(lo[0]), "=&v"(lo[1]), "=&v"(lo[2]), "=&v"(lo[3])
        : "v"(a[0]), "v"(b[0]), "v"(a[1]), "v"(b[1]), "v"(a[2]), "v"(b[2]), "v"(a[3]), "v"(b[3]),
          "v"(a[4]), "v"(b[4]), "v"(a[5]), "v"(b[5]), "v"(a[6]), "v"(b[6]), "v"(a[7]), "v"(b[7]),
          "v"(hi[0]), "v"(hi[1]), "v"(hi[2]), "v"(hi[3]));
}

// Given h0 = the packed (f16(a b), 0), returns (f16(a b), f16(fma(a, b, -hi))):
// the two fp16 parts of one product in one register.
__device__ __forceinline__ unsigned hi_lo_pair(float a, float b, unsigned h0) {
    unsigned r = h0;
    asm("v_fma_mixhi_f16 %0, %1, %2, -%3 op_sel_hi:[0,0,1]\n\t"
        "s_nop 1"
        : "+v"(r) : "v"(a), "v"(b), "v"(h0));
    return r;
}

// Two fp16 parts of x (rounded to nearest): x == hi + lo up to 2^-22 |x|.
__device__ __forceinline__ void split2h(float x, _Float16 &hi, _Float16 &lo) {
    hi = (_Float16)x;
    lo = (_Float16)(x - (float)hi);
}

// Per-datapoint Gram operand of the lane's column m (B side) in the packed
// layout: x_q = (z_mq - mu_q) K_q for the lane group's dimensions
// q = g T + j (zv[j] holds z_mq; z, mu and K are zero past Q) as the fp16
// pairs listed at gram_np, and the bias (lane group 1 only) in its own pair.
// mur and kr point at the row's mu and K at dimension g T.
template <int NK>
__device__ __forceinline__ void gram_operand(const float (&zv)[gram_t(NK)],
                                             const float *__restrict__ mur,
                                             const float *__restrict__ kr, float bias, int g,
                                             v8h (&B)[NK]) {
    constexpr int NP = gram_np(NK), ODD = gram_odd(NK);
    bias = g ? bias : 0.f;  // |bias| < kOperandLimit (range guard)
    unsigned w[4 * NK];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const float d0 = zv[2 * p] - mur[2 * p], k0 = kr[2 * p];
        const float d1 = zv[2 * p + 1] - mur[2 * p + 1], k1 = kr[2 * p + 1];
        const v2h h2 = {(_Float16)(d0 * k0), (_Float16)(d1 * k1)};
        const unsigned hi = __builtin_bit_cast(unsigned, h2);
        w[p] = hi;
        w[NP + p] = lo_pair(d0, k0, d1, k1, hi);
        w[2 * NP + p] = hi;
    }
    if constexpr (ODD != 0) {
        const float d = zv[2 * NP] - mur[2 * NP], k = kr[2 * NP];
        const v2h h2 = {(_Float16)(d * k), (_Float16)0.f};
        const unsigned h0 = __builtin_bit_cast(unsigned, h2);
        w[3 * NP] = hi_lo_pair(d, k, h0);
        w[3 * NP + 1] = h0;
    }
    {
        const v2h h2 = {(_Float16)bias, (_Float16)0.f};
        const unsigned h0 = __builtin_bit_cast(unsigned, h2);
        w[3 * NP + 2 * ODD] = hi_lo_pair(bias, 1.f, h0);
    }
#pragma unroll
    for (int u = 3 * NP + 2 * ODD + 1; u < 4 * NK; ++u) w[u] = 0u;
#pragma unroll
    for (int i = 0; i < NK; ++i) {
        const unsigned q4[4] = {w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
        B[i] = __builtin_bit_cast(v8h, q4);
    }
}

// e += [z_j | 1] B over the NK packed instructions; za_j: the A operand table of
// row block j.
template <int NK>
__device__ __forceinline__ v16f gram16(v16f e, const _Float16 *__restrict__ za_j, int c, int g,
                                       const v8h (&B)[NK]) {
#pragma unroll
    for (int i = 0; i < NK; ++i) {
        const v8h A = *reinterpret_cast<const v8h *>(za_j + ((i * 2 + g) * 32 + c) * 8);
        e = __builtin_amdgcn_mfma_f32_32x32x16_f16(A, B[i], e, 0, 0, 0);
    }
    return e;
}

// Accumulator start of tile rows m' in block j: the row terms b_m' of rows
// crow(t, g) = 8 (t / 4) + 4 g + t % 4, read as four 16-byte runs.
__device__ __forceinline__ v16f row_terms(const float *__restrict__ bbr, int j, int g) {
    v16f e;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        const float4 b4 = *reinterpret_cast<const float4 *>(bbr + j * kTile + 8 * a + 4 * g);
        e[4 * a] = b4.x;
        e[4 * a + 1] = b4.y;
        e[4 * a + 2] = b4.z;
        e[4 * a + 3] = b4.w;
    }
    return e;
}

// [centred z s | 1] rows of blocks blk0 .. blk0 + nblk - 1 (clamped to the last
// block, or with wrap taken mod nb, blk0 < nb, nblk <= nb) as packed Gram A
// operand tables: [nblk][NK][2][32][8] f16 (slot
// contents listed at gram_np; zc is the centring table, [4][Q]), written by the
// nt threads t0 = 0 .. nt - 1.  Each thread issues the loads of U entries
// together from clamped (valid) addresses and masks them afterwards (the range
// guard has passed: every z is finite).
template <int NK>
__device__ void stage_za(_Float16 *za, int blk0, int nblk, int nb, int M, int Q,
                         const float *__restrict__ Z, const float *__restrict__ zc, int t0,
                         int nt, bool wrap = false) {
    constexpr int NP = gram_np(NK), ODD = gram_odd(NK), T = gram_t(NK);
    constexpr int U = 8;
    const int total = nblk * NK * 2 * 32 * 8;
    for (int base = t0; base < total; base += U * nt) {
        float v[U];
        int pt[U];
        bool isz[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int r = base + u * nt;
            const int e = r % 8; r /= 8;
            const int cc = r % 32; r /= 32;
            const int gg = r % 2; r /= 2;
            const int ins = r % NK; r /= NK;
            // blocks past the edge repeat the last one, so that every exponent stays finite
            const int blk = blk0 + r;
            const int m = (wrap ? (blk >= nb ? blk - nb : blk) : min(blk, nb - 1)) * kTile + cc;
            const int w = 4 * ins + e / 2, half = e & 1;
            int q = -1, part = 0;  // part 0: high fp16 part of z, 1: low part
            float one = 0.f;
            if (w < NP) {
                q = 2 * w + half;
            } else if (w < 2 * NP) {
                q = 2 * (w - NP) + half;
            } else if (w < 3 * NP) {
                q = 2 * (w - 2 * NP) + half;
                part = 1;
            } else if (ODD && w == 3 * NP) {
                q = 2 * NP;
            } else if (ODD && w == 3 * NP + 1) {
                if (half == 0) { q = 2 * NP; part = 1; }
            } else if (w == 3 * NP + 2 * ODD) {
                one = 1.f;         // bias multiplier
            }
            if (q >= 0) q += gg * T;
            const int qc = min(max(q, 0), Q - 1);
            // z scaled by s_q (a power of two: exact), |z s_q| <= 1
            const float zl = (Z[(int64_t)min(m, M - 1) * Q + qc] - zc[qc]) * zc[2 * Q + qc];
            isz[u] = q >= 0;
            v[u] = isz[u] ? ((m < M && q < Q) ? zl : 0.f) : one;
            pt[u] = part;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int idx = base + u * nt;
            if (idx < total) {
                if (isz[u]) {
                    _Float16 hi, lo;
                    split2h(v[u], hi, lo);
                    za[idx] = pt[u] == 0 ? hi : lo;
                } else {
                    za[idx] = (_Float16)v[u];
                }
            }
        }
    }
}

// ---------------------------------------------------------------- Psi2 forward
// Pair tiles (i, j), j >= i: rows m' in block j, columns m in block i,
//   e[m'][m] = b_m' + (b + c)_m + sum_q z_m'q (-K d_mq)      (A: [z | 1], B: [-K d | b + c])
// The row terms b_m' are the accumulator's start value; the column bias rides in
// its own pair of k slots.  Wave task: column block i (its per-datapoint operand is split
// once per row) and TPW row blocks j; Psi2 tile sums stay in registers over the
// row chunk.
template <int NK, int TPW>
__global__ __launch_bounds__(kThreads, 2) void psi2_fwd_kernel(
    int64_t N, int M, int Q, int Mp, int nb, int64_t T, int ftasks, int64_t rows_per_chunk,
    const float *__restrict__ mu, const float *__restrict__ Z, const float *__restrict__ zc,
    const float *__restrict__ Kt, const float *__restrict__ bt, const float *__restrict__ bc,
    const int *__restrict__ route, float *__restrict__ partial) {
    extern __shared__ float lds[];
    if (route[0]) return;
    const LdsF L = lds_fwd_layout(Mp, NK, TPW);
    constexpr int GT = gram_t(NK);
    _Float16 *za = reinterpret_cast<_Float16 *>(lds + L.za);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c = lane & 31, g = lane >> 5;
    const int task = blockIdx.x * kWaves + wave;
    const bool active = task < ftasks;         // wave-uniform
    int ti = 0, tj0 = 0;
    if (active) fwd_task(task, nb, TPW, ti, tj0);
    int tj[TPW];
#pragma unroll
    for (int k = 0; k < TPW; ++k) tj[k] = min(tj0 + k, nb - 1);
    const bool single = tj0 + 1 >= nb;       // wave-uniform: the task's second tile is past the edge
    v16f acc[TPW];
#pragma unroll
    for (int k = 0; k < TPW; ++k)
#pragma unroll
        for (int t = 0; t < 16; ++t) acc[k][t] = 0.f;

    // constant tables: packed [z | 1] of the wave's row blocks (LDS, written by the
    // wave itself; the batch loop's first barrier precedes every read) and the
    // centred z of the lane's column m = ti*32 + c at the lane group's dimensions
    // g GT + j (registers, zero past Q)
    _Float16 *zaw = za + wave * TPW * (NK * 2 * 32 * 8);
    if (active) stage_za<NK>(zaw, tj0, TPW, nb, M, Q, Z, zc, lane, 64);
    float zr[GT];
    {
        const int m = ti * kTile + c;
#pragma unroll
        for (int j = 0; j < GT; ++j) {
            // clamped address, masked by a multiplication: the loads issue together
            const int q = g * GT + j, qc = min(q, Q - 1);
            zr[j] = (m < M && q < Q ? 1.f : 0.f) * (Z[(int64_t)min(m, M - 1) * Q + qc] - zc[qc]);
        }
    }

    // Batches of kFRB rows: the next batch is loaded into registers while the
    // current one is computed, then written to LDS between two barriers.
    // (kFRB * 64 == blockDim: one mu / kappa value per thread.)
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    const int tid = threadIdx.x;
    // Each wave loads its own row-table slots (kFRB rows of RS entries: its column
    // block of b + c, then its TPW row blocks of b), RPL entries per lane, from
    // clamped addresses (rows >= cb are never read).
    constexpr int RS = kTile * (1 + TPW), RPL = kFRB * RS / 64;
    static_assert(kFRB * RS % 64 == 0, "whole row-table slots per lane");
    float pf_t[RPL], pf_mu, pf_k;
    auto load = [&](int64_t n0) {
        const int cb = (int)min<int64_t>(kFRB, r1 - n0);
#pragma unroll
        for (int j = 0; j < RPL; ++j) {
            const int e = lane + 64 * j, r = e / RS, x = e - r * RS;
            const int64_t row = (n0 + min(r, cb - 1)) * Mp;
            if (x < kTile) {
                pf_t[j] = bc[row + ti * kTile + x];
            } else {
                const int k = (x - kTile) / kTile;
                pf_t[j] = bt[row + min(tj0 + k, nb - 1) * kTile + (x - kTile - k * kTile)];
            }
        }
        const int r = tid / kRowStride, q = tid - r * kRowStride;
        const bool ok = r < cb && q < Q;
        pf_mu = ok ? mu[(n0 + r) * Q + q] - zc[q] : 0.f;
        pf_k = ok ? Kt[(n0 + r) * Q + q] : 0.f;
    };
    if (r0 < r1) load(r0);
    for (int64_t n0 = r0; n0 < r1; n0 += kFRB) {
        const int cb = (int)min<int64_t>(kFRB, r1 - n0);
        __syncthreads();
        if (active) {
#pragma unroll
            for (int j = 0; j < RPL; ++j) {
                const int e = lane + 64 * j, r = e / RS, x = e - r * RS;
                lds[L.rt + (r * kWaves + wave) * RS + x] = pf_t[j];
            }
        }
        lds[L.mub + tid] = pf_mu;
        lds[L.kb + tid] = pf_k;
        __syncthreads();
        if (n0 + kFRB < r1) load(n0 + kFRB);
        if (!active) continue;
        for (int r = 0; r < cb; ++r) {
            v8h B[NK];
            const float *rtw = lds + L.rt + (r * kWaves + wave) * RS;
            gram_operand<NK>(zr, lds + L.mub + r * kRowStride + g * GT, lds + L.kb + r * kRowStride + g * GT,
                             rtw[c], g, B);
            const float *bbr = rtw + kTile;   // the wave's row blocks tj0 + k at k * kTile
            if constexpr (TPW == 2) {
                // both Gram products first: the matrix cores work on tile 1 while tile
                // 0's exponentials run; the sums follow the exponentials in one run (no
                // exp2 -> add wait state per entry).  A task whose second tile lies past
                // the edge (the last task of a row block with an odd count) computes
                // its one tile only (wave-uniform branch).
                if (single) {
                    const v16f e = gram16<NK>(row_terms(bbr, 0, g), zaw, c, g, B);
                    float x[16];
#pragma unroll
                    for (int t = 0; t < 16; ++t) x[t] = __builtin_amdgcn_exp2f(e[t]);
#pragma unroll
                    for (int t = 0; t < 16; ++t) acc[0][t] += x[t];
                } else {
                    v16f e[TPW];
#pragma unroll
                    for (int k = 0; k < TPW; ++k)
                        e[k] = gram16<NK>(row_terms(bbr, k, g), zaw + k * (NK * 2 * 32 * 8),
                                          c, g, B);
#pragma unroll
                    for (int k = 0; k < TPW; ++k) {
                        float x[16];
#pragma unroll
                        for (int t = 0; t < 16; ++t) x[t] = __builtin_amdgcn_exp2f(e[k][t]);
#pragma unroll
                        for (int t = 0; t < 16; ++t) acc[k][t] += x[t];
                    }
                }
            } else {
#pragma unroll
                for (int k = 0; k < TPW; ++k) {
                    const v16f e = gram16<NK>(row_terms(bbr, k, g), zaw + k * (NK * 2 * 32 * 8),
                                              c, g, B);
#pragma unroll
                    for (int t = 0; t < 16; ++t) acc[k][t] += __builtin_amdgcn_exp2f(e[t]);
                }
            }
        }
    }
    // partial tiles: element [m' - 32 tj][m - 32 ti] (clamped duplicates are skipped)
    if (!active) return;
#pragma unroll
    for (int k = 0; k < TPW; ++k) {
        if (tj0 + k >= nb) continue;
        float *dst = partial + ((int64_t)blockIdx.y * T + tile_index(ti, tj[k], nb)) * (kTile * kTile);
#pragma unroll
        for (int r = 0; r < 16; ++r) dst[crow(r, g) * kTile + c] = acc[k][r];
    }
}

// ---------------------------------------------------------------- Psi2 forward, symmetric
// Forward for Mp <= 512 and NK <= 6: wave w owns column block w, splits its
// per-datapoint Gram operand once per row and computes the tiles (rows m' in
// block j, columns m in block w) of its range of the circulant assignment
// (fsym_tiles): every unordered tile once, 36 at nb = 8 (4 or 5 per wave), 136 at
// nb = 16 (two ranges of at most 5 per wave), with one operand split per column
// block and range instead of one per task.  A tile with j < w is the transpose of
// tile (j, w) and is stored transposed; the reduce kernel is unchanged.  A
// workgroup (four column blocks, one range: blockIdx.x = group + groups * range)
// stages the Gram A operands of its window of blocks and, per batch of kFSRB rows,
// the window's row terms b and the b + c of its own column blocks (the next batch
// prefetched into registers while this one is computed).
template <int NK>
__global__ __launch_bounds__(kThreads, 2) void psi2_fwd_sym_kernel(
    int64_t N, int M, int Q, int Mp, int nb, int64_t T, int64_t rows_per_chunk,
    const float *__restrict__ mu, const float *__restrict__ Z, const float *__restrict__ zc,
    const float *__restrict__ Kt, const float *__restrict__ bt, const float *__restrict__ bc,
    const int *__restrict__ route, float *__restrict__ partial) {
    extern __shared__ float lds[];
    if (route[0]) return;
    const int nzb = fsym_window(nb);
    const LdsFS L = lds_fsym_layout(nzb, NK);
    constexpr int GT = gram_t(NK);
    constexpr int KT = kFSymSlots;             // tile slots per wave and range
    _Float16 *za = reinterpret_cast<_Float16 *>(lds + L.za);
    const int lane = threadIdx.x & 63;
    const int wl = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const bool pairs = fsym_pairs(nb);
    const int ncg = (nb + kWaves - 1) / kWaves;
    const int cg = pairs ? (int)blockIdx.x : (int)blockIdx.x % ncg;   // column group
    const int rg = pairs ? 0 : (int)blockIdx.x / ncg;                 // range
    const int w0 = cg * kWaves;
    // column block of wave slot sl: four consecutive blocks, or the two pairs
    auto slot_block = [&](int sl) { return pairs ? 2 * cg + (sl & 1) + (sl >> 1) * (nb / 2) : w0 + sl; };
    const int w = slot_block(wl);              // column block of the wave
    const int c = lane & 31, g = lane >> 5;
    const bool active = pairs ? 2 * cg + (wl & 1) < nb / 2 : w < nb;   // wave-uniform
    // the wave's tiles in this range: k = k0 .. k0 + nt - 1 (pairs: k = 0 .. kx,
    // and the shared k = nb / 2 on the rows of the wave's parity)
    const int kx = (nb - 1) / 2;
    const int ntw = fsym_tiles(nb, min(w, nb - 1));
    const int half = fsym_ranges(nb) == 1 ? ntw : (ntw + 1) / 2;
    const int k0 = rg == 0 ? 0 : half;
    const int nt = pairs ? kx + 1 : (rg == 0 ? half : ntw - half);   // at most KT
    const int ntall = pairs ? kx + 2 : nt;     // accumulator tiles in use
    // window: blocks jbase .. jbase + nzb - 1 (mod nb); the range's smallest k is
    // that of the group's last wave (the first range starts at k = 0)
    const int kmin = rg == 0 ? 0 : (fsym_tiles(nb, min(w0 + kWaves - 1, nb - 1)) + 1) / 2;
    const int jbase = pairs ? 0 : (w0 + kmin) % nb;
    v16f acc[KT];
#pragma unroll
    for (int s = 0; s < KT; ++s)
#pragma unroll
        for (int t = 0; t < 16; ++t) acc[s][t] = 0.f;

    stage_za<NK>(za, jbase, nzb, nb, M, Q, Z, zc, threadIdx.x, blockDim.x, true);
    float zr[GT];
    {
        const int m = min(w, nb - 1) * kTile + c;
#pragma unroll
        for (int j = 0; j < GT; ++j) {
            const int q = g * GT + j, qc = min(q, Q - 1);
            zr[j] = (m < M && q < Q ? 1.f : 0.f) * (Z[(int64_t)min(m, M - 1) * Q + qc] - zc[qc]);
        }
    }

    // batch tables, prefetched one batch ahead from clamped addresses (entries of
    // rows >= cb and of blocks past the edge are never read): kFSRB rows of b for
    // the window (32 nzb each, at most PB per thread), of b + c for the
    // workgroup's column blocks (PC per thread) and of mu, K (PM each)
    constexpr int PB = kFSRB * kFSymWindow * kTile / kThreads;
    constexpr int PC = kFSRB * kWaves * kTile / kThreads;
    constexpr int PM = kFSRB * kRowStride / kThreads;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    const int tid = threadIdx.x;
    const int WB = nzb * kTile, BB = kFSRB * WB;
    float pb[PB], pc[PC], pmu[PM], pk[PM];
    auto load = [&](int64_t n0) {
        const int cb = (int)min<int64_t>(kFSRB, r1 - n0);
#pragma unroll
        for (int i = 0; i < PB; ++i) {
            const int e = min(tid + i * kThreads, BB - 1), r = e / WB, x = e - r * WB;
            const int blk = jbase + x / kTile;
            pb[i] = bt[(n0 + min(r, cb - 1)) * Mp + (blk >= nb ? blk - nb : blk) * kTile + x % kTile];
        }
#pragma unroll
        for (int i = 0; i < PC; ++i) {
            const int e = tid + i * kThreads, r = e / (kWaves * kTile), x = e - r * (kWaves * kTile);
            pc[i] = bc[(n0 + min(r, cb - 1)) * Mp + min(slot_block(x / kTile), nb - 1) * kTile + x % kTile];
        }
#pragma unroll
        for (int i = 0; i < PM; ++i) {
            const int e = tid + i * kThreads, r = e / kRowStride, q = e - r * kRowStride;
            const float ok = (r < cb && q < Q) ? 1.f : 0.f;
            const int qc = min(q, Q - 1);
            const int64_t rc = n0 + min(r, cb - 1);
            pmu[i] = ok * (mu[rc * Q + qc] - zc[qc]);
            pk[i] = ok * Kt[rc * Q + qc];
        }
    };
    if (r0 < r1) load(r0);
    for (int64_t n0 = r0; n0 < r1; n0 += kFSRB) {
        const int cb = (int)min<int64_t>(kFSRB, r1 - n0);
        __syncthreads();
#pragma unroll
        for (int i = 0; i < PB; ++i)
            if (tid + i * kThreads < BB) lds[L.bb + tid + i * kThreads] = pb[i];
#pragma unroll
        for (int i = 0; i < PC; ++i) lds[L.bcb + tid + i * kThreads] = pc[i];
#pragma unroll
        for (int i = 0; i < PM; ++i) {
            lds[L.mub + tid + i * kThreads] = pmu[i];
            lds[L.kb + tid + i * kThreads] = pk[i];
        }
        __syncthreads();
        if (n0 + kFSRB < r1) load(n0 + kFSRB);
        if (!active) continue;
        for (int r = 0; r < cb; ++r) {
            v8h B[NK];
            gram_operand<NK>(zr, lds + L.mub + r * kRowStride + g * GT,
                             lds + L.kb + r * kRowStride + g * GT,
                             lds[L.bcb + r * (kWaves * kTile) + wl * kTile + c], g, B);
            const float *bbr = lds + L.bb + r * WB;
            // tiles in slot order, each tile's Gram product issued before the
            // previous tile's exponentials, the two products alternating between
            // e0 and e1 (no register copies)
            auto gram_slot = [&](int sl) {
                int jt = (w + k0 + sl) % nb - jbase;      // the window's block index
                jt += jt < 0 ? nb : 0;
                return gram16<NK>(row_terms(bbr, jt, g), za + jt * (NK * 2 * 32 * 8), c, g, B);
            };
            auto add_exp = [&](v16f &a, const v16f &e) {
                float x[16];
#pragma unroll
                for (int t = 0; t < 16; ++t) x[t] = __builtin_amdgcn_exp2f(e[t]);
#pragma unroll
                for (int t = 0; t < 16; ++t) a[t] += x[t];
            };
            const int ntr = nt + ((pairs && (r & 1) == (wl >> 1)) ? 1 : 0);
            v16f e0 = gram_slot(0), e1;
            if (ntr > 1) e1 = gram_slot(1);
            add_exp(acc[0], e0);
            if (ntr > 2) e0 = gram_slot(2);
            if (ntr > 1) add_exp(acc[1], e1);
            if (ntr > 3) e1 = gram_slot(3);
            if (ntr > 2) add_exp(acc[2], e0);
            if (ntr > 4) e0 = gram_slot(4);
            if (ntr > 3) add_exp(acc[3], e1);
            if (ntr > 4) add_exp(acc[4], e0);
        }
    }
    if (pairs) {
        // the shared tile's rows of odd parity (slots 2, 3: rows m' in block p, columns
        // m in block p + nb / 2) join those of even parity (slots 0, 1: the transpose
        // orientation) through LDS, [2][32][33], over the batch tables
        __syncthreads();
        if (active && wl >= 2) {
#pragma unroll
            for (int s = 0; s < KT; ++s)
                if (s == kx + 1)
#pragma unroll
                    for (int t = 0; t < 16; ++t) lds[(wl - 2) * 32 * 33 + c * 33 + crow(t, g)] = acc[s][t];
        }
        __syncthreads();
        if (active && wl < 2) {
#pragma unroll
            for (int s = 0; s < KT; ++s)
                if (s == kx + 1)
#pragma unroll
                    for (int t = 0; t < 16; ++t) acc[s][t] += lds[wl * 32 * 33 + crow(t, g) * 33 + c];
        }
    }
    // partial tiles: element [m' - 32 tj][m - 32 ti] of tile (ti, tj), tj >= ti
    if (!active) return;
#pragma unroll
    for (int s = 0; s < KT; ++s) {
        if (s >= ntall || (pairs && wl >= 2 && s == kx + 1)) continue;
        const int j = (w + k0 + s) % nb;
        if (j >= w) {
            float *dst = partial + ((int64_t)blockIdx.y * T + tile_index(w, j, nb)) * (kTile * kTile);
#pragma unroll
            for (int t = 0; t < 16; ++t) dst[crow(t, g) * kTile + c] = acc[s][t];
        } else {
            // rows m' in block j, columns m in block w: the transpose of tile (j, w)
            float *dst = partial + ((int64_t)blockIdx.y * T + tile_index(j, w, nb)) * (kTile * kTile);
#pragma unroll
            for (int t = 0; t < 16; ++t) dst[c * kTile + crow(t, g)] = acc[s][t];
        }
    }
}

// Fixed-order sum over chunks, times the pair factor 2^C; both triangles written
// from the same value.  One workgroup per (upper tile, 32 consecutive partial
// entries): 8 groups of 32 threads take chunks g, g + 8, ... (one 128-byte
// segment per group), the 8 group sums are added in order.  Entry e of a tile is
// (m' mod 32) * 32 + (m mod 32).
__global__ __launch_bounds__(256) void psi2_reduce_kernel(int64_t N, int M, int Q, int nb, int64_t T,
                                                          int64_t chunks,
                                                          const float *__restrict__ partial,
                                                          const float *__restrict__ Z, Hyp<float> h,
                                                          const int *__restrict__ route,
                                                          float *__restrict__ psi0,
                                                          float *__restrict__ Psi2, int accumulate) {
    __shared__ float red[256];
    if (route[0]) return;
    const int t = threadIdx.x, o = t & 31, g = t >> 5;
    const int64_t tile = blockIdx.x >> 5;
    const int eb = blockIdx.x & 31;
    if (blockIdx.x == 0 && t == 0) psi0[0] = (accumulate ? psi0[0] : 0.f) + (float)N * h.sf2;
    const float *src = partial + tile * (kTile * kTile) + eb * kTile + o;
    const int64_t stride = T * (kTile * kTile);
    float s = 0.f;
#pragma unroll 8
    for (int64_t ch = g; ch < chunks; ch += 8) s += src[ch * stride];
    red[t] = s;
    __syncthreads();
    if (g != 0) return;
    int ti = 0;
    int64_t rem = tile;
    while (rem >= nb - ti) { rem -= nb - ti; ++ti; }
    const int tj = ti + (int)rem;
    const int m = ti * kTile + o, mp = tj * kTile + eb;
    if (m >= M || mp >= M || m > mp) return;
    float v = 0.f;
    for (int k = 0; k < 8; ++k) v += red[k * 32 + o];
    v *= __builtin_amdgcn_exp2f(pair_const(m, mp, Q, Z, h));
    v += accumulate ? Psi2[(int64_t)m * M + mp] : 0.f;
    Psi2[(int64_t)m * M + mp] = v;
    Psi2[(int64_t)mp * M + m] = v;
}

// ---------------------------------------------------------------- Psi2 gradient
// Column blocks blk0 .. blk0 + nblk - 1 of [Z | 1] as two fp16 parts (rounded to
// nearest), in the B operand order of the 32x32x16 f16 MFMA: for instruction h
// and lane group g the 8 k-values are the rows crow(8h + e, g), e = 0..7, of the
// block.
__device__ void stage_zh(_Float16 *zh, int blk0, int nblk, int M, int Q, int nqb,
                         const float *__restrict__ Z, const float *__restrict__ zc) {
    const int QV = 32 * nqb;
    const int total = nblk * 2 * 2 * 2 * QV * 8;
    for (int idx = threadIdx.x; idx < total; idx += blockDim.x) {
        int r = idx;
        const int e = r % 8; r /= 8;
        const int q = r % QV; r /= QV;
        const int gg = r % 2; r /= 2;
        const int h = r % 2; r /= 2;
        const int part = r % 2; r /= 2;
        const int k = r;
        const int m = (blk0 + k) * kTile + crow(8 * h + e, gg);
        float v = 0.f;
        if (m < M) {
            if (q < Q) v = Z[(int64_t)m * Q + q] - zc[q];
            else if (q == Q) v = 1.f;
        }
        const _Float16 hi = (_Float16)v;
        zh[idx] = part == 0 ? hi : (_Float16)(v - (float)hi);
    }
}

// Every gradient term is linear in (r_n, V_n), so the M x M tile grid may be
// split freely.  Wave task: row block i (the m index of W) and the JPW column
// blocks j (the m' index) of the workgroup's range jr.  Tile (j, i), rows m' in
// block j, columns m in block i:
//   e[m'][m] = b_m' + (b + c)_m + sum_q z_m'q (-K d_mq)   (A: [z | 1], B: [-K d | b + c])
// W = G2s o exp2(e); then V' += W [Z | 1].  Both products run on f16 MFMAs with
// both operands split into two fp16 parts (three cross products, the Gram's in
// the packed K layout), which keeps fp32 accuracy.  The column term rides in its
// own pair of k slots, the row term is the accumulator's start value.  The
// task's dL/dPsi2 tiles stay in registers for the whole kernel; the epilogue
// turns V' into the task's share of dZ (registers) and of the per-row sums,
// which the workgroup combines in LDS and writes per (group, row) for
// psi2_finalize_kernel.
template <int NK, int NQB, int JPW = grad_jpw(NQB)>
__global__ __launch_bounds__(grad_waves(NQB) * 64) void psi2_grad_kernel(
    int64_t N, int M, int Q, int Mp, int nb, int DSF, int njr, int wpg, int igroups, int cross,
    int slot0, int64_t rows_per_chunk, const float *__restrict__ mu, const float *__restrict__ Z,
    const float *__restrict__ zc, const float *__restrict__ Kt, const float *__restrict__ bt,
    const float *__restrict__ bc, const float *__restrict__ w1t, const float *__restrict__ w2t,
    const float *__restrict__ t1g, const float *__restrict__ G2p, const float *__restrict__ hl,
    const float *__restrict__ gmax, const float *__restrict__ bmax, Hyp<float> h,
    const int *__restrict__ route, float *__restrict__ rowsum, float *__restrict__ part_dz) {
    extern __shared__ float lds[];
    if (route[0]) return;
    const LdsG L = lds_grad_layout(Mp, DSF, Q, NQB, NK, wpg);
    constexpr int GT = gram_t(NK);
    _Float16 *zh = reinterpret_cast<_Float16 *>(lds + L.zb);
    _Float16 *za = reinterpret_cast<_Float16 *>(lds + L.za);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int c = lane & 31, g = lane >> 5;
    const int ones_src = 32 * g + (Q & 31);    // lane holding column Q (the row sums r)
    const int ones_qb = Q >> 5;
    const int RED = 5 * Q + 2;                 // X, Y, P, X1, P1 per dimension, then R, T1
    const int QV = 32 * NQB;
    const int group = blockIdx.x;
    // cross (tiles between the halves of the symmetric kernel's two workgroups):
    // group g takes row blocks 0 .. 7 (g < 2) or 8 .. 15 against the column
    // ranges of the other half (JPW = 4, wpg = 8); the Psi1 terms are the
    // symmetric kernel's
    const int jr = cross ? (group < 2 ? 2 + group : group - 2)
                         : group / igroups;    // range of column blocks of W (m')
    const int ib0 = cross ? (group / 2) * wpg
                          : (group % igroups) * wpg;  // first row block of the workgroup
    const int i0 = ib0 + wave;
    const bool active = i0 < nb;               // wave-uniform
    const int i = active ? i0 : 0;             // row block of W (m)
    const bool has1 = !cross && active && jr == 0;   // this task also adds the Psi1 terms of block i

    // dL/dPsi2 tiles of the task (zero for column blocks past the edge)
    int jb[JPW];
    float g2r[JPW][16];
#pragma unroll
    for (int k = 0; k < JPW; ++k) {
        const int j = jr * JPW + k;
        const bool ok = active && j < nb;
        jb[k] = ok ? j : nb - 1;
        const float *g2 = G2p + (int64_t)jb[k] * kTile * Mp + i * kTile + c;
#pragma unroll
        for (int t = 0; t < 16; ++t) g2r[k][t] = ok ? g2[(int64_t)crow(t, g) * Mp] : 0.f;
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

    // constant tables: centred z (fp32) of the row blocks, split [Z | 1] and z of
    // the column blocks
    for (int k = threadIdx.x; k < wpg * kTile * DSF; k += blockDim.x) {
        const int lr = k / DSF, q = k - lr * DSF;
        const int m = ib0 * kTile + lr;
        lds[L.zx + k] = (m < M && q < Q) ? Z[(int64_t)m * Q + q] - zc[q] : 0.f;
    }
    stage_zh(zh, jr * JPW, JPW, M, Q, NQB, Z, zc);
    // |W_n| = |G2c| 2^E'_n is bounded by max|G2c| 2^(2 hl_n) (E' <= 2 hl_n, hl_n: log2
    // of the half prefactor), and, Psi2_n being positive semidefinite (|Psi2_n[m, m']|
    // <= max_m Psi2_n[m, m]), by max|G2s| 2^(4 bmax_n - 2 hl_n); the per-row scale 2^sc
    // brings the smaller bound to 2^14, inside fp16 and well above its subnormals
    const float lgc = gmax[0] > 0.f ? __builtin_amdgcn_logf(gmax[0]) : 0.f;
    const float lgs = gmax[1] > 0.f ? __builtin_amdgcn_logf(gmax[1]) : 0.f;
    const int nbm = (Mp + 255) / 256;          // bmax parts (ranges of 256 inducing inputs)
    stage_za<NK>(za, jr * JPW, JPW, nb, M, Q, Z, zc, threadIdx.x, blockDim.x);

    // Batches of kRB rows staged in LDS between two barriers.  All loads of a
    // batch are issued before any LDS write (the first kGPF * blockDim entries of
    // each row table and one entry of each [kRB][64] table per thread; any rest
    // is loaded afterwards), so that the batch waits for one round trip to memory
    // rather than one per loop pass.  The row tables hold the workgroup's column
    // blocks jr*JPW .. (bb: JB entries per row) and row blocks ib0 .. (bcb, t1: BW
    // entries per row, which kGPF slots always cover); entries of rows >= cb or of
    // blocks past the edge are never read, and their loads use clamped addresses.
    const int JB = JPW * kTile, BW = wpg * kTile;
    const int jcol0 = jr * JPW * kTile, icol0 = ib0 * kTile;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    const int tid = threadIdx.x, nthr = blockDim.x;
    for (int64_t n0 = r0; n0 < r1; n0 += kRB) {
        const int cb = (int)min<int64_t>(kRB, r1 - n0);
        __syncthreads();
        {
            float pb[kGPF], pc[kGPF], pt[kGPF], pmu = 0.f, pk = 0.f, pw1 = 0.f, pw2 = 0.f, phl = 0.f;
#pragma unroll
            for (int j = 0; j < kGPF; ++j) {
                const int k = tid + j * nthr;
                const int rb = min(k / JB, cb - 1), rc = min(k / BW, cb - 1);
                const int64_t ob = (n0 + rb) * Mp + min(jcol0 + k % JB, Mp - 1);
                const int64_t oc = (n0 + rc) * Mp + min(icol0 + k % BW, Mp - 1);
                pb[j] = bt[ob];
                pc[j] = bc[oc];
                pt[j] = t1g[oc];
            }
            const int r = tid / kRowStride, q = tid - r * kRowStride;
            const bool okr = tid < kRB * kRowStride && r < cb && q < Q;
            if (okr) {
                pmu = mu[(n0 + r) * Q + q] - zc[q];
                pk = Kt[(n0 + r) * Q + q];
                pw1 = w1t[(n0 + r) * Q + q];
                pw2 = w2t[(n0 + r) * Q + q];
            }
            float pbm = -INFINITY;
            if (tid < cb) {
                phl = hl[n0 + tid];
                for (int y = 0; y < nbm; ++y) pbm = fmaxf(pbm, bmax[(int64_t)y * N + n0 + tid]);
            }
#pragma unroll
            for (int j = 0; j < kGPF; ++j) {
                const int k = tid + j * nthr;
                if (k < kRB * JB) lds[L.bb + k] = pb[j];
                if (k < kRB * BW) {
                    lds[L.bcb + k] = pc[j];
                    lds[L.t1 + k] = pt[j];
                }
            }
            if (tid < kRB * kRowStride) {
                lds[L.mub + tid] = pmu;
                lds[L.kb + tid] = pk;
                lds[L.w1b + tid] = pw1;
                lds[L.w2b + tid] = pw2;
            }
            if (tid < kRB) {
                const float wb = fminf(2.f * phl + lgc, 4.f * pbm - 2.f * phl + lgs);
                lds[L.sc + tid] = tid < cb ? fminf(120.f, fmaxf(-120.f, floorf(14.f - wb))) : 0.f;
            }
        }
        for (int k = tid + kGPF * nthr; k < kRB * JB; k += nthr)   // narrow workgroups only
            lds[L.bb + k] = bt[(n0 + min(k / JB, cb - 1)) * Mp + min(jcol0 + k % JB, Mp - 1)];
        for (int k = tid + nthr; k < kRB * kRowStride; k += nthr) {
            const int r = k / kRowStride, q = k - r * kRowStride;
            const bool ok = r < cb && q < Q;
            lds[L.mub + k] = ok ? mu[(n0 + r) * Q + q] - zc[q] : 0.f;
            lds[L.kb + k] = ok ? Kt[(n0 + r) * Q + q] : 0.f;
            lds[L.w1b + k] = ok ? w1t[(n0 + r) * Q + q] : 0.f;
            lds[L.w2b + k] = ok ? w2t[(n0 + r) * Q + q] : 0.f;
        }
        __syncthreads();
        for (int r = 0; r < cb; ++r) {
            float *rs = lds + L.red + (r * wpg + wave) * RED;
            if (!active) {
                for (int k = lane; k < RED; k += 64) rs[k] = 0.f;
                continue;
            }
            // Gram B operand: -K d = (z - mu) K for column block i and (b + c)_m (+ the
            // row scale) in the last k slot
            const float sc = lds[L.sc + r];
            const float bcol = lds[L.bcb + r * BW + wave * kTile + c] + sc;
            v8h GB[NK];
            {
                const float *zi = lds + L.zx + (wave * kTile + c) * DSF + g * GT;
                float zv[GT];
#pragma unroll
                for (int j = 0; j < GT; ++j) zv[j] = zi[j];
                gram_operand<NK>(zv, lds + L.mub + r * kRowStride + g * GT,
                                 lds + L.kb + r * kRowStride + g * GT, bcol, g, GB);
            }
            const float *bbr = lds + L.bb + r * JB;
            v16f V[NQB];
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
                for (int t = 0; t < 16; ++t) V[qb][t] = 0.f;
#pragma unroll
            for (int k = 0; k < JPW; ++k) {
                const int j = jb[k];
                const v16f e = gram16<NK>(row_terms(bbr, j - jr * JPW, g), za + k * (NK * 2 * 32 * 8), c, g, GB);
                // W tile (scaled by 2^sc), split into two fp16 parts; A operand of
                // instruction hh takes the lane's rows crow(8 hh + e, g), as the B
                // operand tables do
                v8h Wh[2], Wl[2];
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    unsigned wh[4], wl[4];
                    float gv[8], xv[8];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int t = 8 * hh + 2 * u;
                        xv[2 * u] = __builtin_amdgcn_exp2f(e[t]);
                        xv[2 * u + 1] = __builtin_amdgcn_exp2f(e[t + 1]);
                        gv[2 * u] = g2r[k][t];
                        gv[2 * u + 1] = g2r[k][t + 1];
                        const v2h h2 = {(_Float16)(gv[2 * u] * xv[2 * u]),
                                        (_Float16)(gv[2 * u + 1] * xv[2 * u + 1])};
                        wh[u] = __builtin_bit_cast(unsigned, h2);
                    }
                    lo_quad(gv, xv, wh, wl);
                    Wh[hh] = __builtin_bit_cast(v8h, wh);
                    Wl[hh] = __builtin_bit_cast(v8h, wl);
                }
#pragma unroll
                for (int qb = 0; qb < NQB; ++qb) {
#pragma unroll
                    for (int hh = 0; hh < 2; ++hh) {
                        const v8h Bh = *reinterpret_cast<const v8h *>(
                            zh + ((((k * 2 + 0) * 2 + hh) * 2 + g) * QV + qb * 32 + c) * 8);
                        const v8h Bl = *reinterpret_cast<const v8h *>(
                            zh + ((((k * 2 + 1) * 2 + hh) * 2 + g) * QV + qb * 32 + c) * 8);
                        V[qb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(Wh[hh], Bh, V[qb], 0, 0, 0);
                        V[qb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(Wh[hh], Bl, V[qb], 0, 0, 0);
                        V[qb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(Wl[hh], Bh, V[qb], 0, 0, 0);
                    }
                }
            }
            // V' carries the row scale 2^sc: the epilogue's coefficients and row sums
            // undo it (exact: a power of two)
            const float us = __builtin_amdgcn_exp2f(-sc);
            // epilogue for rows m = i*32 + crow(t, g); V' = W [Z | 1] -> V = r mu^T - V'
            float muq[NQB], alpha[NQB], beta[NQB], w1q[NQB];
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) {
                const int q = qb * 32 + c;
                muq[qb] = lds[L.mub + r * kRowStride + q];
                const float w2 = lds[L.w2b + r * kRowStride + q];
                w1q[qb] = lds[L.w1b + r * kRowStride + q];
                alpha[qb] = (w2 - il2[qb]) * us;
                beta[qb] = (w2 + il2[qb]) * us;
            }
            float X[NQB], Y[NQB], P[NQB], X1[NQB], P1[NQB], R = 0.f, T1 = 0.f;
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) X[qb] = Y[qb] = P[qb] = X1[qb] = P1[qb] = 0.f;
            const float *zblk = lds + L.zx + wave * kTile * DSF;
            const float *t1r = lds + L.t1 + r * BW + wave * kTile;
            // one pass over the rows of block i, with the Psi1 terms of (n, m),
            // t = dL/dPsi1 * Psi1, where this task adds them (d formed once)
            auto epilogue = [&](auto psi1) {
#pragma unroll
                for (int t = 0; t < 16; ++t) {
                    const int rr = crow(t, g);
                    const float rt = __int_as_float(__builtin_amdgcn_ds_bpermute(
                        ones_src * 4, __float_as_int(ones_qb == 0 ? V[0][t] : V[NQB - 1][t])));
                    R += rt;
                    float tv = 0.f;
                    if constexpr (decltype(psi1)::value) {
                        tv = t1r[rr];
                        T1 += tv;
                    }
#pragma unroll
                    for (int qb = 0; qb < NQB; ++qb) {
                        const int q = qb * 32 + c;
                        const float d = muq[qb] - zblk[rr * DSF + q];
                        const float v = fmaf(rt, muq[qb], -V[qb][t]);
                        const float dr = d * rt;
                        if constexpr (decltype(psi1)::value) {
                            const float td = tv * d;
                            dz[qb][t] = fmaf(alpha[qb], v, fmaf(beta[qb], dr, fmaf(td, w1q[qb], dz[qb][t])));
                            X1[qb] = fmaf(td, d, X1[qb]);
                            P1[qb] += td;
                        } else {
                            dz[qb][t] = fmaf(alpha[qb], v, fmaf(beta[qb], dr, dz[qb][t]));
                        }
                        X[qb] = fmaf(dr, d, X[qb]);
                        P[qb] += dr;
                        Y[qb] = fmaf(d, v, Y[qb]);
                    }
                }
            };
            if (has1)
                epilogue(std::true_type{});
            else
                epilogue(std::false_type{});
            // combine the two lane halves, publish this wave's sums for row r
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) {
                const float x2 = __shfl_xor(X[qb], 32), y2 = __shfl_xor(Y[qb], 32),
                            p2 = __shfl_xor(P[qb], 32), x12 = __shfl_xor(X1[qb], 32),
                            p12 = __shfl_xor(P1[qb], 32);
                const int q = qb * 32 + c;
                if (g == 0 && q < Q) {
                    rs[q] = (X[qb] + x2) * us;
                    rs[Q + q] = (Y[qb] + y2) * us;
                    rs[2 * Q + q] = (P[qb] + p2) * us;
                    rs[3 * Q + q] = X1[qb] + x12;
                    rs[4 * Q + q] = P1[qb] + p12;
                }
            }
            const float R2 = __shfl_xor(R, 32), T12 = __shfl_xor(T1, 32);
            if (lane == 0) {
                rs[5 * Q] = (R + R2) * us;
                rs[5 * Q + 1] = T1 + T12;
            }
        }
        __syncthreads();
        // per-(group, row) sums over the waves, fixed order
        for (int k = threadIdx.x; k < cb * RED; k += blockDim.x) {
            const int r = k / RED, e = k - r * RED;
            const float *rs = lds + L.red + r * wpg * RED + e;
            float v = 0.f;
            for (int w = 0; w < wpg; ++w) v += rs[w * RED];
            rowsum[((int64_t)(slot0 + group) * N + n0 + r) * RED + e] = v;
        }
    }

    // this task's share of dZ for the rows of block i: slab [chunk][jr][M][Q]
    // (cross: [chunk][group % 2][M][Q], the two halves' rows in one slab)
    if (active) {
        float *pdz = part_dz + ((int64_t)blockIdx.y * (cross ? 2 : njr) + (cross ? group % 2 : jr)) * M * Q;
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

// ---------------------------------------------------------------- Psi2 gradient, symmetric
// W_n = G2s o Psi2_n is symmetric, so one exponential per unordered pair serves
// both of its V sums when one workgroup covers every block pair of its rows
// (Alg. 1 takes each pair once): nb waves, wave w owning block w of the m index
// (its V sums, epilogue and dZ share).  Per row, wave w computes the tiles
// (rows m' in block j, columns m in block w) for j = w (diagonal), j = w + k
// (mod nb) for k = 1 .. kx = (nb - 1) / 2, and, nb even, j = w + nb / 2, which
// both partners compute, so that every wave has the same work.  A tile feeds the
// wave's own V sum as in psi2_grad_kernel (W in the MFMA output layout is the A
// operand of V' += W [Z_j | 1]); each tile of the rounds k = 1 .. kx also feeds block j's
// sum: the wave writes its two fp16 parts to LDS with m' contiguous, and wave j
// reads them back transposed (ds_read_b64_tr_b16: within each 16 lanes, element
// e of lane i comes from sub-element i % 4 of the 8 bytes lane 4 e + i / 4
// addressed), which gives the A operand of V'_j += W^T [Z_w | 1] with no VALU
// work.  At nb = 8 a row takes 40 tiles instead of 64 and 8 epilogues instead
// of 16, for 24 tile exchanges and two barriers per round.
template <int NK, int RB>
__global__ __launch_bounds__(512) void psi2_grad_sym_kernel(
    int64_t N, int M, int Q, int Mp, int nb, int blk0, int Mg, int nbg, int slot, int DSF,
    int64_t rows_per_chunk,
    const float *__restrict__ mu, const float *__restrict__ Z, const float *__restrict__ zc,
    const float *__restrict__ Kt, const float *__restrict__ bt, const float *__restrict__ bc,
    const float *__restrict__ w1t, const float *__restrict__ w2t, const float *__restrict__ t1g,
    const float *__restrict__ G2p, const float *__restrict__ hl, const float *__restrict__ gmax,
    const float *__restrict__ bmax, Hyp<float> h, const int *__restrict__ route,
    float *__restrict__ rowsum, float *__restrict__ part_dz) {
    typedef short v4s __attribute__((vector_size(8)));
    typedef __attribute__((address_space(3))) v4s lds_v4s;
    extern __shared__ float lds[];
    if (route[0]) return;
    const LdsS L = lds_sym_layout(nb, DSF, Q, NK, RB);
    constexpr int GT = gram_t(NK);
    constexpr int KT = 5;                      // tile slots: 0 diagonal, 1 .. 3 rounds, 4 shared
    _Float16 *zh = reinterpret_cast<_Float16 *>(lds + L.zb);
    _Float16 *za = reinterpret_cast<_Float16 *>(lds + L.za);
    _Float16 *xw = reinterpret_cast<_Float16 *>(lds + L.xw);
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int c = lane & 31, g = lane >> 5;
    const int ones_src = 32 * g + Q;           // lane holding column Q of V (the row sums r)
    const int RED = 5 * Q + 2;                 // X, Y, P, X1, P1 per dimension, then R, T1
    const int kx = (nb - 1) / 2;               // exchange rounds
    const bool shared_tile = nb > 1 && (nb & 1) == 0;

    // dL/dPsi2 tiles of the wave's slots, rows m' in block j, columns m in block w
    // (clamped loads, masked: unused slots hold zeros)
    float g2r[KT][16];
#pragma unroll
    for (int s = 0; s < KT; ++s) {
        const bool ok = s == 0 || (s < KT - 1 ? s <= kx : shared_tile);
        const int k = s < KT - 1 ? s : nb / 2;
        const int j = (w + (ok ? k : 0)) % nb;
        const float okf = ok ? 1.f : 0.f;
        const float *g2 = G2p + (int64_t)(blk0 + j) * kTile * Mg + (blk0 + w) * kTile + c;
#pragma unroll
        for (int t = 0; t < 16; ++t) g2r[s][t] = okf * g2[(int64_t)crow(t, g) * Mg];
    }
    v16f dz;
#pragma unroll
    for (int t = 0; t < 16; ++t) dz[t] = 0.f;
    const float il2 = c < Q ? 1.f / h.l2[c] : 0.f;

    // constant tables: centred z (fp32), [Z | 1] (V-product B operands) and
    // [centred z | 1] (Gram A operands) of every block
    for (int k = threadIdx.x; k < nb * kTile * DSF + 32; k += blockDim.x) {
        const int ml = k / DSF, q = k - ml * DSF, m = blk0 * kTile + ml;
        lds[L.zx + k] = (ml < nb * kTile && m < M && q < Q) ? Z[(int64_t)m * Q + q] - zc[q] : 0.f;
    }
    stage_zh(zh, blk0, nb, M, Q, 1, Z, zc);
    stage_za<NK>(za, blk0, nb, nbg, M, Q, Z, zc, threadIdx.x, blockDim.x);
    // per-row scale of W: as in psi2_grad_kernel
    const float lgc = gmax[0] > 0.f ? __builtin_amdgcn_logf(gmax[0]) : 0.f;
    const float lgs = gmax[1] > 0.f ? __builtin_amdgcn_logf(gmax[1]) : 0.f;

    // the exchange: this wave's slot (written) and the transpose read's lane
    // offsets (rows 4 g + (lane / 4) % 4 of each run of 8, columns 16 ((lane / 16)
    // % 2) + 4 (lane % 4) of the writer's tile)
    _Float16 *xo = xw + w * (2 * 32 * kXS);
    const int xr_row = 4 * g + ((lane >> 2) & 3);
    const int xr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

    // RB Mp = RB 32 nb row-table entries per batch over 64 nb threads: RB / 2 each
    constexpr int PT = RB / 2;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
    const int64_t r1 = min(N, r0 + rows_per_chunk);
    const int tid = threadIdx.x, nthr = blockDim.x;
    for (int64_t n0 = r0; n0 < r1; n0 += RB) {
        const int cb = (int)min<int64_t>(RB, r1 - n0);
        __syncthreads();
        // batch tables (clamped loads): with eight-row batches each thread's loads
        // are all issued before its writes; four-row batches keep the plain loop
        // (fewer registers held across it, no spill reloads in the row loop)
        if constexpr (RB == kSymRBMax) {
            float vb[PT], vc[PT], vt[PT];
#pragma unroll
            for (int i = 0; i < PT; ++i) {
                const int k = tid + i * nthr;
                const int rr = min(k / Mp, cb - 1);
                const int64_t o = (n0 + rr) * Mg + blk0 * kTile + (k - (k / Mp) * Mp);
                vb[i] = bt[o];
                vc[i] = bc[o];
                vt[i] = t1g[o];
            }
#pragma unroll
            for (int i = 0; i < PT; ++i) {
                const int k = tid + i * nthr;
                lds[L.bb + k] = vb[i];
                lds[L.bcb + k] = vc[i];
                lds[L.t1 + k] = vt[i];
            }
        } else {
            for (int k = tid; k < RB * Mp; k += nthr) {
                const int rr = min(k / Mp, cb - 1);
                const int64_t o = (n0 + rr) * Mg + blk0 * kTile + (k - (k / Mp) * Mp);
                const float vb = bt[o], vc = bc[o], vt = t1g[o];
                lds[L.bb + k] = vb;
                lds[L.bcb + k] = vc;
                lds[L.t1 + k] = vt;
            }
        }
        for (int k = tid; k < RB * kRowStride; k += nthr) {
            const int r = k / kRowStride, q = k - r * kRowStride;
            const float ok = (r < cb && q < Q) ? 1.f : 0.f;
            const int qc = min(q, Q - 1);
            const int64_t rc = n0 + min(r, cb - 1);
            const float vm = mu[rc * Q + qc] - zc[qc], vk = Kt[rc * Q + qc],
                        v1 = w1t[rc * Q + qc], v2 = w2t[rc * Q + qc];
            lds[L.mub + k] = ok * vm;
            lds[L.kb + k] = ok * vk;
            lds[L.w1b + k] = ok * v1;
            lds[L.w2b + k] = ok * v2;
        }
        if (tid < RB) {
            float sc = 0.f;
            if (tid < cb) {
                const float phl = hl[n0 + tid];
                float pbm = -INFINITY;
                for (int y = 0; y < (Mg + 255) / 256; ++y) pbm = fmaxf(pbm, bmax[(int64_t)y * N + n0 + tid]);
                const float wb = fminf(2.f * phl + lgc, 4.f * pbm - 2.f * phl + lgs);
                sc = fminf(120.f, fmaxf(-120.f, floorf(14.f - wb)));
            }
            lds[L.sc + tid] = sc;
        }
        __syncthreads();
        for (int r = 0; r < cb; ++r) {
            const float sc = lds[L.sc + r];
            const float bcol = lds[L.bcb + r * Mp + w * kTile + c] + sc;
            v8h GB[NK];
            {
                const float *zi = lds + L.zx + (w * kTile + c) * DSF + g * GT;
                float zv[GT];
#pragma unroll
                for (int j = 0; j < GT; ++j) zv[j] = zi[j];
                gram_operand<NK>(zv, lds + L.mub + r * kRowStride + g * GT,
                                 lds + L.kb + r * kRowStride + g * GT, bcol, g, GB);
            }
            const float *bbr = lds + L.bb + r * Mp;
            v16f V;
#pragma unroll
            for (int t = 0; t < 16; ++t) V[t] = 0.f;
            // W tile of slot s (block j), scaled by 2^sc, as two fp16 parts packed
            // in pairs of the rows crow(t, g), crow(t + 1, g)
            auto tile = [&](int s, int j, unsigned (&wh)[2][4], unsigned (&wl)[2][4]) {
                const v16f e = gram16<NK>(row_terms(bbr, j, g), za + j * (NK * 2 * 32 * 8), c, g, GB);
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    float gv[8], xv[8];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int t = 8 * hh + 2 * u;
                        xv[2 * u] = __builtin_amdgcn_exp2f(e[t]);
                        xv[2 * u + 1] = __builtin_amdgcn_exp2f(e[t + 1]);
                        gv[2 * u] = g2r[s][t];
                        gv[2 * u + 1] = g2r[s][t + 1];
                        const v2h h2 = {(_Float16)(gv[2 * u] * xv[2 * u]),
                                        (_Float16)(gv[2 * u + 1] * xv[2 * u + 1])};
                        wh[hh][u] = __builtin_bit_cast(unsigned, h2);
                    }
                    lo_quad(gv, xv, wh[hh], wl[hh]);
                }
            };
            // V' += W [Z_j | 1], W's two parts as A operands (three cross products)
            auto product = [&](int j, const unsigned (&wh)[2][4], const unsigned (&wl)[2][4]) {
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const v8h Ah = __builtin_bit_cast(v8h, wh[hh]);
                    const v8h Al = __builtin_bit_cast(v8h, wl[hh]);
                    const v8h Bh = *reinterpret_cast<const v8h *>(
                        zh + ((((j * 2 + 0) * 2 + hh) * 2 + g) * 32 + c) * 8);
                    const v8h Bl = *reinterpret_cast<const v8h *>(
                        zh + ((((j * 2 + 1) * 2 + hh) * 2 + g) * 32 + c) * 8);
                    V = __builtin_amdgcn_mfma_f32_32x32x16_f16(Ah, Bh, V, 0, 0, 0);
                    V = __builtin_amdgcn_mfma_f32_32x32x16_f16(Ah, Bl, V, 0, 0, 0);
                    V = __builtin_amdgcn_mfma_f32_32x32x16_f16(Al, Bh, V, 0, 0, 0);
                }
            };
            {
                unsigned wh[2][4], wl[2][4];
                tile(0, w, wh, wl);
                product(w, wh, wl);
            }
            if (shared_tile) {
                const int j = (w + nb / 2) % nb;
                unsigned wh[2][4], wl[2][4];
                tile(KT - 1, j, wh, wl);
                product(j, wh, wl);
            }
#pragma unroll
            for (int k = 1; k < KT - 1; ++k) {
                if (k > kx) break;                       // uniform over the workgroup
                const int j = (w + k) % nb, src = (w + nb - k) % nb;
                unsigned wh[2][4], wl[2][4];
                tile(k, j, wh, wl);
                __syncthreads();                         // the previous round's reads are done
#pragma unroll
                for (int T = 0; T < 4; ++T) {
                    const int hh = T >> 1, u = 2 * (T & 1);
                    const int o = c * kXS + 8 * T + 4 * g;
                    *reinterpret_cast<uint2 *>(xo + o) = make_uint2(wh[hh][u], wh[hh][u + 1]);
                    *reinterpret_cast<uint2 *>(xo + 32 * kXS + o) = make_uint2(wl[hh][u], wl[hh][u + 1]);
                }
                __syncthreads();                         // this round's tiles are written
                const _Float16 *xs = xw + src * (2 * 32 * kXS);
                unsigned rh[2][4], rl[2][4];
#pragma unroll
                for (int hh = 0; hh < 2; ++hh)
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2) {
                        const int o = (16 * hh + 8 * h2 + xr_row) * kXS + xr_col;
                        const v4s a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(xs + o));
                        const v4s b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (lds_v4s *)(xs + 32 * kXS + o));
                        const uint2 a2 = __builtin_bit_cast(uint2, a), b2 = __builtin_bit_cast(uint2, b);
                        rh[hh][2 * h2] = a2.x;
                        rh[hh][2 * h2 + 1] = a2.y;
                        rl[hh][2 * h2] = b2.x;
                        rl[hh][2 * h2 + 1] = b2.y;
                    }
                product(j, wh, wl);                      // covers the transpose reads' latency
                product(src, rh, rl);
            }
            // V' carries the row scale 2^sc: the epilogue's coefficients and row sums
            // undo it (exact: a power of two)
            const float us = __builtin_amdgcn_exp2f(-sc);
            // epilogue for rows m = w*32 + crow(t, g); V' = W [Z | 1] -> V = r mu^T - V'
            const float muq = lds[L.mub + r * kRowStride + c];
            const float w2 = lds[L.w2b + r * kRowStride + c];
            const float w1q = lds[L.w1b + r * kRowStride + c];
            const float alpha = (w2 - il2) * us, beta = (w2 + il2) * us;
            float X = 0.f, Y = 0.f, P = 0.f, X1 = 0.f, P1 = 0.f, R = 0.f, T1 = 0.f;
            const float *zblk = lds + L.zx + w * kTile * DSF;
            const float *t1r = lds + L.t1 + r * Mp + w * kTile;
            // with the Psi1 terms of (n, m), t = dL/dPsi1 * Psi1, for the same rows
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int rr = crow(t, g);
                const float rt = __int_as_float(__builtin_amdgcn_ds_bpermute(ones_src * 4, __float_as_int(V[t])));
                const float tv = t1r[rr];
                R += rt;
                T1 += tv;
                const float d = muq - zblk[rr * DSF + c];
                const float v = fmaf(rt, muq, -V[t]);
                const float dr = d * rt;
                const float td = tv * d;
                dz[t] = fmaf(alpha, v, fmaf(beta, dr, fmaf(td, w1q, dz[t])));
                X = fmaf(dr, d, X);
                P += dr;
                Y = fmaf(d, v, Y);
                X1 = fmaf(td, d, X1);
                P1 += td;
            }
            // combine the two lane halves, publish this wave's sums for row r
            float *rs = lds + L.red + (r * nb + w) * RED;
            {
                const float x2 = __shfl_xor(X, 32), y2 = __shfl_xor(Y, 32), p2 = __shfl_xor(P, 32),
                            x12 = __shfl_xor(X1, 32), p12 = __shfl_xor(P1, 32);
                if (g == 0 && c < Q) {
                    rs[c] = (X + x2) * us;
                    rs[Q + c] = (Y + y2) * us;
                    rs[2 * Q + c] = (P + p2) * us;
                    rs[3 * Q + c] = X1 + x12;
                    rs[4 * Q + c] = P1 + p12;
                }
            }
            const float R2 = __shfl_xor(R, 32), T12 = __shfl_xor(T1, 32);
            if (lane == 0) {
                rs[5 * Q] = (R + R2) * us;
                rs[5 * Q + 1] = T1 + T12;
            }
        }
        __syncthreads();
        // per-row sums over the waves, fixed order
        for (int k = threadIdx.x; k < cb * RED; k += blockDim.x) {
            const int r = k / RED, e = k - r * RED;
            const float *rs = lds + L.red + r * nb * RED + e;
            float v = 0.f;
            for (int ww = 0; ww < nb; ++ww) v += rs[ww * RED];
            rowsum[((int64_t)slot * N + n0 + r) * RED + e] = v;
        }
    }

    // this wave's share of dZ for the rows of block w: slab [chunk][M][Q]
    if (c < Q) {
        float *pdz = part_dz + (int64_t)blockIdx.y * M * Q;
#pragma unroll
        for (int t = 0; t < 16; ++t) {
            const int m = (blk0 + w) * kTile + crow(t, g);
            if (m < M) pdz[(int64_t)m * Q + c] = dz[t];
        }
    }
}

// Per row: the task groups' sums (fixed order), then with w1 = 1/(l^2 + S)
//   dmu = -2 w2 P - w1 P1
//   dS  = w2^2 (X + Y) - w2 R + 1/2 w1^2 X1 - 1/2 w1 T1
// (P1 = sum_m t d, X1 = sum_m t d^2, T1 = sum_m t, t = dL/dPsi1 * Psi1), and per
// block of kFinRows rows the partial sums of dl and dsf2.
__global__ __launch_bounds__(256) void psi2_finalize_kernel(
    int64_t N, int Q, int groups, const float *__restrict__ rowsum,
    const float *__restrict__ w2t, const float *__restrict__ S, Hyp<float> h,
    const int *__restrict__ route, float *__restrict__ dmu, float *__restrict__ dS,
    float *__restrict__ part_dl) {
    // thread (row slot r, dimension q): R = 256 / Q row slots, so that all but
    // 256 mod Q lanes work; slot r takes rows r, r + R, ... of the block
    __shared__ float red_dl[256], red_sf[256];
    if (route[0]) return;
    const int R = 256 / Q, t = threadIdx.x, r = t / Q, q = t - r * Q;
    const bool act = r < R;
    const int RED = 5 * Q + 2;
    const int64_t n0 = (int64_t)blockIdx.x * kFinRows;
    float dl = 0.f, dsf = 0.f;
    if (act) {
        const float l = h.l[q], l2 = h.l2[q];
        for (int k = r; k < kFinRows; k += R) {
            const int64_t n = n0 + k;
            if (n >= N) break;
            float X = 0.f, Y = 0.f, P = 0.f, X1 = 0.f, P1 = 0.f, Rr = 0.f, T1 = 0.f;
            for (int gi = 0; gi < groups; ++gi) {
                const float *rs = rowsum + ((int64_t)gi * N + n) * RED;
                X += rs[q];
                Y += rs[Q + q];
                P += rs[2 * Q + q];
                X1 += rs[3 * Q + q];
                P1 += rs[4 * Q + q];
                Rr += rs[5 * Q];
                T1 += rs[5 * Q + 1];
            }
            const float w2 = w2t[n * Q + q];
            const float s = S[n * Q + q];
            const float w1 = 1.f / (l2 + s);
            dmu[n * Q + q] = -2.f * w2 * P - w1 * P1;
            dS[n * Q + q] = w2 * w2 * (X + Y) - w2 * Rr + 0.5f * w1 * (w1 * X1 - T1);
            dl += (2.f * s * w2 / l) * Rr + l * w2 * w2 * (X + Y) + (X - Y) / (l2 * l) +
                  (s * w1 / l) * T1 + l * w1 * w1 * X1;
            dsf += 2.f * Rr + T1;
        }
        red_dl[t] = dl;
        if (q == 0) red_sf[r] = dsf;
    }
    __syncthreads();
    // block partials: the row slots in order
    if (t < Q) {
        float v = 0.f;
        for (int j = 0; j < R; ++j) v += red_dl[j * Q + t];
        part_dl[(int64_t)blockIdx.x * (Q + 1) + t] = v;
    } else if (t == Q) {
        float v = 0.f;
        for (int j = 0; j < R; ++j) v += red_sf[j];
        part_dl[(int64_t)blockIdx.x * (Q + 1) + Q] = v / h.sf2;
    }
}

// dZ, dl, dsf2 from the per-slab and per-block partials, fixed order.
// Workgroups below zblocks: 32 dZ entries each, 8 groups of 32 threads taking
// slabs g, g + 8, ... (two coalesced 128-byte segments per wave), the 8 group
// sums added in order.  Then one workgroup per dl_q and one for dsf2: thread t
// takes blocks t, t + 256, ..., then a fixed tree.
constexpr int kRedOut = 32, kRedGroups = 8;
__global__ __launch_bounds__(256) void grad_reduce_kernel(int64_t N, int M, int Q, int64_t zblocks,
                                                          const float *__restrict__ pdz,
                                                          int64_t dz_slabs, const float *__restrict__ pdl,
                                                          int64_t dl_parts, float dL_dpsi0,
                                                          const int *__restrict__ route,
                                                          float *__restrict__ dZ,
                                                          float *__restrict__ dsf2,
                                                          float *__restrict__ dl, int accumulate) {
    __shared__ float red[256];
    if (route[0]) return;
    const int t = threadIdx.x;
    const int64_t MQ = (int64_t)M * Q;
    if ((int64_t)blockIdx.x < zblocks) {
        const int o = t % kRedOut, g = t / kRedOut;
        const int64_t i = (int64_t)blockIdx.x * kRedOut + o;
        float s = 0.f;
        if (i < MQ) {
#pragma unroll 8
            for (int64_t sl = g; sl < dz_slabs; sl += kRedGroups) s += pdz[sl * MQ + i];
        }
        red[t] = s;
        __syncthreads();
        if (g == 0 && i < MQ) {
            float v = 0.f;
            for (int k = 0; k < kRedGroups; ++k) v += red[k * kRedOut + o];
            dZ[i] = (accumulate ? dZ[i] : 0.f) + v;
        }
        return;
    }
    const int k = (int)(blockIdx.x - zblocks);  // k < Q: dl_k; k == Q: dsf2
    float s = 0.f;
    for (int64_t b = t; b < dl_parts; b += 256) s += pdl[b * (Q + 1) + k];
    red[t] = s;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if (t < w) red[t] += red[t + w];
        __syncthreads();
    }
    if (t != 0) return;
    s = red[0];
    if (k < Q) {
        dl[k] = (accumulate ? dl[k] : 0.f) + s;
    } else {
        s += dL_dpsi0 * (float)N;
        dsf2[0] = (accumulate ? dsf2[0] : 0.f) + s;
    }
}

// ---------------------------------------------------------------- dispatch
template <int NK, int TPW>
hipError_t launch_fwd(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                      const int *route, void *ws, hipStream_t st) {
    auto k = psi2_fwd_kernel<NK, TPW>;
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_fwd);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)p.fgroups, (unsigned)p.fchunks);
    TimedScope ts(st, "mfma_psi2_fwd");
    k<<<grid, kThreads, p.lds_fwd, st>>>(s.N, (int)s.M, (int)s.Q, (int)p.Mp, p.nb, p.T,
                                         p.ftasks, p.frows, mu, Z, fat(ws, p.off_zc),
                                         fat(ws, p.off_K), fat(ws, p.off_bt), fat(ws, p.off_bc),
                                         route, fat(ws, p.off_fp));
    return hipGetLastError();
}

template <int NK, int NQB>
hipError_t launch_grad(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                       const Hyp<float> &h, const int *route, void *ws, hipStream_t st) {
    auto k = psi2_grad_kernel<NK, NQB>;
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_grad);
    if (e != hipSuccess) return e;
    // split: the tiles between the halves only, row sums from group 2 on, dZ
    // slabs after the halves'
    dim3 grid((unsigned)(p.gsplit ? 4 : p.ggroups), (unsigned)p.gchunks);
    TimedScope ts(st, "mfma_psi2_grad");
    k<<<grid, p.wpg * 64, p.lds_grad, st>>>(
        s.N, (int)s.M, (int)s.Q, (int)p.Mp, p.nb, p.DSF, p.njr, p.wpg, p.igroups, p.gsplit ? 1 : 0,
        p.gsplit ? 2 : 0, p.grows, mu, Z, fat(ws, p.off_zc), fat(ws, p.off_K), fat(ws, p.off_bt),
        fat(ws, p.off_bc), fat(ws, p.off_w1), fat(ws, p.off_w2), fat(ws, p.off_t1),
        fat(ws, p.off_g2), fat(ws, p.off_hl), fat(ws, p.off_gmax), fat(ws, p.off_bmax), h, route,
        fat(ws, p.off_rs), fat(ws, p.off_dz) + (p.gsplit ? p.sgchunks * s.M * s.Q : 0));
    return hipGetLastError();
}

template <int NK, int RB>
hipError_t launch_grad_sym(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                           const Hyp<float> &h, const int *route, void *ws, hipStream_t st) {
    auto k = psi2_grad_sym_kernel<NK, RB>;
    const size_t lds = p.gsplit ? p.lds_sym : p.lds_grad;
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
    // every block, or (split) blocks 0 .. 7 and 8 .. nb - 1 in launches of their own
    const int halves = p.gsplit ? 2 : 1;
    for (int hf = 0; hf < halves; ++hf) {
        const int blk0 = hf * 8, nbl = p.gsplit ? (hf == 0 ? 8 : p.nb - 8) : p.nb;
        const size_t ldsh = sizeof(float) * lds_sym_layout(nbl, p.DSFs, (int)s.Q, NK, RB).total;
        dim3 grid(1u, (unsigned)(p.gsplit ? p.sgchunks : p.gchunks));
        TimedScope ts(st, "mfma_psi2_grad");
        k<<<grid, nbl * 64, ldsh, st>>>(
            s.N, (int)s.M, (int)s.Q, nbl * kTile, nbl, blk0, (int)p.Mp, p.nb, hf, p.DSFs,
            p.gsplit ? p.sgrows : p.grows, mu, Z, fat(ws, p.off_zc), fat(ws, p.off_K),
            fat(ws, p.off_bt), fat(ws, p.off_bc), fat(ws, p.off_w1), fat(ws, p.off_w2),
            fat(ws, p.off_t1), fat(ws, p.off_g2), fat(ws, p.off_hl), fat(ws, p.off_gmax),
            fat(ws, p.off_bmax), h, route, fat(ws, p.off_rs), fat(ws, p.off_dz));
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int NK>
hipError_t launch_fwd_sym(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                          const int *route, void *ws, hipStream_t st) {
    auto k = psi2_fwd_sym_kernel<NK>;
    hipError_t e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)p.lds_fwd);
    if (e != hipSuccess) return e;
    dim3 grid((unsigned)p.fgroups, (unsigned)p.fchunks);
    TimedScope ts(st, "mfma_psi2_fwd");
    k<<<grid, kThreads, p.lds_fwd, st>>>(s.N, (int)s.M, (int)s.Q, (int)p.Mp, p.nb, p.T, p.frows,
                                         mu, Z, fat(ws, p.off_zc), fat(ws, p.off_K),
                                         fat(ws, p.off_bt), fat(ws, p.off_bc), route,
                                         fat(ws, p.off_fp));
    return hipGetLastError();
}

hipError_t dispatch_fwd(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                        const int *route, void *ws, hipStream_t st) {
    if (p.fsym) {
#define GPPS_FS(I) \
    if (p.nk == I) return launch_fwd_sym<I>(p, s, mu, Z, route, ws, st);
        GPPS_FS(1) GPPS_FS(2) GPPS_FS(3) GPPS_FS(4) GPPS_FS(6)
#undef GPPS_FS
        return hipErrorInvalidValue;
    }
#define GPPS_F(I, T) \
    if (p.nk == I && p.tpw == T) return launch_fwd<I, T>(p, s, mu, Z, route, ws, st);
    GPPS_F(1, 1) GPPS_F(1, 2) GPPS_F(1, 3) GPPS_F(1, 4)
    GPPS_F(2, 1) GPPS_F(2, 2) GPPS_F(2, 3) GPPS_F(2, 4)
    GPPS_F(3, 1) GPPS_F(3, 2)
    GPPS_F(4, 1) GPPS_F(4, 2)
    GPPS_F(6, 1) GPPS_F(6, 2) GPPS_F(8, 1) GPPS_F(10, 1) GPPS_F(12, 1)
#undef GPPS_F
    return hipErrorInvalidValue;
}

hipError_t dispatch_grad(const MPlan &p, const Shape &s, const float *mu, const float *Z,
                         const Hyp<float> &h, const int *route, void *ws, hipStream_t st) {
    if (p.gsym || p.gsplit) {
        hipError_t e = hipErrorInvalidValue;
#define GPPS_GS(I)                                                                 \
    if (p.nk == I && p.grb == kSymRBMax) e = launch_grad_sym<I, kSymRBMax>(p, s, mu, Z, h, route, ws, st); \
    if (p.nk == I && p.grb == kSymRBMax / 2) e = launch_grad_sym<I, kSymRBMax / 2>(p, s, mu, Z, h, route, ws, st);
        GPPS_GS(1) GPPS_GS(2) GPPS_GS(3) GPPS_GS(4) GPPS_GS(6) GPPS_GS(8)
#undef GPPS_GS
        if (p.gsym || e != hipSuccess) return e;
        // split: then the tiles between the halves
    }
#define GPPS_G(I, Q) \
    if (p.nk == I && p.nqb == Q) return launch_grad<I, Q>(p, s, mu, Z, h, route, ws, st);
    GPPS_G(1, 1) GPPS_G(2, 1) GPPS_G(3, 1) GPPS_G(4, 1) GPPS_G(6, 1) GPPS_G(8, 1)
    GPPS_G(8, 2) GPPS_G(10, 2) GPPS_G(12, 2)
#undef GPPS_G
    return hipErrorInvalidValue;
}

// The centring table, the per-row tables, the range guard (route word), and
// the row terms plus Psi1 (forward, psi1 != NULL) or dL/dPsi1 * Psi1 (grad).
void prepare(const MPlan &p, const Shape &s, const float *mu, const float *S, const float *Z,
             const Hyp<float> &h, const float *G1, float *psi1, bool grad, int *route, void *ws,
             hipStream_t st) {
    {
        TimedScope ts(st, "mfma_centre");
        mfma_centre_kernel<<<1, 256, 0, st>>>((int)s.M, (int)s.Q, Z, fat(ws, p.off_zc));
    }
    const int64_t rblocks = cdiv(s.N, kRowsPerBlock);
    {
        TimedScope ts(st, "mfma_rows");
        mfma_rows_kernel<<<(unsigned)rblocks, 256, 0, st>>>(
            s.N, (int)s.Q, mu, S, fat(ws, p.off_zc), h, fat(ws, p.off_K), fat(ws, p.off_hq),
            fat(ws, p.off_w2), fat(ws, p.off_hl), fat(ws, p.off_w1), fat(ws, p.off_l1),
            fat(ws, p.off_gpart));
    }
    {
        TimedScope ts(st, "mfma_guard");
        mfma_guard_kernel<<<1, 256, 0, st>>>(rblocks, (int)s.Q, fat(ws, p.off_gpart),
                                             fat(ws, p.off_zc), h, route);
    }
    dim3 grid((unsigned)cdiv(s.N, kRTRows), (unsigned)cdiv(p.Mp, 256));
    float *t1 = grad ? fat(ws, p.off_t1) : nullptr;
    TimedScope ts(st, "mfma_rowterm");
#define GPPS_RT(QM)                                                                            \
    do {                                                                                       \
        if (grad)                                                                              \
            mfma_rowterm_kernel<QM, true><<<grid, 256, 0, st>>>(                               \
                s.N, (int)s.M, (int)s.Q, (int)p.Mp, mu, Z, fat(ws, p.off_zc), fat(ws, p.off_hq), \
                fat(ws, p.off_hl), fat(ws, p.off_w1), fat(ws, p.off_l1), G1, route,            \
                fat(ws, p.off_bt), fat(ws, p.off_bc), nullptr, t1, fat(ws, p.off_bmax));       \
        else                                                                                   \
            mfma_rowterm_kernel<QM, false><<<grid, 256, 0, st>>>(                              \
                s.N, (int)s.M, (int)s.Q, (int)p.Mp, mu, Z, fat(ws, p.off_zc), fat(ws, p.off_hq), \
                fat(ws, p.off_hl), fat(ws, p.off_w1), fat(ws, p.off_l1), G1, route,            \
                fat(ws, p.off_bt), fat(ws, p.off_bc), psi1, nullptr, nullptr);                 \
    } while (0)
    if (s.Q <= 8) GPPS_RT(8);
    else if (s.Q <= 12) GPPS_RT(12);
    else if (s.Q <= 16) GPPS_RT(16);
    else if (s.Q <= 20) GPPS_RT(20);
    else if (s.Q <= 24) GPPS_RT(24);
    else if (s.Q <= 32) GPPS_RT(32);
    else if (s.Q <= 48) GPPS_RT(48);
    else GPPS_RT(64);
#undef GPPS_RT
}

}  // namespace

bool mfma_supports(const Shape &s) {
    const int64_t Mp = cdiv(s.M, kTile) * kTile;
    if (!((Mp <= 512 && s.Q <= 31) || (Mp <= 256 && s.Q <= GPPS_MAX_Q_MFMA))) return false;
    const MPlan p = make_mplan(s);
    return p.nk > 0 && p.lds_grad <= 160 * 1024 && p.lds_fwd <= 160 * 1024;
}

size_t mfma_workspace_bytes(const Shape &s) { return make_mplan(s).total; }

hipError_t mfma_psi_stats(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float *psi0, float *Psi1, float *Psi2,
                          int accumulate, int *route, void *ws, hipStream_t st) {
    const MPlan p = make_mplan(s);
    prepare(p, s, mu, S, Z, h, nullptr, Psi1, false, route, ws, st);
    hipError_t e = dispatch_fwd(p, s, mu, Z, route, ws, st);
    if (e != hipSuccess) return e;
    TimedScope ts(st, "mfma_psi2_reduce");
    psi2_reduce_kernel<<<(unsigned)(p.T * 32), 256, 0, st>>>(
        s.N, (int)s.M, (int)s.Q, p.nb, p.T, p.fchunks, fat(ws, p.off_fp), Z, h, route, psi0, Psi2,
        accumulate);
    return hipGetLastError();
}

hipError_t mfma_psi_grads(const Shape &s, const float *mu, const float *S, const float *Z,
                          const Hyp<float> &h, float dL_dpsi0, const float *G1,
                          const float *G2, float *dmu, float *dS, float *dZ, float *dsf2,
                          float *dl, int accumulate, int *route, void *ws, hipStream_t st) {
    const MPlan p = make_mplan(s);
    prepare(p, s, mu, S, Z, h, G1, nullptr, true, route, ws, st);
    {
        // NULL dL/dPsi2 means zero: the kernel then adds only the Psi1 terms
        TimedScope ts(st, "mfma_sym");
        mfma_sym_kernel<<<(unsigned)cdiv(p.Mp * p.Mp, 256), 256, 0, st>>>(
            (int)s.M, (int)p.Mp, (int)s.Q, G2, Z, h, route, fat(ws, p.off_g2), fat(ws, p.off_smax));
    }
    {
        TimedScope ts(st, "mfma_absmax");
        mfma_absmax_kernel<<<1, 1024, 0, st>>>(cdiv(p.Mp * p.Mp, 256), fat(ws, p.off_smax), route,
                                               fat(ws, p.off_gmax));
    }
    hipError_t e = dispatch_grad(p, s, mu, Z, h, route, ws, st);
    if (e != hipSuccess) return e;
    {
        TimedScope ts(st, "mfma_psi2_finalize");
        psi2_finalize_kernel<<<(unsigned)p.fin_blocks, 256, 0, st>>>(
            s.N, (int)s.Q, (int)p.ggroups, fat(ws, p.off_rs), fat(ws, p.off_w2), S, h, route, dmu,
            dS, fat(ws, p.off_dl));
    }
    const int64_t zblocks = cdiv(s.M * s.Q, kRedOut);
    TimedScope ts(st, "mfma_grad_reduce");
    grad_reduce_kernel<<<(unsigned)(zblocks + s.Q + 1), 256, 0, st>>>(
        s.N, (int)s.M, (int)s.Q, zblocks, fat(ws, p.off_dz), p.dzslabs, fat(ws, p.off_dl),
        p.fin_blocks, dL_dpsi0, route, dZ, dsf2, dl, accumulate);
    return hipGetLastError();
}

}  // namespace gpps
