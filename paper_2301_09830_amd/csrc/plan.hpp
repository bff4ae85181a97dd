// Per-matrix launch plan and device descriptor of liboptcc.
//
// The host computes, for every matrix of a call, the tiling of each kernel
// and the byte offsets of that matrix's scratch regions inside the caller's
// workspace.  Kernels receive the descriptor either by value (one matrix) or
// as a table in the workspace (batched calls), and map their flattened block
// index to (matrix, tile) with the per-kernel block offsets stored here.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <algorithm>

namespace occ {

constexpr int kMaxRank = 128;
constexpr int kWave = 64;
constexpr int kBlock = 256;  // threads per block of every streaming kernel

// Kernel kinds that have a per-matrix tiled grid.
enum Kind : int {
  K_QPAD = 0,    // copy the warm-start Q into the padded layout
  K_PASS_P,      // P partials = A Q over column splits
  K_PGRAM,       // reduce the splits -> P; Gram partials (fp64)
  K_GSUM,        // sum Gram partials -> G
  K_GRAM2,       // CholeskyQR2 second Gram: (P T1)^T (P T1) partials
  K_APPLY,       // P_hat = P T (padded copy and caller's P)
  K_PASS_Q,      // Q partials = A^T P_hat over row splits
  K_QRED,        // reduce Q partials -> Q (caller and padded copy)
  K_MHAT,        // M_hat = P_hat Q^T, err = A - M_hat
  K_NUM
};

struct Desc {
  // caller buffers
  const void* M;
  const float* err_in;   // may be null (zero error)
  float* err_out;        // may be null (compress-only: not written)
  float* P;              // m x r
  float* Q;              // n x r
  float* Mhat;           // may be null
  // workspace regions (device addresses)
  float* qpad;           // n_pad x rp, zero padded
  float* phat;           // m x rp
  float* praw;           // m x rp
  float* ppart;          // sp x m x rp
  float* qpart;          // sq x n x rp (fp64 on the small-rank path)
  double* gpart;         // ng x rp x rp
  double* gsum;          // rp x rp
  double* t1;            // rp x rp
  double* tm;            // rp x rp (large-rank path: T2 of the second pass)
  uint32_t* info;        // [0] = second CholeskyQR pass needed
  float* phat_t;         // large-rank path: P_hat transposed, rp x m_pad
  uint16_t* qbf;         // large-rank path, bf16 M: Q as bf16 hi/lo parts, [2][rp][n_pad],
                         // rank k in row (k % (rp/32)) * 32 + k / (rp/32)
  const int32_t* rmap;   // row-sparse step: row i of the compressed matrix is row rmap[i]
                         // of M, err and M_hat (validated copy in the workspace); else null
  float* err_fin;        // row-sparse step, padded rank > 16: the caller's error buffer, which
                         // the reconstruction pass writes (rows through rmap); err_out then
                         // holds the stored A compactly (n_rows x lde_out) in the workspace
  int32_t lde_fin;
  // shapes
  int32_t m, n, r;
  int32_t ldm, lde_in, lde_out, ldh;
  int32_t n_pad;
  int32_t sp, p_cols;    // left product: column splits and columns per split (multiple of 32)
  int32_t ng;            // Gram partials (one per block of the Gram kernel)
  int32_t grows;         // large-rank path: rows per block of the Gram kernel (multiple of 32)
  int32_t sq, q_rows;    // right product: row splits and rows per split
  int32_t blk[K_NUM];    // first block of this matrix in each kernel's grid
  int32_t fused;         // 1: small-rank path (rank padded to <= 16)
  int32_t m_pad;         // large-rank path: rows of phat_t (multiple of 32)
  int32_t mr;            // rows per block of the reconstruction pass
  int32_t vec;           // large-rank path: 16-byte vector loads allowed
  int32_t qr_cols;       // large-rank path: columns per block of the Q reduction (8 or 32)
};

// Tiling of one matrix (host side).
struct Tiling {
  int sp, p_cols, ng, grows, sq, q_rows, n_pad, m_pad, mr, qr_cols;
  int64_t blocks[K_NUM];
};

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return cdiv(a, b) * b; }
inline int64_t clamp64(int64_t v, int64_t lo, int64_t hi) { return v < lo ? lo : (v > hi ? hi : v); }

inline int padded_rank(int r) {
  int p = 4;
  while (p < r) p *= 2;
  return p;
}

// Small-rank path (padded rank <= 16): tile constants shared with
// kernels_small.hpp and kernels_mfma16.hpp.
constexpr int kFusedMaxRank = 16;
constexpr int F_PROWS = 32;       // left product: rows per row block
constexpr int F_PM_MAXBLOCKS = 512;  // left product: blocks (each one Gram partial), at most
constexpr int F_PM_WAVES = 4;        // left product: waves per block
// left product: waves sharing one row block's 32-column K-steps, all of
// them unless the matrix has fewer K-steps than waves (n <= 96); the other
// waves of the block take the next row blocks
__host__ __device__ constexpr int pm_waves_per_rb(int n) { return n > 96 ? 4 : (n > 32 ? 2 : 1); }
constexpr int F_QCOLS = 128;      // right product: columns per block
constexpr int F_MHCOLS = 128;     // reconstruction: columns per block
constexpr int F_MHGROUP = 64;     // reconstruction: rows per block step (4 waves x 16 rows)
constexpr int F_MHBLOCKS = 1024;  // reconstruction: target number of blocks
constexpr int F_QBLOCKS = 512;    // right product: resident blocks (2 per CU on 256 CUs)
// finishing kernel: threads that share the sum of one element's sq row-split
// partials (each thread at most 32 of them)
__host__ __device__ constexpr int qfin_slices(int sq) {
  return sq > 256 ? 16 : sq > 128 ? 8 : sq > 64 ? 4 : sq > 32 ? 2 : 1;
}

// Large-rank path (padded rank 32, 64, 128): tile constants shared with
// kernels_large.hpp.
constexpr int L_PROWS = 128;      // left product: rows per block (4 waves x 32) ...
// ... and 256 (8 waves) for bf16 M at padded rank 128, where a 4-wave block
// runs one wave per SIMD (its LDS tiles and Q stages) and reads a Q tile as
// large as its A tile
__host__ __device__ constexpr int lp_block_rows(int rp, bool x3) { return rp >= 128 && x3 ? 256 : L_PROWS; }
constexpr int L_KC = 32;          // left product: columns per K-step
constexpr int L_GROWS = 256;      // Gram partials: rows per block
constexpr int L_AROWS = 128;      // P_hat = P T: rows per block
constexpr int L_QG = 8;           // right product: rows per LDS stage
constexpr int64_t L_SPLIT_BLOCKS = 1024;  // split products: blocks over the whole batch
constexpr int64_t L_MIN_COLS = 1024;      // left product: columns per split, at least
constexpr int64_t L_MIN_ROWS = 1024;      // right product: rows per split, at least
constexpr int64_t L_MIN_NARROW = 256;     // the same for matrices that cannot fill a round
// right product: columns per lane and per block
__host__ __device__ constexpr int lq_cpl(int rp) { return rp >= 128 ? 1 : 128 / rp; }
// waves per block of the split bf16 right product (k_lqx): 8 at padded rank
// 128, so that a block's P_hat^T tile of each 16-row group (as many bytes
// as 128 columns of A) serves 256 columns
__host__ __device__ constexpr int lqx_waves(int rp) { return rp >= 128 ? 8 : 4; }
__host__ __device__ constexpr int lq_block_cols(int rp, bool x3 = false) {
  return (x3 ? 32 * lqx_waves(rp) : 128) * lq_cpl(rp);
}
// reconstruction: 32-column MFMA tiles per wave and columns per block
__host__ __device__ constexpr int lm_tiles(int rp) { return rp >= 64 ? 1 : 2; }
__host__ __device__ constexpr int lm_block_cols(int rp) { return 128 * lm_tiles(rp); }
// reconstruction of fp32 M (k_ml): outputs through an LDS tile and stored by
// rows with 16-byte accesses at padded rank 64 (51200 x 3072: 393 -> 369 us);
// at rank 32 (two 32-column tiles per wave) stored straight from the MFMA
// layout, which measured faster there (2.50 vs 2.81 ms on 36 stage matrices)
__host__ __device__ constexpr bool lm_lds_epilogue(int rp) { return rp == 64; }

// Blocks of each large-rank streaming kernel that are resident on the
// device at once (compute units x blocks per compute unit).  Grids are
// sized in whole multiples of these: blocks of a pass do equal work, so a
// grid of 1.33 rounds takes as long as 2.
struct Slots {
  int64_t p = 1024, q = 1024, m = 1024;   // left product, right product, reconstruction
};

// The multiple of `slots` nearest to `want`, at least one round.
inline int64_t whole_rounds(int64_t want, int64_t slots) {
  const int64_t k = std::max<int64_t>(1, (want + slots / 2) / slots);
  return k * slots;
}

// share: this matrix's fraction of the elements of the whole call (the
// large-rank grids are sized for the batch).
inline Tiling make_tiling(int64_t m, int64_t n, int rp, double share = 1.0,
                          const Slots& sl = Slots{}, bool x3 = false) {
  Tiling t{};
  t.qr_cols = 32;
  t.n_pad = (int)round_up(n, 32);
  t.m_pad = (int)round_up(m, 32);
  if (rp <= kFusedMaxRank) {
    // left product: whole rows per block, no column splits
    const int64_t p_blocks = cdiv(m, F_PROWS);
    t.sp = 1;
    t.p_cols = (int)round_up(n, 32);
    const int64_t p_groups = cdiv(p_blocks, F_PM_WAVES / pm_waves_per_rb((int)n));
    t.ng = (int)std::min<int64_t>(p_groups, F_PM_MAXBLOCKS);
    // right product: at most F_QBLOCKS - 1 blocks, so that they and the
    // block forming T run in one round
    const int64_t col_tiles = cdiv(n, F_QCOLS);
    const int64_t sq = clamp64((F_QBLOCKS - 1) / col_tiles, 1, cdiv(m, 32));
    t.q_rows = (int)round_up(cdiv(m, sq), 4);
    t.sq = (int)cdiv(m, t.q_rows);
    // reconstruction: 128-column tiles x row blocks (multiple of 64 rows),
    // about F_MHBLOCKS blocks
    const int64_t ctm = cdiv(n, F_MHCOLS);
    const int64_t rbm = clamp64(cdiv(F_MHBLOCKS, ctm), 1, cdiv(m, F_MHGROUP));
    t.mr = (int)round_up(cdiv(m, rbm), F_MHGROUP);
    t.blocks[K_QPAD] = cdiv((int64_t)t.n_pad * rp, kBlock);
    t.blocks[K_PASS_P] = t.ng;
    t.blocks[K_PASS_Q] = col_tiles * t.sq;   // plus one block per matrix forming T
    t.blocks[K_QRED] = cdiv(n * rp * qfin_slices(t.sq), kBlock);
    t.blocks[K_APPLY] = cdiv(m * (rp / 4), kBlock);
    t.blocks[K_MHAT] = ctm * cdiv(m, t.mr);
    return t;
  }
  // Grid sizes.  The split kernels aim at about L_SPLIT_BLOCKS blocks over
  // the whole batch (the reconstruction, which has no partials, at twice
  // as many), rounded to whole rounds of resident blocks; each matrix takes
  // its share by element count (`share` = this matrix's fraction of the
  // call's elements), but at least a quarter round.  Each split adds a
  // partial (rows x rank for the left product, summed by the Gram kernel;
  // cols x rank for the right product), so splits stay at least L_MIN_COLS
  // columns / L_MIN_ROWS rows wide.
  auto target_of = [&](int64_t want, int64_t slots) {
    const int64_t total = whole_rounds(want, slots);
    return std::max<int64_t>(std::max<int64_t>(1, total / 4), (int64_t)(share * (double)total + 0.5));
  };
  // the bf16 rank-128 left product (one 8-wave block per compute unit) aims
  // at half as many blocks: half the column splits, so half the P partials
  // written and summed (4 x 16384 x 8192: 4.11 -> 4.07 ms; a quarter: 4.10)
  const int64_t target = target_of(x3 && rp >= 128 ? L_SPLIT_BLOCKS / 2 : L_SPLIT_BLOCKS, sl.p);
  // the bf16 rank-128 right product (two 8-wave blocks per compute unit)
  // aims at half as many blocks: one round, half the row splits, so half
  // the partials for the Q reduction (4 x 16384 x 8192: 4.16 -> 4.12 ms)
  const int64_t target_q = target_of(x3 && rp >= 128 ? L_SPLIT_BLOCKS / 2 : L_SPLIT_BLOCKS, sl.q);
  const int64_t target_m = target_of(2 * L_SPLIT_BLOCKS, sl.m);
  // left product: 128-row tiles, columns split, splits at least L_MIN_COLS
  // wide -- narrower, down to L_MIN_NARROW, while this matrix's blocks would
  // leave its share of one round of resident blocks partly empty (a matrix of
  // few rows, e.g. the rows of a row-sparse step)
  const int64_t row_tiles = cdiv(m, lp_block_rows(rp, x3));
  int64_t min_cols = L_MIN_COLS;
  auto sp_of = [&](int64_t mc) { return clamp64(cdiv(target, row_tiles), 1, cdiv(n, mc)); };
  while (min_cols > L_MIN_NARROW && row_tiles * sp_of(min_cols) < (int64_t)(share * (double)sl.p))
    min_cols /= 2;
  const int64_t sp = sp_of(min_cols);
  t.p_cols = (int)round_up(cdiv(n, sp), L_KC);
  t.sp = (int)cdiv(n, t.p_cols);
  // Gram partials: L_GROWS rows per block, fewer (down to 32) for a matrix
  // too short to give its share of about 128 blocks (a row-sparse step's
  // rows); every block also sums the column splits of its rows
  const int64_t g_want = std::max<int64_t>(1, (int64_t)(share * 128.0));
  t.grows = (int)clamp64(round_up(cdiv(m, g_want), 32), 32, L_GROWS);
  t.ng = (int)cdiv(m, t.grows);
  // right product: column tiles, rows split
  const int64_t ctq = cdiv(n, lq_block_cols(rp, x3));
  // splits of L_MIN_ROWS rows, halved (down to L_MIN_NARROW) while they
  // would leave this matrix's share of one round of resident blocks partly
  // empty (a single 51200 x 3072 matrix at rank 64: 600 of 1024 slots, so
  // 512-row splits; 0.24 -> 0.20 ms)
  int64_t min_rows = L_MIN_ROWS;
  while (min_rows > L_MIN_NARROW && ctq * cdiv(m, min_rows) < (int64_t)(share * (double)sl.q))
    min_rows /= 2;
  const int64_t sq = clamp64(cdiv(target_q, ctq), 1, cdiv(m, min_rows));
  // splits start on 16-row boundaries: the bf16 right product walks 16-row
  // groups, and its P_hat^T parts are stored in 16-row tiles
  t.q_rows = (int)round_up(cdiv(m, sq), 2 * L_QG);
  t.sq = (int)cdiv(m, t.q_rows);
  // reconstruction: column tiles x row blocks (multiple of 32 rows)
  const int64_t ctm = cdiv(n, lm_block_cols(rp));
  const int64_t rbm = clamp64(cdiv(target_m, ctm), 1, cdiv(m, 32));
  t.mr = (int)round_up(cdiv(m, rbm), 32);
  t.blocks[K_QPAD] = cdiv(t.n_pad, 32);   // 32-column tiles (k_qpadl)
  t.blocks[K_PASS_P] = row_tiles * t.sp;
  t.blocks[K_PGRAM] = t.ng;
  t.blocks[K_GSUM] = cdiv((int64_t)rp * rp, kBlock / 8);   // 32 entries per block
  t.blocks[K_GRAM2] = t.ng;
  t.blocks[K_APPLY] = cdiv(m, L_AROWS);
  t.blocks[K_PASS_Q] = ctq * t.sq;
  // Q reduction: 32-column tiles, or 8-column ones (four times the blocks)
  // where 32-column tiles would leave this matrix's share of one round of
  // resident blocks mostly empty: each element sums sq partials, so few
  // blocks serialise the whole sq x n x rp read (51200 x 3072 at rank 64:
  // 100 partials, 96 blocks; 50 -> 16 us)
  t.qr_cols = cdiv(n, 32) < (int64_t)(share * 512.0) ? 8 : 32;
  t.blocks[K_QRED] = cdiv(n, t.qr_cols);
  t.blocks[K_MHAT] = ctm * cdiv(m, t.mr);
  return t;
}

// Workspace layout: [header 256 B: sticky flags word][descriptor table]
// [per-matrix regions].  occ_workspace_init zeroes the header.
constexpr size_t kHeaderBytes = 256;
constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Regions {
  size_t qpad, phat, praw, ppart, qpart, gpart, gsum, t1, tm, info, phat_t, qbf, total;
};

inline Regions matrix_regions(int64_t m, int64_t n, int rp, const Tiling& t) {
  Regions g{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  g.qpad = take((size_t)t.n_pad * rp * 4);
  g.phat = take((size_t)m * rp * 4);
  g.praw = take((size_t)m * rp * 4);
  g.ppart = take((size_t)t.sp * m * rp * 4);
  g.qpart = take((size_t)t.sq * n * rp * (rp <= kFusedMaxRank ? 8 : 4));   // fp64 at rank <= 16
  g.gpart = take((size_t)t.ng * rp * rp * 8);
  g.gsum = take((size_t)rp * rp * 8);
  g.t1 = take((size_t)rp * rp * 8);
  g.tm = take((size_t)rp * rp * 8);
  g.info = take(64);
  g.phat_t = take(rp > kFusedMaxRank ? (size_t)rp * t.m_pad * 4 : 0);
  g.qbf = take(rp > kFusedMaxRank ? (size_t)2 * rp * t.n_pad * 2 : 0);
  g.total = off;
  return g;
}

}  // namespace occ
