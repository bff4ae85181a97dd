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

// Tile constants of the small-rank vector-ALU path.
constexpr int PP_ROWS = 64;     // pass P: rows per block (one lane per row)
constexpr int PP_SUB = 32;      // pass P: columns per wave sub-tile
constexpr int PP_PITCH = 36;    // pass P: LDS row pitch in floats
constexpr int G_ROWS = 256;     // Gram partial: rows per block
constexpr int MH_ROWS = 64;     // M_hat pass: rows per block

// Rank chunk and columns per lane of the streaming kernels for a padded rank.
__host__ __device__ constexpr int cols_per_lane(int rp) { return rp <= 16 ? 4 : 1; }
__host__ __device__ constexpr int q_rank_chunk(int rp) { return rp <= 16 ? rp : 32; }

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
  float* qpart;          // sq x n x rp
  double* gpart;         // ng x rp x rp
  double* gsub;          // ceil(ng / 16) x rp x rp (group sums of the Gram tree)
  double* gsum;          // rp x rp
  double* t1;            // rp x rp
  double* tm;            // rp x rp
  uint32_t* info;        // [0] = second CholeskyQR pass needed
  // shapes
  int32_t m, n, r;
  int32_t ldm, lde_in, lde_out, ldh;
  int32_t n_pad;
  int32_t sp, p_cols;    // pass P: column splits and columns per split (multiple of PP_SUB)
  int32_t ng;            // Gram partial blocks (G_ROWS rows each)
  int32_t sq, q_rows;    // pass Q: row splits and rows per split
  int32_t gb;            // fused path: blocks of the Gram-sum/Cholesky kernel
  int32_t blk[K_NUM];    // first block of this matrix in each kernel's grid
  int32_t fused;         // 1: fused small-rank path (rank padded to <= 16)
  int32_t pad_;
};

// Tiling of one matrix (host side).
struct Tiling {
  int sp, p_cols, ng, sq, q_rows, n_pad, gb;
  int64_t blocks[K_NUM];
};

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return cdiv(a, b) * b; }

inline int padded_rank(int r) {
  int p = 4;
  while (p < r) p *= 2;
  return p;
}

// Fused small-rank path: tile constants shared with kernels_small.hpp.
constexpr int kFusedMaxRank = 16;
constexpr int F_PROWS = 32;       // left product: rows per block
constexpr int F_QCOLS = 128;      // right product: columns per block
constexpr int F_QMAXROWS = 512;   // right product: rows per block (P_hat rows in LDS)
constexpr int F_MHROWS = 256;     // reconstruction: rows per block
constexpr int F_MHCOLS = 256;     // reconstruction: columns per block (4 per lane)
constexpr int F_QBLOCKS = 512;    // right product: target number of blocks
constexpr int F_ORTHROWS = 128;   // Cholesky/P_hat kernel: rows of P_hat per block

inline Tiling make_tiling(int64_t m, int64_t n, int rp, bool fused) {
  Tiling t{};
  t.n_pad = (int)round_up(n, PP_SUB);
  // pass P: 64-row tiles; split the columns until there are enough blocks,
  // keeping at least 128 (fused: 256) columns per split.
  int64_t row_tiles = cdiv(m, PP_ROWS);
  const int64_t p_blocks = fused ? cdiv(m, F_PROWS) : row_tiles;
  int64_t sp = cdiv(1024, p_blocks);
  int64_t max_sp = cdiv(n, fused ? 256 : 128);
  if (sp > max_sp) sp = max_sp;
  if (sp < 1) sp = 1;
  t.p_cols = (int)round_up(cdiv(n, sp), PP_SUB);
  t.sp = (int)cdiv(n, t.p_cols);
  t.ng = fused ? (int)p_blocks : (int)cdiv(m, G_ROWS);
  if (fused) {
    // left product: whole rows per block, no column splits
    t.sp = 1;
    t.p_cols = (int)round_up(n, PP_SUB);
    t.ng = (int)p_blocks;
    t.gb = 1;
    const int64_t col_tiles = cdiv(n, F_QCOLS);
    int64_t sq = cdiv(F_QBLOCKS, col_tiles);
    const int64_t max_sq = cdiv(m, 32);
    if (sq > max_sq) sq = max_sq;
    if (sq < 1) sq = 1;
    t.q_rows = (int)round_up(cdiv(m, sq), 4);
    t.sq = (int)cdiv(m, t.q_rows);
    t.blocks[K_QPAD] = cdiv((int64_t)t.n_pad * rp, kBlock);
    t.blocks[K_PASS_P] = p_blocks;
    t.blocks[K_PGRAM] = cdiv(m, F_ORTHROWS);
    t.blocks[K_GSUM] = 0;
    t.blocks[K_GRAM2] = 0;
    t.blocks[K_APPLY] = 0;
    t.blocks[K_PASS_Q] = col_tiles * t.sq;
    t.blocks[K_QRED] = cdiv(n * rp, kBlock);
    t.blocks[K_MHAT] = cdiv(n, F_MHCOLS) * cdiv(m, F_MHROWS);
    return t;
  }
  // pass Q: column tiles of 64*cols_per_lane; row splits up to ~1024 blocks
  int cpl = cols_per_lane(rp);
  int64_t col_tiles = cdiv(n, (int64_t)kWave * cpl);
  int rchunks = rp / q_rank_chunk(rp);
  int64_t sq = cdiv(1024, col_tiles * rchunks);
  int64_t max_sq = cdiv(m, 64);
  if (sq > max_sq) sq = max_sq;
  if (sq < 1) sq = 1;
  t.q_rows = (int)round_up(cdiv(m, sq), 4);
  t.sq = (int)cdiv(m, t.q_rows);

  t.blocks[K_QPAD] = cdiv((int64_t)t.n_pad * rp, kBlock);
  t.blocks[K_PASS_P] = row_tiles * t.sp;
  t.blocks[K_PGRAM] = t.ng;
  t.blocks[K_GSUM] = cdiv((int64_t)rp * rp, kBlock);
  t.blocks[K_GRAM2] = t.ng;
  t.blocks[K_APPLY] = cdiv(m, 64);
  t.blocks[K_PASS_Q] = col_tiles * t.sq * rchunks;
  t.blocks[K_QRED] = cdiv(n * rp, kBlock);
  t.blocks[K_MHAT] = cdiv(n, (int64_t)kWave * cpl) * cdiv(m, MH_ROWS);
  return t;
}

// Workspace layout: [header 256 B: sticky flags word][descriptor table]
// [per-matrix regions].  occ_workspace_init zeroes the header.
constexpr size_t kHeaderBytes = 256;
constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Regions {
  size_t qpad, phat, praw, ppart, qpart, gpart, gsub, gsum, t1, tm, info, total;
};

inline Regions matrix_regions(int64_t m, int64_t n, int rp, const Tiling& t) {
  Regions g{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  g.qpad = take((size_t)t.n_pad * rp * 4);
  g.phat = take((size_t)m * rp * 4);
  g.praw = take((size_t)m * rp * 4);
  g.ppart = take((size_t)t.sp * m * rp * 4);
  g.qpart = take((size_t)t.sq * n * rp * 4);
  g.gpart = take((size_t)t.ng * rp * rp * 8);
  g.gsub = take((size_t)(t.gb > 0 ? t.gb : cdiv(t.ng, 16)) * rp * rp * 8);
  g.gsum = take((size_t)rp * rp * 8);
  g.t1 = take((size_t)rp * rp * 8);
  g.tm = take((size_t)rp * rp * 8);
  g.info = take(64);
  g.total = off;
  return g;
}

}  // namespace occ
