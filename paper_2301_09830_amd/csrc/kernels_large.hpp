// Large-rank path (padded rank RP = 32, 64 or 128) on the matrix cores.
//
// Every product of a power-iteration round is a dense contraction with a
// 32..128-wide factor, so all three streaming passes run on
// v_mfma_f32_32x32x2_f32 (fp32 operands, fp32 accumulation).  Lane layout
// (lane l = 32*g + li):
//   A operand  a = A[i = li][k = g]       B operand  b = B[k = g][j = li]
//   result     D[i = 8*(v/4) + 4*g + v%4][j = li] in component v (16 floats)
// so each half-wave of an output register holds 32 consecutive columns of
// one row.
//
// A pass takes A = M + err_prev from one of three places (template SA):
//   SA_MERR       M and err_prev, added on the fly (compress-only calls);
//   SA_MERR_SAVE  the same, and the pass stores A over err (first left
//                 product of a fused step: the error buffer is about to be
//                 replaced by A - M_hat anyway);
//   SA_SAVED      A read back from the error buffer (every later pass of a
//                 fused step), 4 bytes per element instead of s_M + 4.
// The stored A is exactly the fp32 sum the other modes form in registers, so
// all three give bitwise the same products.
//
//   k_lp      P partials = A Q.  A block owns 128 rows (32 per wave) and a
//             column split; its waves walk the same 32-column K-steps, the
//             Q tile of the step staged once in LDS.  Lane (g, li) loads 16
//             consecutive columns of its row and feeds 16 MFMAs per rank
//             tile.  Output ranks are interleaved (lane li of rank tile u
//             holds rank RP/32*li + u) so one LDS vector read gives a lane
//             all its B values and one vector store writes its P values.
//   k_lg      P = sum of the splits (stored), fp64 Gram partial of 256 rows.
//   k_lchol   one block per matrix: T = R^-1 of the Gram G = R^T R (fp64),
//             right-looking, one barrier per column.
//   k_lapply  P_hat = P T (fp64 arithmetic, fp32 result), also stored
//             transposed for the reconstruction pass.
//   k_lq      Q partials = A^T P_hat over row splits; the waves of a block
//             own adjacent column strips and share the P_hat rows of each
//             8-row step through LDS.
//   k_ml      M_hat = P_hat Q^T and err = A - M_hat; a wave keeps its Q
//             columns in registers and walks 32-row tiles whose P_hat block
//             is staged (transposed) in LDS; at padded rank 64 the outputs
//             pass through LDS to be stored by rows.
#pragma once

#include <type_traits>

#include "kernels_mfma16.hpp"

namespace occ {

typedef float f16v __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f16v mfma32(float a, float b, f16v c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Row inside a 32x32 MFMA tile of accumulator component v, lanes of half g.
__device__ __forceinline__ constexpr int mf32_row(int v, int g) {
  return 8 * (v >> 2) + 4 * g + (v & 3);
}

enum { SA_MERR = 0, SA_MERR_SAVE = 1, SA_SAVED = 2 };

// W consecutive floats / 32-bit words (W a power of two, naturally aligned).
template <int W>
__device__ __forceinline__ void ld_f(const float* p, float* o) {
  if constexpr (W == 1) {
    o[0] = *p;
  } else if constexpr (W == 2) {
    const float2 v = *(const float2*)p;
    o[0] = v.x; o[1] = v.y;
  } else {
#pragma unroll
    for (int j = 0; j < W; j += 4) {
      const float4 v = *(const float4*)(p + j);
      o[j] = v.x; o[j + 1] = v.y; o[j + 2] = v.z; o[j + 3] = v.w;
    }
  }
}

template <int W>
__device__ __forceinline__ void ld_u(const uint32_t* p, uint32_t* o) {
  if constexpr (W == 1) {
    o[0] = *p;
  } else if constexpr (W == 2) {
    const uint2 v = *(const uint2*)p;
    o[0] = v.x; o[1] = v.y;
  } else {
#pragma unroll
    for (int j = 0; j < W; j += 4) {
      const uint4 v = *(const uint4*)(p + j);
      o[j] = v.x; o[j + 1] = v.y; o[j + 2] = v.z; o[j + 3] = v.w;
    }
  }
}

template <int W>
__device__ __forceinline__ void st_f(float* p, const float* v) {
  if constexpr (W == 1) {
    *p = v[0];
  } else if constexpr (W == 2) {
    *(float2*)p = make_float2(v[0], v[1]);
  } else {
#pragma unroll
    for (int j = 0; j < W; j += 4) *(float4*)(p + j) = make_float4(v[j], v[j + 1], v[j + 2], v[j + 3]);
  }
}

// W consecutive elements of A (columns c..c+W-1 of one row) as raw loads,
// converted only when used so that the loads stay in flight.  Elements that
// are out of range, or that the vector path cannot take, hold the exact A
// value (0 out of range) in e and -0 in m (x + -0 == x for every x).
template <int DT, int SA, int W>
struct RawA {
  static constexpr int MW = SA == SA_SAVED ? 1 : (DT == DT_BF16 ? (W >= 2 ? W / 2 : 1) : W);
  uint32_t m[MW];
  float e[W];
};

template <int DT, int SA, int W, bool RM = false>
__device__ __forceinline__ RawA<DT, SA, W> rawa_load(const Desc& d, bool vec, int row, int c,
                                                    int c_hi) {
  RawA<DT, SA, W> x;
  if (vec && row < d.m && c + W <= c_hi) {
    // M and err_prev rows through the row map; the stored A is compact
    const int64_t pr = SA == SA_SAVED ? (int64_t)row : prow<RM>(d, row);
    if constexpr (SA == SA_SAVED) {
      ld_f<W>(d.err_out + pr * d.lde_out + c, x.e);
      x.m[0] = 0u;
    } else {
      if constexpr (DT == DT_BF16) {
        const uint16_t* mp = (const uint16_t*)d.M + pr * d.ldm + c;
        if constexpr (W == 1) x.m[0] = (uint32_t)(*mp) << 16;
        else ld_u<W / 2>((const uint32_t*)mp, x.m);
      } else {
        ld_u<W>((const uint32_t*)((const float*)d.M + pr * d.ldm + c), x.m);
      }
      if (d.err_in) {
        ld_f<W>(d.err_in + pr * d.lde_in + c, x.e);
      } else {
#pragma unroll
        for (int j = 0; j < W; ++j) x.e[j] = -0.f;
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < W; ++j) {
      float v = 0.f;
      if (row < d.m && c + j < c_hi) {
        const int64_t pr = SA == SA_SAVED ? (int64_t)row : prow<RM>(d, row);
        if constexpr (SA == SA_SAVED) {
          v = d.err_out[pr * d.lde_out + c + j];
        } else {
          v = m_elem<DT>(d, pr * d.ldm + c + j);
          if (d.err_in) v = v + d.err_in[pr * d.lde_in + c + j];
        }
      }
      x.e[j] = v;
    }
    const uint32_t nz = (SA != SA_SAVED && DT == DT_BF16 && W >= 2) ? 0x80008000u : 0x80000000u;
#pragma unroll
    for (int w = 0; w < RawA<DT, SA, W>::MW; ++w) x.m[w] = nz;
  }
  return x;
}

template <int DT, int SA, int W>
__device__ __forceinline__ float rawa_val(const RawA<DT, SA, W>& x, int j) {
  if constexpr (SA == SA_SAVED) {
    return x.e[j];
  } else if constexpr (DT == DT_BF16) {
    if constexpr (W == 1) return __uint_as_float(x.m[0]) + x.e[0];
    else return ((j & 1) ? bf16_hi(x.m[j >> 1]) : bf16_lo(x.m[j >> 1])) + x.e[j];
  } else {
    return __uint_as_float(x.m[j]) + x.e[j];
  }
}

// Store W values of A over the error buffer (row < m).  Plain stores: the
// stored A is read back by the next pass, and nontemporal stores measured
// slower for the whole step.
template <int W>
__device__ __forceinline__ void a_store(const Desc& d, bool vec, int row, int c, int c_hi,
                                        const float* a) {
  if (row >= d.m) return;
  float* p = d.err_out + (int64_t)row * d.lde_out + c;
  if (vec && c + W <= c_hi) {
    st_f<W>(p, a);
  } else {
#pragma unroll
    for (int j = 0; j < W; ++j)
      if (c + j < c_hi) p[j] = a[j];
  }
}

// First column of K-step `it` of a split starting at c_lo whose walk starts at
// K-step ks0 and wraps around after nk steps (it < nk).
__device__ __forceinline__ int kcol_of(int c_lo, int ks0, int it, int nk) {
  int k = ks0 + it;
  if (k >= nk) k -= nk;
  return c_lo + L_KC * k;
}

// -------------------------------------------------------------------------
// k_lp: P partials = A Q for one row tile (lp_block_rows: 32 rows per wave)
// and one column split.
//
// X3 (bf16 M): the products run on v_mfma_f32_32x32x16_bf16 with each
// operand split in two bf16 parts, x = x_hi + x_lo (x - x_hi - x_lo is below
// 2^-16 |x|), and A Q accumulated in fp32 as A_hi Q_hi + A_hi Q_lo +
// A_lo Q_hi: about 1e-5 relative accuracy at 3/16 of the matrix-core cycles
// of the fp32 v_mfma_f32_32x32x2_f32 form.  Lane (g, li) of a K-step holds
// columns 16g..16g+15 of its row; MFMA c (0, 1) takes its columns
// 16g + 8c .. 16g + 8c + 7 as K indices 8g..8g+7, and the B operand reads the
// same columns of the Q tile, which is staged as bf16 hi/lo rows (one row per
// rank, 32 columns) in the order k -> (k % NU) * 32 + k / NU so that lane li
// of rank tile u finds rank NU li + u in row 32 u + li.
// -------------------------------------------------------------------------
constexpr int LB_P = L_KC + 8;   // LDS pitch (bf16) of a staged Q row: 80 bytes

template <int RP>
struct LPSmem {
  float q[2][L_KC * (RP + 4)];   // Q rows of the current and next K-step
};
template <int RP>
struct LPXSmem {
  uint16_t q[2][2][RP * LB_P];   // [stage][hi, lo][rank row][column]
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f16v mfma32bf(bf16x8 a, bf16x8 b, f16v c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// A tiles of the left product through LDS (16-byte aligned rows, whole
// 32-column K-steps).  With A fed straight from registers, lane li of a
// 32x32 operand owns row li, so each load instruction touches 32 rows with
// 32 bytes each and every 128-byte line is requested four times; the L1
// address path then stalls the texture addresser for 40-70 % of the pass.
// global_load_lds_dwordx4 writes lane l's 16 bytes to LDS at base + 16 l, so
// a wave brings its 32 x 32 tile in with whole lines per instruction (8 rows
// x 128 bytes of fp32, 16 rows x 64 bytes of bf16), lanes taking their
// chunks in an XOR-swizzled order so that the operand reads (lane (g, li):
// row li, columns 16g..16g+15) are free of bank conflicts.  Two stages per
// wave: the wave reads its operands, issues the next K-step's tile, then
// runs the products.  The stored A of a first pass is written from the
// tile in the same whole-line order.
constexpr int LP_ESLOT = 1024 + 128;   // 8 rows x 128 B of fp32; the pad shifts banks by 32 words
constexpr int LP_BSLOT = 1024;         // 16 rows x 64 B of bf16
template <int DT, int SA>
struct LPTile {
  static constexpr int A_BYTES = 4 * LP_ESLOT;   // err (or the stored A)
  static constexpr int M_BYTES = SA == SA_SAVED ? 0 : (DT == DT_BF16 ? 2 * LP_BSLOT : 4 * LP_ESLOT);
  static constexpr int BYTES = A_BYTES + M_BYTES;
};

// Rows of M and err_prev a lane's tile loads read (the tile rows are the same
// for every K-step of a wave): with the row map, looked up once before the
// K-loop, so the loop issues nothing but the tile DMA its wait counts assume.
struct LPRows {
  int64_t a[4];   // err_prev rows 8q + l / 8
  int64_t m[4];   // M rows: bf16 16q + l / 4 (q < 2), fp32 as a
};

template <int DT, bool RM>
__device__ __forceinline__ LPRows lp_rows(const Desc& d, int row0) {
  LPRows r{};
  if constexpr (RM) {
    const int lane = threadIdx.x & 63, last = d.m - 1;
#pragma unroll
    for (int q = 0; q < 4; ++q) r.a[q] = prow<RM>(d, min(row0 + 8 * q + (lane >> 3), last));
#pragma unroll
    for (int q = 0; q < 4; ++q)
      r.m[q] = DT == DT_BF16 ? (q < 2 ? prow<RM>(d, min(row0 + 16 * q + (lane >> 2), last)) : 0)
                             : r.a[q];
  }
  return r;
}

// Cache policy of tile loads (2: non-temporal) for data read once in whole
// lines: the stored A of later passes and fp32 M.  err is read and then
// overwritten by the stored A in the same lines, and a bf16 K-step reads half
// of each M line (the other half comes with the next K-step), so both keep
// the default policy.  Measured (same session): the later rank-128 left
// product 507 -> 471 us, the stage matrices' 801 -> 747 us and their first
// pass 2457 -> 2408 us, the embedding's first pass 414 -> 396 us; bf16 M
// non-temporal made the rank-128 first pass 1161 -> 1267 us.
constexpr int LP_NT = 2;
template <int DT, int SA, bool RM = false>
__device__ __forceinline__ void lp_tile_issue(const Desc& d, int row0, int c0, uint8_t* dst,
                                              const LPRows& pr = LPRows{}) {
  const int lane = threadIdx.x & 63;
  const int last = d.m - 1;
  const float* asrc = SA == SA_SAVED ? d.err_out : d.err_in;
  const int64_t lda = SA == SA_SAVED ? d.lde_out : d.lde_in;
  // the stored A is compact: only M and err_prev go through the row map
  constexpr bool MAP = RM && SA != SA_SAVED;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    // rows 8q .. 8q+7: lane l takes row l / 8, chunk (l % 8) ^ (l / 8)
    const int rr = lane >> 3, ch = (lane & 7) ^ rr;
    const int64_t row = MAP ? pr.a[q] : (int64_t)min(row0 + 8 * q + rr, last);
    __builtin_amdgcn_global_load_lds((gvoid_t*)(asrc + row * lda + c0 + 4 * ch),
                                     (lvoid_t*)(dst + q * LP_ESLOT), 16, 0,
                                     SA == SA_SAVED ? LP_NT : 0);
  }
  if constexpr (SA != SA_SAVED) {
    uint8_t* mdst = dst + LPTile<DT, SA>::A_BYTES;
    if constexpr (DT == DT_BF16) {
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        // rows 16q .. 16q+15: lane l takes row l / 4, chunk (l % 4) ^ (l / 16)
        const int rr = lane >> 2, ch = (lane & 3) ^ (rr >> 2);
        const int64_t row = MAP ? pr.m[q] : (int64_t)min(row0 + 16 * q + rr, last);
        __builtin_amdgcn_global_load_lds(
            (gvoid_t*)((const uint16_t*)d.M + row * d.ldm + c0 + 8 * ch),
            (lvoid_t*)(mdst + q * LP_BSLOT), 16, 0, 0);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int rr = lane >> 3, ch = (lane & 7) ^ rr;
        const int64_t row = MAP ? pr.m[q] : (int64_t)min(row0 + 8 * q + rr, last);
        __builtin_amdgcn_global_load_lds(
            (gvoid_t*)((const float*)d.M + row * d.ldm + c0 + 4 * ch),
            (lvoid_t*)(mdst + q * LP_ESLOT), 16, 0, LP_NT);
      }
    }
  }
}

// A[row li][columns 16g .. 16g+15] of a tile (the values rawa_val gives).
template <int DT, int SA>
__device__ __forceinline__ void lp_tile_read(const uint8_t* src, int li, int g, float a[16]) {
  const int q = li >> 3, rr = li & 7;
  const uint8_t* e = src + q * LP_ESLOT + rr * 128;
  float ev[16];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const float4 v = *(const float4*)(e + 16 * ((4 * g + t) ^ rr));
    ev[4 * t] = v.x; ev[4 * t + 1] = v.y; ev[4 * t + 2] = v.z; ev[4 * t + 3] = v.w;
  }
  if constexpr (SA == SA_SAVED) {
#pragma unroll
    for (int j = 0; j < 16; ++j) a[j] = ev[j];
  } else if constexpr (DT == DT_BF16) {
    const int qb = li >> 4, rb = li & 15;
    const uint8_t* m = src + LPTile<DT, SA>::A_BYTES + qb * LP_BSLOT + rb * 64;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const uint4 w = *(const uint4*)(m + 16 * ((2 * g + t) ^ (rb >> 2)));
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        a[8 * t + 2 * k] = bf16_lo(ww[k]) + ev[8 * t + 2 * k];
        a[8 * t + 2 * k + 1] = bf16_hi(ww[k]) + ev[8 * t + 2 * k + 1];
      }
    }
  } else {
    const uint8_t* m = src + LPTile<DT, SA>::A_BYTES + q * LP_ESLOT + rr * 128;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float4 v = *(const float4*)(m + 16 * ((4 * g + t) ^ rr));
      a[4 * t] = v.x + ev[4 * t]; a[4 * t + 1] = v.y + ev[4 * t + 1];
      a[4 * t + 2] = v.z + ev[4 * t + 2]; a[4 * t + 3] = v.w + ev[4 * t + 3];
    }
  }
}

// First pass: A = M + err_prev of the wave's tile stored over err, each lane
// taking its own tile slots (whole 128-byte lines per store instruction).
template <int DT>
__device__ __forceinline__ void lp_tile_store_a(const Desc& d, const uint8_t* src, int row0, int c0) {
  const int lane = threadIdx.x & 63;
  const int rr = lane >> 3, ch = (lane & 7) ^ rr;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int r = 8 * q + rr;          // row within the wave's 32
    const float4 e = *(const float4*)(src + q * LP_ESLOT + 16 * lane);
    float a[4];
    if constexpr (DT == DT_BF16) {
      const int qb = r >> 4, rb = r & 15;
      const uint2 w = *(const uint2*)(src + LPTile<DT, SA_MERR_SAVE>::A_BYTES + qb * LP_BSLOT + rb * 64 +
                                      16 * ((ch >> 1) ^ (rb >> 2)) + 8 * (ch & 1));
      a[0] = bf16_lo(w.x) + e.x; a[1] = bf16_hi(w.x) + e.y;
      a[2] = bf16_lo(w.y) + e.z; a[3] = bf16_hi(w.y) + e.w;
    } else {
      const float4 m = *(const float4*)(src + LPTile<DT, SA_MERR_SAVE>::A_BYTES + q * LP_ESLOT + 16 * lane);
      a[0] = m.x + e.x; a[1] = m.y + e.y; a[2] = m.z + e.z; a[3] = m.w + e.w;
    }
    const int row = row0 + r;
    if (row < d.m)
      *(float4*)(d.err_out + (int64_t)row * d.lde_out + c0 + 4 * ch) = make_float4(a[0], a[1], a[2], a[3]);
  }
}

// RM (row-sparse step): M and err_prev rows through the row map; the stored A
// (SA_MERR_SAVE writes it, SA_SAVED reads it) is compact.
template <int DT, int RP, int SA, bool X3, bool TILES, bool RM = false>
__device__ __forceinline__ void lp_body(const Desc& d, int b,
                                        std::conditional_t<X3, LPXSmem<RP>, LPSmem<RP>>& sm,
                                        uint8_t* tiles) {
  constexpr int NU = RP / 32;               // rank tiles
  constexpr int QP = RP + 4;                // LDS pitch of a Q row (fp32 form)
  constexpr int LR = lp_block_rows(RP, X3);  // rows per block, 32 per wave
  constexpr int NT = LR / 32 * kWave;        // threads per block
  // 16-byte chunks of one K-step's Q tile per thread: fp32 form RP x 32 x 4 B,
  // bf16 form 2 x RP x 32 x 2 B (the same count)
  constexpr int QF4 = L_KC * RP / 4 / NT;
  static_assert(QF4 * 4 * NT == L_KC * RP, "Q tile must split evenly");
  const bool vec = d.vec != 0;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
  const int row_tiles = (d.m + LR - 1) / LR;
  const int rt = b % row_tiles, s = b / row_tiles;
  const int row = rt * LR + 32 * wave + li;
  const int c_lo = s * d.p_cols;
  const int c_hi = min(d.n, c_lo + d.p_cols);
  const int nk = (c_hi - c_lo + L_KC - 1) / L_KC;
  // Row tiles start their walk at staggered K-steps (and wrap around) so the
  // device does not read one column stripe of every row at a time.
  const int ks0 = (int)(((int64_t)rt * 4) % nk);

  f16v acc[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) acc[u] = f16v{};

  // Source and LDS slot of this thread's chunk x of the Q tile at column c.
  // fp32 form: qpad has n_pad (a multiple of 32) rows, so every K-step's Q
  // tile is in bounds (rows past n are zero); bf16 form: qbf rows have n_pad
  // columns, likewise zero past n.
  auto q_src_ptr = [&](int c, int x) -> const f4v* {
    const int f = threadIdx.x + NT * x;
    if constexpr (X3) {
      const int h = f / (RP * 4), rem = f % (RP * 4);
      return (const f4v*)(d.qbf + ((int64_t)h * RP + rem / 4) * d.n_pad + c + 8 * (rem % 4));
    } else {
      return (const f4v*)(d.qpad + (int64_t)c * RP + 4 * f);
    }
  };
  auto q_lds_ptr = [&](int stage, int x) -> f4v* {
    const int f = threadIdx.x + NT * x;
    if constexpr (X3) {
      const int h = f / (RP * 4), rem = f % (RP * 4);
      return (f4v*)(&sm.q[stage][h][(rem / 4) * LB_P + 8 * (rem % 4)]);
    } else {
      return (f4v*)(&sm.q[stage][((4 * f) / RP) * QP + (4 * f) % RP]);
    }
  };

  // Q tiles are fetched LP_QAHEAD K-steps before they are needed (a register
  // ring) and written to the LDS buffer of the next K-step at the end of each
  // step; A loads run LP_DEPTH K-steps ahead.
  constexpr int LP_QAHEAD = RP >= 128 ? 1 : 3;
  constexpr int LP_DEPTH = RP >= 128 ? 2 : 1;
  f4v qr[LP_QAHEAD][QF4];
#pragma unroll
  for (int y = 0; y < LP_QAHEAD; ++y)
    if (y < nk) {
      const int c = kcol_of(c_lo, ks0, y, nk);
#pragma unroll
      for (int x = 0; x < QF4; ++x) qr[y][x] = *q_src_ptr(c, x);
    }
#pragma unroll
  for (int x = 0; x < QF4; ++x) *q_lds_ptr(0, x) = qr[0][x];
  auto mfma_step = [&](const float a[16], int stage) {
    if constexpr (X3) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x8 ahi, alo;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float v = a[8 * c + e];
          const __bf16 h = (__bf16)v;
          ahi[e] = h;
          alo[e] = (__bf16)(v - (float)h);
        }
        const uint16_t* qh = &sm.q[stage][0][li * LB_P + 16 * g + 8 * c];
        const uint16_t* ql = &sm.q[stage][1][li * LB_P + 16 * g + 8 * c];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          const bf16x8 bh = *(const bf16x8*)(qh + 32 * u * LB_P);
          const bf16x8 bl = *(const bf16x8*)(ql + 32 * u * LB_P);
          acc[u] = mfma32bf(ahi, bh, acc[u]);
          acc[u] = mfma32bf(ahi, bl, acc[u]);
          acc[u] = mfma32bf(alo, bh, acc[u]);
        }
      }
    } else {
      const float* qb = sm.q[stage] + 16 * g * QP + NU * li;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        float bv[NU];
        ld_f<NU>(qb + j * QP, bv);
#pragma unroll
        for (int u = 0; u < NU; ++u) acc[u] = mfma32(a[j], bv[u], acc[u]);
      }
    }
  };
  // Q ring: slot y holds K-step it + y; fetch K-step it + LP_QAHEAD
  auto q_advance = [&](int it) {
#pragma unroll
    for (int y = 0; y + 1 < LP_QAHEAD; ++y)
#pragma unroll
      for (int x = 0; x < QF4; ++x) qr[y][x] = qr[y + 1][x];
    if (it + LP_QAHEAD < nk) {
      const int c = kcol_of(c_lo, ks0, it + LP_QAHEAD, nk);
#pragma unroll
      for (int x = 0; x < QF4; ++x) qr[LP_QAHEAD - 1][x] = *q_src_ptr(c, x);
    }
  };

  // TILES: A tiles through LDS (the host picks this instance when rows are
  // 16-byte aligned, every K-step is whole and A has a source); else A goes
  // straight into registers.
  if constexpr (TILES) {
    constexpr int SB = LPTile<DT, SA>::BYTES;
    uint8_t* const wt = tiles + wave * 2 * SB;   // this wave's two stages
    const int wrow0 = rt * LR + 32 * wave;
    const LPRows prw = lp_rows<DT, RM && SA != SA_SAVED>(d, wrow0);
    lp_tile_issue<DT, SA, RM>(d, wrow0, kcol_of(c_lo, ks0, 0, nk), wt, prw);
    __syncthreads();
    for (int it = 0; it < nk; ++it) {
      const int kc0 = kcol_of(c_lo, ks0, it, nk);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      q_advance(it);
      const uint8_t* cur = wt + (it & 1) * SB;
      float a[16];
      lp_tile_read<DT, SA>(cur, li, g, a);
      if constexpr (SA == SA_MERR_SAVE) lp_tile_store_a<DT>(d, cur, wrow0, kc0);
      if (it + 1 < nk)
        lp_tile_issue<DT, SA, RM>(d, wrow0, kcol_of(c_lo, ks0, it + 1, nk), wt + ((it + 1) & 1) * SB, prw);
      mfma_step(a, it & 1);
      if (it + 1 < nk) {
#pragma unroll
        for (int x = 0; x < QF4; ++x) *q_lds_ptr((it + 1) & 1, x) = qr[0][x];
      }
      __syncthreads();
    }
  } else {
    RawA<DT, SA, 16> ring[LP_DEPTH + 1];
#pragma unroll
    for (int x = 0; x <= LP_DEPTH; ++x)
      if (x < nk) ring[x] = rawa_load<DT, SA, 16, RM>(d, vec, row, kcol_of(c_lo, ks0, x, nk) + 16 * g, c_hi);
    __syncthreads();

    int kc = kcol_of(c_lo, ks0, 0, nk);
    for (int it = 0; it < nk; ++it) {
      q_advance(it);
      float a[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) a[j] = rawa_val<DT, SA, 16>(ring[0], j);
      if constexpr (SA == SA_MERR_SAVE) a_store<16>(d, vec, row, kc + 16 * g, c_hi, a);
      mfma_step(a, it & 1);
#pragma unroll
      for (int x = 0; x < LP_DEPTH; ++x) ring[x] = ring[x + 1];
      if (it + LP_DEPTH + 1 < nk)
        ring[LP_DEPTH] = rawa_load<DT, SA, 16, RM>(d, vec, row, kcol_of(c_lo, ks0, it + LP_DEPTH + 1, nk) + 16 * g, c_hi);
      if (it + 1 < nk) {
        // slot 0 now holds K-step it + 1
#pragma unroll
        for (int x = 0; x < QF4; ++x) *q_lds_ptr((it + 1) & 1, x) = qr[0][x];
        kc = kcol_of(c_lo, ks0, it + 1, nk);
      }
      __syncthreads();
    }
  }

  // acc[u][v] = P[rt*LR + 32*wave + mf32_row(v, g)][NU*li + u] (this split)
  float* dst = d.ppart + (int64_t)s * d.m * RP;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int r = rt * LR + 32 * wave + mf32_row(v, g);
    if (r < d.m) {
      float o[NU];
#pragma unroll
      for (int u = 0; u < NU; ++u) o[u] = acc[u][v];
      st_f<NU>(dst + (int64_t)r * RP + NU * li, o);
    }
  }
}

template <int DT, int RP, int SA, bool X3, bool TILES, bool RM = false>
__global__ __launch_bounds__(lp_block_rows(RP, X3) / 32 * kWave) void k_lp(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) std::conditional_t<X3, LPXSmem<RP>, LPSmem<RP>> sm;
  __shared__ __attribute__((aligned(16))) uint8_t
      tiles[TILES ? lp_block_rows(RP, X3) / 32 * 2 * LPTile<DT, SA>::BYTES : 16];
#define B_(d, b) lp_body<DT, RP, SA, X3, TILES, RM>(d, b, sm, tiles)
  OCC_DISPATCH(K_PASS_P, B_)
#undef B_
}

// -------------------------------------------------------------------------
// k_lg: Gram partial of d.grows rows (256, fewer for short matrices) in
// fp64.  MODE 0: the rows are P (sum of the left product's column splits,
// stored to praw).  MODE 1 (second CholeskyQR pass, skipped unless the first
// pass asked for it): the rows are the first pass's P_hat.  Rows are staged in LDS as doubles, 32 at a
// time; the upper-triangle 16 x 16 tiles of G (ta <= tb) are shared out
// over the four waves and accumulated on v_mfma_f64_16x16x4f64, four rows
// per instruction: lane (q, li) supplies P[row 4s + q][16 ta + li] (A
// operand) and P[row 4s + q][16 tb + li] (B operand) and ends with
// G[16 ta + 4v + q][16 tb + li] in component v.  Only the upper tiles are
// written; the Gram sum zeroes the lower triangle (the Cholesky reads only
// the upper one).
// -------------------------------------------------------------------------
typedef double d4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ d4v mfma64(double a, double b, d4v c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

template <int RP>
struct LGSmem {
  double rows[32][RP + 2];
};

// upper-triangle tiles of an NTT x NTT tile grid, in row-major order
__host__ __device__ constexpr int lg_ntiles(int rp) { return (rp / 16) * (rp / 16 + 1) / 2; }
__host__ __device__ constexpr int lg_per_wave(int rp) { return (lg_ntiles(rp) + 3) / 4; }

template <int RP, int MODE>
__device__ __forceinline__ void lg_body(const Desc& d, int b, LGSmem<RP>& sm) {
  if (MODE == 1 && !d.info[0]) return;
  constexpr int NTT = RP / 16, NTL = lg_ntiles(RP), PW = lg_per_wave(RP);
  const int t = threadIdx.x;
  const int wave = wave_id(), lane = t & 63;
  const int q = lane >> 4, li = lane & 15;
  // this wave's tiles: indices wave, wave + 4, ... of the upper triangle
  int ta[PW], tb[PW];
#pragma unroll
  for (int x = 0; x < PW; ++x) {
    int idx = wave + 4 * x, r = 0;
    if (idx >= NTL) idx = NTL - 1;   // padding slot (not written)
    while (idx >= NTT - r) { idx -= NTT - r; ++r; }
    ta[x] = r;
    tb[x] = r + idx;
  }
  d4v acc[PW];
#pragma unroll
  for (int x = 0; x < PW; ++x) acc[x] = d4v{0.0, 0.0, 0.0, 0.0};
  // Staging: thread t owns float4 e of each 32-row chunk (E4 per thread).
  // The next chunk's loads (the first LG_PB column splits in MODE 0) are
  // issued before the current chunk's products so their latency overlaps
  // them; further splits are added after, in split order.
  constexpr int E4 = 32 * RP / 4 / kBlock;
  constexpr int LG_PB = 4;
  static_assert(E4 >= 1 && 32 * RP / 4 == E4 * kBlock, "staging layout");
  const int r_lo = b * d.grows, r_hi = min(d.m, r_lo + d.grows);
  float4 pre[E4][LG_PB];
  auto fetch = [&](int c0) {
#pragma unroll
    for (int e = 0; e < E4; ++e) {
      const int idx = t + kBlock * e, i = idx / (RP / 4), k4 = idx % (RP / 4);
      const int64_t row = c0 + i;
#pragma unroll
      for (int p = 0; p < LG_PB; ++p) {
        pre[e][p] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row < r_hi && (p == 0 || (MODE == 0 && p < d.sp))) {
          const float* base = MODE == 0 ? d.ppart + ((int64_t)p * d.m + row) * RP : d.phat + row * RP;
          pre[e][p] = *(const float4*)(base + 4 * k4);
        }
      }
    }
  };
  auto stage = [&](int c0) {
#pragma unroll
    for (int e = 0; e < E4; ++e) {
      const int idx = t + kBlock * e, i = idx / (RP / 4), k4 = idx % (RP / 4);
      const int64_t row = c0 + i;
      float4 v = pre[e][0];
      if (MODE == 0 && row < r_hi) {
#pragma unroll
        for (int p = 1; p < LG_PB; ++p)
          if (p < d.sp) v = make_float4(v.x + pre[e][p].x, v.y + pre[e][p].y, v.z + pre[e][p].z,
                                        v.w + pre[e][p].w);
        for (int p = LG_PB; p < d.sp; ++p) {
          const float4 w = *(const float4*)(d.ppart + ((int64_t)p * d.m + row) * RP + 4 * k4);
          v = make_float4(v.x + w.x, v.y + w.y, v.z + w.z, v.w + w.w);
        }
        *(float4*)(d.praw + row * RP + 4 * k4) = v;
      }
      double2* dst = (double2*)&sm.rows[i][4 * k4];
      dst[0] = make_double2((double)v.x, (double)v.y);
      dst[1] = make_double2((double)v.z, (double)v.w);
    }
  };
  fetch(r_lo);
  for (int c0 = r_lo; c0 < r_hi; c0 += 32) {
    stage(c0);
    __syncthreads();
    if (c0 + 32 < r_hi) fetch(c0 + 32);

#pragma unroll 2
    for (int s4 = 0; s4 < 8; ++s4) {
      const double* rowp = sm.rows[4 * s4 + q];
#pragma unroll
      for (int x = 0; x < PW; ++x) {
        const double av = rowp[16 * ta[x] + li];
        const double bv = rowp[16 * tb[x] + li];
        acc[x] = mfma64(av, bv, acc[x]);
      }
    }
    __syncthreads();
  }
  double* gp = d.gpart + (int64_t)b * RP * RP;
#pragma unroll
  for (int x = 0; x < PW; ++x) {
    if (wave + 4 * x >= NTL) continue;
#pragma unroll
    for (int v = 0; v < 4; ++v) gp[(16 * ta[x] + 4 * v + q) * RP + 16 * tb[x] + li] = acc[x][v];
  }
}

template <int RP, int MODE>
__global__ __launch_bounds__(kBlock) void k_lg(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) LGSmem<RP> sm;
#define B_(d, b) lg_body<RP, MODE>(d, b, sm)
  OCC_DISPATCH(MODE == 0 ? K_PGRAM : K_GRAM2, B_)
#undef B_
}

// -------------------------------------------------------------------------
// k_lchol: T = R^-1 with G = R^T R (fp64), one block of 1024 threads per
// matrix, blocked in 16 x 16 tiles (NB = RP/16 tile rows, tiles of the
// upper triangle only, held in LDS).  Step j:
//   1. wave 0 factors the diagonal tile W_jj = R_jj^T R_jj with the
//      right-looking column recurrence (Cholesky of W_jj together with the
//      column recurrence of its inverse factor; each lane reads the pivot
//      row of W and the pivot column of T from the owning lanes' registers
//      with cross-lane shuffles, so a column step waits for one round of
//      shuffles instead of an LDS write and read), giving T_jj = R_jj^-1
//      and the pivots, while the other waves finish column block j-1 of T
//      (step 4);
//   2. row panel R_jk = T_jj^T W_jk (k > j) and U_kj = R_kj T_jj (k < j);
//   3. trailing update W_kl -= R_jk^T R_jl (j < k <= l);
//   4. T_ij = -sum_{k=i..j-1} T_ik U_kj (i < j), from T R = I.
// Tile products run on v_mfma_f64_16x16x4f64, four per 16-deep product:
// lane (q, li) supplies X[li][4s+q] (A operand) and Y[4s+q][li] (B
// operand), and holds D[4v+q][li] in component v.  Tiles are stored with
// element (r, c) at r*16 + (c ^ r), so both operand patterns are free of
// bank conflicts.  A pivot <= kPivotTol * max diag(G), or a padding column
// (k >= r), is dependent: its row of R and its row and column of T are zero,
// which drops that direction exactly as the unblocked recurrence does.
//   MODE 0: T -> t1; decide whether a second pass is needed (info[0]).
//   MODE 1: only when info[0]; T of the first pass's P_hat -> tm.
// -------------------------------------------------------------------------
constexpr int LC_THREADS = 1024;
constexpr int LC_WAVES = LC_THREADS / kWave;

__host__ __device__ constexpr int lc_ntiles(int nb) { return nb * (nb + 1) / 2; }
// index of upper tile (a, b), a <= b, in row-major order of the triangle
__device__ __forceinline__ int lc_ut(int nb, int a, int b) { return a * nb - a * (a - 1) / 2 + (b - a); }
__device__ __forceinline__ int lc_sw(int r, int c) { return r * 16 + (c ^ r); }

template <int RP>
struct LCSmem {
  double W[lc_ntiles(RP / 16)][256];   // G, then R (row panels) and U
  double T[lc_ntiles(RP / 16)][256];
  double sdiag[RP];    // sqrt of each pivot (0 when dependent)
  int dep[RP];
  double thr;
};

// 1/v for v > 0: hardware estimate refined by two Newton steps
// (y <- y + y (1 - v y)), accurate to an ulp or two.
__device__ __forceinline__ double rcp_nr(double v) {
  double y = __builtin_amdgcn_rcp(v);
  double e = fma(-v, y, 1.0);
  y = fma(y, e, y);
  e = fma(-v, y, 1.0);
  return fma(y, e, y);
}

// D (+)= sum over 16 of A * B for one tile product; fa(s) / fb(s) give the
// lane's A / B operand of step s.
template <class FA, class FB>
__device__ __forceinline__ d4v lc_mm(FA fa, FB fb, d4v acc) {
#pragma unroll
  for (int s = 0; s < 4; ++s) acc = mfma64(fa(s), fb(s), acc);
  return acc;
}

template <int RP, int MODE>
__device__ __forceinline__ void lchol_body(const Desc& d, uint32_t* flags, LCSmem<RP>& sm) {
  if (MODE == 1 && !d.info[0]) return;
  constexpr int NB = RP / 16, NUT = lc_ntiles(NB);
  const int t = threadIdx.x, wave = t / kWave, lane = t % kWave;
  const int q = lane >> 4, li = lane & 15;
  const int r = d.r;
  const double* G = d.gsum;
  // operand readers on swizzled tiles
  auto rdA = [&](const double* X, int s) { return X[lc_sw(li, 4 * s + q)]; };   // X[li][4s+q]
  auto rdB = [&](const double* X, int s) { return X[lc_sw(4 * s + q, li)]; };   // X[4s+q][li]
  auto ldD = [&](const double* X) {
    d4v v;
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = X[lc_sw(4 * c + q, li)];
    return v;
  };
  auto stD = [&](double* X, d4v v) {
#pragma unroll
    for (int c = 0; c < 4; ++c) X[lc_sw(4 * c + q, li)] = v[c];
  };

  // G's upper tiles into LDS, all of a thread's loads in flight at once
  constexpr int GL = (NUT * 256 + LC_THREADS - 1) / LC_THREADS;
  double gl[GL];
#pragma unroll
  for (int x = 0; x < GL; ++x) {
    const int idx = t + LC_THREADS * x;
    gl[x] = 0.0;
    if (idx < NUT * 256) {
      const int u = idx >> 8, e = idx & 255, rr = e >> 4, cc = e & 15;
      int a = 0, rem = u;
      while (rem >= NB - a) { rem -= NB - a; ++a; }
      gl[x] = G[(16 * a + rr) * RP + 16 * (a + rem) + cc];
    }
  }
#pragma unroll
  for (int x = 0; x < GL; ++x) {
    const int idx = t + LC_THREADS * x;
    if (idx < NUT * 256) sm.W[idx >> 8][lc_sw((idx & 255) >> 4, idx & 15)] = gl[x];
  }
  __syncthreads();
  if (t < kWave) {
    // max of diag(G) over the first wave (max is order-independent), from LDS
    double mx = 0.0;
    int nonfinite = 0;
    for (int j = t; j < RP; j += kWave) {
      const double gv = sm.W[lc_ut(NB, j >> 4, j >> 4)][lc_sw(j & 15, j & 15)];
      if (!isfinite(gv)) nonfinite = 1;
      if (gv > mx) mx = gv;
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      const double o = __shfl_xor(mx, off);
      mx = o > mx ? o : mx;
      nonfinite |= __shfl_xor(nonfinite, off);
    }
    if (t == 0) {
      sm.thr = kPivotTol * mx;
      if (nonfinite && flags) atomicOr(flags, FLAG_NONFINITE);
    }
  }
  __syncthreads();
  const double thr = sm.thr;

  // step 4 for column block jc: wave w (from w0) takes T_ij, i = w - w0
  auto t_column = [&](int jc, int w0) {
    const int i = wave - w0;
    if (i < 0 || i >= jc) return;
    d4v acc = d4v{0.0, 0.0, 0.0, 0.0};
    for (int k = i; k < jc; ++k) {
      const double* Tik = sm.T[lc_ut(NB, i, k)];
      const double* Ukj = sm.W[lc_ut(NB, k, jc)];
      acc = lc_mm([&](int s) { return -rdA(Tik, s); }, [&](int s) { return rdB(Ukj, s); }, acc);
    }
    stD(sm.T[lc_ut(NB, i, jc)], acc);
  };

#pragma unroll 1
  for (int j = 0; j < NB; ++j) {
    if (wave == 0) {
      // 1. diagonal tile: lane (q, li) holds W_jj[4v+q][li] and T_jj[4v+q][li]
      double* Wd = sm.W[lc_ut(NB, j, j)];
      double W[4], T[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        W[v] = Wd[lc_sw(4 * v + q, li)];
        T[v] = (4 * v + q == li) ? 1.0 : 0.0;
      }
      double mypiv = 0.0;
      bool mydep = true;
      // fully unrolled: each column's register and source lanes are fixed at
      // compile time, and the compiler overlaps one column's independent
      // shuffles with the previous column's updates (rank 64: 32 -> 26 us)
#pragma unroll
      for (int jv = 0; jv < 4; ++jv) {
#pragma unroll
        for (int jq = 0; jq < 4; ++jq) {
          const int jj = 4 * jv + jq;
          // Row jj of W is W[jv] of lanes (jq, 0..15); column jj of T is T[v]
          // of lanes (q, jj).  Read straight from those lanes' registers.
          double w = W[0];
#pragma unroll
          for (int v = 1; v < 4; ++v) w = (jv == v) ? W[v] : w;
          const double piv = __shfl(w, 16 * jq + jj);
          const double wk = __shfl(w, 16 * jq + li);
          double wi[4], tl[4];
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            wi[v] = __shfl(w, 16 * jq + 4 * v + q);
            tl[v] = __shfl(T[v], 16 * q + jj);
          }
          const bool dep = (16 * j + jj >= r) || (piv <= thr);
          if (li == jj) {
            mypiv = piv;
            mydep = dep;
          }
          if (!dep && li > jj) {
            const double ip = rcp_nr(piv);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int i = 4 * v + q;
              if (i > jj) {
                if (i <= li) W[v] = fma(-(wi[v] * ip), wk, W[v]);
              } else {
                T[v] = fma(-(tl[v] * ip), wk, T[v]);
              }
            }
          }
        }
      }
      const double isq = mydep ? 0.0 : rsqrt_nr(mypiv);
      const double sq = mypiv * isq;   // sqrt of the pivot (0 when dependent)
      double* Td = sm.T[lc_ut(NB, j, j)];
#pragma unroll
      for (int v = 0; v < 4; ++v) Td[lc_sw(4 * v + q, li)] = (4 * v + q <= li && !mydep) ? T[v] * isq : 0.0;
      if (q == 0) {
        sm.sdiag[16 * j + li] = sq;
        sm.dep[16 * j + li] = mydep ? 1 : 0;
        if (mydep && 16 * j + li < r && flags) atomicOr(flags, FLAG_RANK_DEFICIENT);
      }
    } else if (j > 0) {
      t_column(j - 1, 1);
    }
    __syncthreads();
    // 2. row panel and U, one tile per wave
    {
      const double* Tjj = sm.T[lc_ut(NB, j, j)];
      for (int x = wave; x < NB - 1; x += LC_WAVES) {
        const int k = x < j ? x : x + 1;
        if (k > j) {
          double* Wjk = sm.W[lc_ut(NB, j, k)];
          const d4v o = lc_mm([&](int s) { return rdB(Tjj, s); }, [&](int s) { return rdB(Wjk, s); },
                              d4v{0.0, 0.0, 0.0, 0.0});
          stD(Wjk, o);
        } else {
          double* Rkj = sm.W[lc_ut(NB, k, j)];
          const d4v o = lc_mm([&](int s) { return rdA(Rkj, s); }, [&](int s) { return rdB(Tjj, s); },
                              d4v{0.0, 0.0, 0.0, 0.0});
          stD(Rkj, o);
        }
      }
    }
    __syncthreads();
    // 3. trailing update over the upper tiles (k, l), j < k <= l
    if (j + 1 < NB) {
      const int nr = NB - 1 - j;
      for (int x = wave; x < nr * (nr + 1) / 2; x += LC_WAVES) {
        int a = 0, rem = x;
        while (rem >= nr - a) { rem -= nr - a; ++a; }
        const int k = j + 1 + a, l = k + rem;
        const double* Rjk = sm.W[lc_ut(NB, j, k)];
        const double* Rjl = sm.W[lc_ut(NB, j, l)];
        double* Wkl = sm.W[lc_ut(NB, k, l)];
        const d4v o = lc_mm([&](int s) { return -rdB(Rjk, s); }, [&](int s) { return rdB(Rjl, s); }, ldD(Wkl));
        stD(Wkl, o);
      }
      __syncthreads();
    }
  }
  // 4. for the last column block
  t_column(NB - 1, 0);
  __syncthreads();

  double* out = MODE == 0 ? d.t1 : d.tm;
  for (int idx = t; idx < RP * RP; idx += LC_THREADS) {
    const int l = idx / RP, k = idx % RP, a = l >> 4, b = k >> 4;
    out[idx] = (a <= b) ? sm.T[lc_ut(NB, a, b)][lc_sw(l & 15, k & 15)] : 0.0;
  }
  if (MODE == 0 && t < kWave) {
    double dmax = 0.0, dmin = 1e308;
    for (int j = t; j < r; j += kWave) {
      if (sm.dep[j]) continue;
      const double v = sm.sdiag[j];
      dmax = v > dmax ? v : dmax;
      dmin = v < dmin ? v : dmin;
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      const double a = __shfl_xor(dmax, off), c = __shfl_xor(dmin, off);
      dmax = a > dmax ? a : dmax;
      dmin = c < dmin ? c : dmin;
    }
    if (t == 0) d.info[0] = (dmax > 0.0 && dmax > kSecondPassCond * dmin) ? 1u : 0u;
  }
}

template <int RP, int MODE>
__global__ __launch_bounds__(LC_THREADS) void k_lchol(OCC_KARGS, uint32_t* flags) {
  __shared__ LCSmem<RP> sm;
  if (count == 1) lchol_body<RP, MODE>(single, flags, sm);
  else lchol_body<RP, MODE>(table[blockIdx.x], flags, sm);
}

// -------------------------------------------------------------------------
// k_lapply: P_hat = S T for 128 rows, S = praw, T = t1 (MODE 0) or, in the
// second pass, S = the first pass's P_hat, T = tm (in place).  fp64
// products on v_mfma_f64_16x16x4f64, fp32 result.  T is upper triangular,
// so column tile jt of P_hat needs only k < 16 (jt + 1).  The column tiles
// are paired (jt, NTT-1-jt), which makes every pair the same amount of
// work; wave w takes pair w % NP and row tiles 2 (w / NP), 2 (w / NP) + 1
// of each chunk of CR rows, and keeps its two T column tiles in registers
// for the whole block.  In step s lane (q, li) supplies S[16 rt + li][4 s + q]
// (A operand, from the staged chunk) and T[4 s + q][16 jt + li] (B operand)
// and ends with P_hat[16 rt + 4 v + q][16 jt + li] in component v.  The
// chunk's results are written back into the staging buffer and stored as
// whole rows to phat and, for the final P_hat (no second pass pending), to
// the caller's P and transposed to phat_t.
// -------------------------------------------------------------------------
template <int RP>
struct LAShape {
  static constexpr int NTT = RP / 16, NP = NTT / 2, WPP = 4 / NP, CR = 32 * WPP;
  static constexpr int LD = RP + 4;
};

template <int RP>
struct LASmem {
  float buf[LAShape<RP>::CR][LAShape<RP>::LD];
};

template <int RP, int MODE>
__device__ __forceinline__ void la_body(const Desc& d, int b, LASmem<RP>& sm) {
  const uint32_t need = d.info[0];
  if (MODE == 1 && !need) return;
  using S_ = LAShape<RP>;
  constexpr int NTT = S_::NTT, NP = S_::NP, CR = S_::CR;
  static_assert(L_AROWS % CR == 0, "apply chunk must divide the block's rows");
  constexpr int KA_MAX = 4 * NP;        // steps of the pair's first tile (jt = pair <= NP-1)
  constexpr int KB_MAX = 4 * NTT;       // steps of the pair's second tile (jt = NTT-1-pair)
  const bool fin = (MODE == 1) || !need;
  const double* Tg = MODE == 0 ? d.t1 : d.tm;
  const float* src = MODE == 0 ? d.praw : d.phat;
  const int t = threadIdx.x, wave = wave_id(), lane = t & 63;
  const int q = lane >> 4, li = lane & 15;
  const int pair = wave % NP, rsub = wave / NP;
  const int ja = pair, jb = NTT - 1 - pair;
  const int ka = 4 * (ja + 1), kb = 4 * (jb + 1);   // steps per tile
  // T column tiles in registers (B operands)
  double ta[KA_MAX], tb[KB_MAX];
#pragma unroll
  for (int s = 0; s < KA_MAX; ++s) ta[s] = (s < ka) ? Tg[(4 * s + q) * RP + 16 * ja + li] : 0.0;
#pragma unroll
  for (int s = 0; s < KB_MAX; ++s) tb[s] = (s < kb) ? Tg[(4 * s + q) * RP + 16 * jb + li] : 0.0;

  const int r_lo = b * L_AROWS, r_hi = min(d.m, r_lo + L_AROWS);
  // the rows of S of the next chunk are loaded into registers while this
  // chunk's products and stores run (rows past m as zeros)
  constexpr int SF = CR * RP / 4 / kBlock;   // float4s per thread per chunk
  static_assert(SF * kBlock == CR * RP / 4, "chunk staging layout");
  float4 nx[SF];
  auto fetch = [&](int c0) {
#pragma unroll
    for (int x = 0; x < SF; ++x) {
      const int idx = t + kBlock * x, i = idx / (RP / 4), k4 = idx % (RP / 4);
      nx[x] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (c0 + i < r_hi) nx[x] = *(const float4*)(src + (int64_t)(c0 + i) * RP + 4 * k4);
    }
  };
  if (r_lo < r_hi) fetch(r_lo);
  for (int c0 = r_lo; c0 < r_hi; c0 += CR) {
#pragma unroll
    for (int x = 0; x < SF; ++x) {
      const int idx = t + kBlock * x, i = idx / (RP / 4), k4 = idx % (RP / 4);
      *(float4*)&sm.buf[i][4 * k4] = nx[x];
    }
    __syncthreads();
    if (c0 + CR < r_hi) fetch(c0 + CR);
    d4v acc[2][2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      acc[u][0] = d4v{0.0, 0.0, 0.0, 0.0};
      acc[u][1] = d4v{0.0, 0.0, 0.0, 0.0};
    }
    const float* srow0 = sm.buf[32 * rsub + li];
    const float* srow1 = sm.buf[32 * rsub + 16 + li];
#pragma unroll
    for (int s = 0; s < KB_MAX; ++s) {
      if (s < kb) {
        const double a0 = (double)srow0[4 * s + q], a1 = (double)srow1[4 * s + q];
        acc[0][1] = mfma64(a0, tb[s], acc[0][1]);
        acc[1][1] = mfma64(a1, tb[s], acc[1][1]);
        if (s < KA_MAX && s < ka) {
          acc[0][0] = mfma64(a0, ta[s], acc[0][0]);
          acc[1][0] = mfma64(a1, ta[s], acc[1][0]);
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float* orow = sm.buf[16 * (2 * rsub + u) + 4 * v + q];
        orow[16 * ja + li] = (float)acc[u][0][v];
        orow[16 * jb + li] = (float)acc[u][1][v];
      }
    __syncthreads();
    // whole rows out
    for (int idx = t; idx < CR * RP / 4; idx += kBlock) {
      const int i = idx / (RP / 4), k4 = idx % (RP / 4);
      const int row = c0 + i;
      if (row < r_hi) {
        const float4 v = *(const float4*)&sm.buf[i][4 * k4];
        *(float4*)(d.phat + (int64_t)row * RP + 4 * k4) = v;
        if (fin) {
          const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (4 * k4 + e < d.r) d.P[(int64_t)row * d.r + 4 * k4 + e] = vv[e];
        }
      }
    }
    if (fin) {
      // transposed: rank k, four consecutive rows per thread (rows past m
      // carry zeros, their source rows were staged as 0).  For bf16 M (qbf
      // set) the right product wants the bf16 hi/lo parts of P_hat in 16-row
      // tiles, so the same bytes hold [m_pad / 16][hi, lo][rank][16] uint16
      // instead of fp32 [rank][m_pad]: one group's tile is contiguous.
      uint16_t* tb = d.qbf ? (uint16_t*)d.phat_t : nullptr;
      for (int idx = t; idx < RP * CR / 4; idx += kBlock) {
        const int k = idx / (CR / 4), i4 = idx % (CR / 4);
        if (c0 + 4 * i4 < d.m_pad) {
          const float v[4] = {sm.buf[4 * i4][k], sm.buf[4 * i4 + 1][k], sm.buf[4 * i4 + 2][k],
                              sm.buf[4 * i4 + 3][k]};
          const int64_t o = (int64_t)k * d.m_pad + c0 + 4 * i4;
          if (tb) {
            uint16_t hi[4], lo[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const __bf16 h = (__bf16)v[e];
              hi[e] = bf16_bits(h);
              lo[e] = bf16_bits((__bf16)(v[e] - (float)h));
            }
            const int row = c0 + 4 * i4;
            const int64_t ot = ((int64_t)(row >> 4) * 2 * RP + k) * 16 + (row & 15);
            *(uint2*)(tb + ot) = make_uint2(hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16));
            *(uint2*)(tb + ot + RP * 16) =
                make_uint2(lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16));
          } else {
            *(float4*)(d.phat_t + o) = make_float4(v[0], v[1], v[2], v[3]);
          }
        }
      }
    }
    __syncthreads();
  }
}

template <int RP, int MODE>
__global__ __launch_bounds__(kBlock) void k_lapply(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) LASmem<RP> sm;
#define B_(d, b) la_body<RP, MODE>(d, b, sm)
  OCC_DISPATCH(K_APPLY, B_)
#undef B_
}

// -------------------------------------------------------------------------
// k_lq: Q partials = A^T P_hat for one column tile and one row split.
// Lane (g, li) of wave w loads lq_cpl columns starting at
// ct*BC + 32*cpl*w + cpl*li of rows 2ks + g; MFMA tile t of rank tile u then
// holds Q[col = base + cpl*i + t][rank = NU*j + u].
// -------------------------------------------------------------------------
template <int RP>
struct LQSmem {
  float p[2][L_QG][RP + 4];
};

template <int DT, int RP, int SA, bool RM = false>
__device__ __forceinline__ void lq_body(const Desc& d, int b, LQSmem<RP>& sm) {
  constexpr int NU = RP / 32, CPL = lq_cpl(RP), BC = lq_block_cols(RP);
  constexpr int PF = L_QG * RP / 4;   // float4s of one P_hat stage
  static_assert(PF <= kBlock, "one float4 per thread per stage");
  const bool vec = d.vec != 0;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
  const int t = threadIdx.x;
  const int col_tiles = (d.n + BC - 1) / BC;
  const int ct = b % col_tiles, s = b / col_tiles;
  const int cw = ct * BC + wave * 32 * CPL;
  const int col = cw + CPL * li;
  const int r_lo = s * d.q_rows, r_hi = min(d.m, r_lo + d.q_rows);
  const int ngrp = (r_hi - r_lo + L_QG - 1) / L_QG;
  const int pi = (4 * t) / RP, pk = (4 * t) % RP;   // this thread's staging slot

  f16v acc[CPL][NU];
#pragma unroll
  for (int x = 0; x < CPL; ++x)
#pragma unroll
    for (int u = 0; u < NU; ++u) acc[x][u] = f16v{};

  // P_hat rows of a group are fetched LQ_PAHEAD groups before they are
  // needed (a register ring) and written to the LDS buffer of the next group
  // at the end of each group; A loads run one group ahead.
  constexpr int LQ_PAHEAD = 3;
  f4v pr[LQ_PAHEAD];
#pragma unroll
  for (int y = 0; y < LQ_PAHEAD; ++y) {
    pr[y] = f4v{0.f, 0.f, 0.f, 0.f};
    const int row = r_lo + L_QG * y + pi;
    if (t < PF && row < r_hi) pr[y] = *(const f4v*)(d.phat + (int64_t)row * RP + pk);
  }
  if (t < PF) *(f4v*)(&sm.p[0][pi][pk]) = pr[0];
  RawA<DT, SA, CPL> cur[4], nxt[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int row = r_lo + 2 * ks + g;
    cur[ks] = rawa_load<DT, SA, CPL, RM>(d, vec, row < r_hi ? row : d.m, col, d.n);
  }
  __syncthreads();

  for (int grp = 0; grp < ngrp; ++grp) {
    const bool more = grp + 1 < ngrp;
    const int rn = r_lo + L_QG * (grp + 1);
#pragma unroll
    for (int y = 0; y + 1 < LQ_PAHEAD; ++y) pr[y] = pr[y + 1];
    {
      const int row = r_lo + L_QG * (grp + LQ_PAHEAD) + pi;
      pr[LQ_PAHEAD - 1] = f4v{0.f, 0.f, 0.f, 0.f};
      if (t < PF && row < r_hi) pr[LQ_PAHEAD - 1] = *(const f4v*)(d.phat + (int64_t)row * RP + pk);
    }
    if (more) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int row = rn + 2 * ks + g;
        nxt[ks] = rawa_load<DT, SA, CPL, RM>(d, vec, row < r_hi ? row : d.m, col, d.n);
      }
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      float bv[NU];
      ld_f<NU>(&sm.p[grp & 1][2 * ks + g][NU * li], bv);
#pragma unroll
      for (int x = 0; x < CPL; ++x) {
        const float a = rawa_val<DT, SA, CPL>(cur[ks], x);
#pragma unroll
        for (int u = 0; u < NU; ++u) acc[x][u] = mfma32(a, bv[u], acc[x][u]);
      }
    }
    if (more) {
      // slot 0 now holds group grp + 1
      if (t < PF) *(f4v*)(&sm.p[(grp + 1) & 1][pi][pk]) = pr[0];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) cur[ks] = nxt[ks];
    }
    __syncthreads();
  }

#pragma unroll
  for (int x = 0; x < CPL; ++x)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int c = cw + CPL * mf32_row(v, g) + x;
      if (c < d.n) {
        float o[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u) o[u] = acc[x][u][v];
        st_f<NU>(d.qpart + ((int64_t)s * d.n + c) * RP + NU * li, o);
      }
    }
}

// TILES form of k_lq for the stored fp32 A (rows 16-byte aligned, n a
// multiple of 32): both operands of a group come into LDS by DMA, AST - 1
// groups ahead, so the loads in flight are not bounded by registers.
//   A: each wave's 8 rows x 32 CPL columns, 8/CPL rows per 1 KB
//      global_load_lds_dwordx4 (lane l: row l / (8 CPL), chunk l % (8 CPL));
//      rows are contiguous in LDS, so the operand reads (lane (g, li): CPL
//      floats of row 2ks + g at column CPL li) are conflict-free;
//   P: the block's 8 rows x RP of P_hat (contiguous in memory), each wave
//      copying RP/32 runs of 256 bytes with global_load_lds_dword.
// Every wave issues the same number of loads per group, so one wait count
// covers the groups still in flight; the operand reads are inline ds_read
// instructions (the compiler would wait for every DMA in flight before a
// plain LDS read).
template <int RP>
struct LQTile {
  static constexpr int CPL = lq_cpl(RP), NU = RP / 32;
  static constexpr int NI = CPL;                       // A loads per wave and group
  static constexpr int NP = RP / 32;                   // P loads per wave and group
  static constexpr int A_BYTES = 1024 * CPL;           // one wave's A tile
  static constexpr int P_BYTES = L_QG * RP * 4;        // the block's P tile
  static constexpr int STAGE = 4 * A_BYTES + P_BYTES;
  static constexpr int AST = RP >= 128 ? 4 : 3;        // stages (3 blocks per CU at rank 32)
};

template <int RP>
__device__ __forceinline__ void lq_tile_issue(const Desc& d, int r0, int r_last, int cw, int wave,
                                              uint8_t* stage) {
  using T = LQTile<RP>;
  constexpr int CH = 8 * T::CPL, RPI = 8 / T::CPL;
  const int lane = threadIdx.x & 63;
  const int rr = lane / CH, ch = lane % CH;
  const int c = min(cw + 4 * ch, d.n - 4);
  uint8_t* adst = stage + wave * T::A_BYTES;
#pragma unroll
  for (int q = 0; q < T::NI; ++q) {
    const int row = min(r0 + q * RPI + rr, r_last);
    __builtin_amdgcn_global_load_lds((gvoid_t*)(d.err_out + (int64_t)row * d.lde_out + c),
                                     (lvoid_t*)(adst + q * 1024), 16, 0, 0);
  }
  uint8_t* pdst = stage + 4 * T::A_BYTES;
#pragma unroll
  for (int j = 0; j < T::NP; ++j) {
    const int run = wave * T::NP + j;                  // 64-float run of the P tile
    const int idx = run * 64 + lane;
    const int row = min(r0 + idx / RP, d.m - 1);        // rows past m: any finite value
    __builtin_amdgcn_global_load_lds((gvoid_t*)(d.phat + (int64_t)row * RP + idx % RP),
                                     (lvoid_t*)(pdst + run * 256), 4, 0, 0);
  }
}

template <int RP>
__device__ __forceinline__ void lq_tiles_body(const Desc& d, int b, uint8_t* tiles) {
  using T = LQTile<RP>;
  constexpr int NU = T::NU, CPL = T::CPL, BC = lq_block_cols(RP), AST = T::AST;
  constexpr int PER_GROUP = T::NI + T::NP;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
  const int col_tiles = (d.n + BC - 1) / BC;
  const int ct = b % col_tiles, s = b / col_tiles;
  const int cw = ct * BC + wave * 32 * CPL;
  const int col = cw + CPL * li;
  const int r_lo = s * d.q_rows, r_hi = min(d.m, r_lo + d.q_rows);
  const int ngrp = (r_hi - r_lo + L_QG - 1) / L_QG;
  const int r_last = r_hi - 1;

  f16v acc[CPL][NU];
#pragma unroll
  for (int x = 0; x < CPL; ++x)
#pragma unroll
    for (int u = 0; u < NU; ++u) acc[x][u] = f16v{};

#pragma unroll
  for (int y = 0; y + 1 < AST; ++y)
    if (y < ngrp) lq_tile_issue<RP>(d, r_lo + L_QG * y, r_last, cw, wave, tiles + y * T::STAGE);

  const uint32_t tbase = (uint32_t)(size_t)(lvoid_t*)tiles;
  int st_cur = 0;
  for (int grp = 0; grp < ngrp; ++grp) {
    const int r0 = r_lo + L_QG * grp;
    // groups issued after this one and possibly still in flight
    const int after = min(grp + AST - 2, ngrp - 1) - grp;
    static_assert(AST <= 4 && 2 * PER_GROUP <= 63, "vmcnt immediates");
    if (after <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else if (after == 1) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(PER_GROUP) : "memory");
    else asm volatile("s_waitcnt vmcnt(%0)" :: "n"(2 * PER_GROUP) : "memory");
    asm volatile("s_barrier" ::: "memory");   // every wave's P share is in

    typename LdsVec<CPL>::T av[4];
    typename LdsVec<NU>::T pv[4];
    const uint32_t sb = tbase + st_cur * T::STAGE;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int r = 2 * ks + g;
      ds_read_asm<CPL>(av[ks], sb + wave * T::A_BYTES + r * 128 * CPL + 4 * CPL * li);
      ds_read_asm<NU>(pv[ks], sb + 4 * T::A_BYTES + (r * RP + NU * li) * 4);
    }
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(av[0]), "+v"(av[1]), "+v"(av[2]), "+v"(av[3]),
                   "+v"(pv[0]), "+v"(pv[1]), "+v"(pv[2]), "+v"(pv[3]));

    const int st_new = st_cur == 0 ? AST - 1 : st_cur - 1;   // stage of group grp + AST - 1
    if (grp + AST - 1 < ngrp)
      lq_tile_issue<RP>(d, r0 + L_QG * (AST - 1), r_last, cw, wave, tiles + st_new * T::STAGE);
    st_cur = st_cur + 1 == AST ? 0 : st_cur + 1;

    const int nvalid = r_hi - r0 - g;   // rows 2ks + g of this group inside the split: 2ks < nvalid
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int x = 0; x < CPL; ++x) {
        const float a = 2 * ks < nvalid ? lds_elem<CPL>(av[ks], x) : 0.f;
#pragma unroll
        for (int u = 0; u < NU; ++u) acc[x][u] = mfma32(a, lds_elem<NU>(pv[ks], u), acc[x][u]);
      }
    }
  }

#pragma unroll
  for (int x = 0; x < CPL; ++x)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int c = cw + CPL * mf32_row(v, g) + x;
      if (c < d.n) {
        float o[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u) o[u] = acc[x][u][v];
        st_f<NU>(d.qpart + ((int64_t)s * d.n + c) * RP + NU * li, o);
      }
    }
  (void)col;
}

template <int DT, int RP, int SA, bool TILES, bool RM = false>
__global__ __launch_bounds__(kBlock) void k_lq(OCC_KARGS) {
  static_assert(!(TILES && RM), "the row map runs on the register form");
  if constexpr (TILES) {
    static_assert(DT == DT_F32 && SA == SA_SAVED, "tiles hold the stored fp32 A");
    __shared__ __attribute__((aligned(16))) uint8_t tiles[LQTile<RP>::AST * LQTile<RP>::STAGE];
#define B_(d, b) lq_tiles_body<RP>(d, b, tiles)
    OCC_DISPATCH_X(K_PASS_Q, B_)
#undef B_
  } else {
    __shared__ __attribute__((aligned(16))) LQSmem<RP> sm;
#define B_(d, b) lq_body<DT, RP, SA, RM>(d, b, sm)
    OCC_DISPATCH_X(K_PASS_Q, B_)
#undef B_
  }
}

// -------------------------------------------------------------------------
// k_lqx: the right product for bf16 M on the bf16 matrix cores, with split
// operands as in k_lp (X3): Q^T partial = P_hat^T A over 16-row groups, as
// v_mfma_f32_32x32x16_bf16 with
//   A operand  P_hat^T: lane (g, li) supplies rank 32u + li, rows 8g..8g+7 of
//              the group, from an LDS tile of bf16 hi/lo rows (16 rows per
//              rank) staged from the transposed P_hat (phat_t);
//   B operand  A: lane (g, li) supplies rows 8g..8g+7 of its column
//              ct*BC + 32*CPL*w + CPL*li + x (the same 2-row x 32-lane loads
//              as k_lq);
// so acc[x][u][v] = Q[col][rank 32u + mf32_row(v, g)] of this split.
// -------------------------------------------------------------------------
constexpr int LQX_G = 16;            // rows per group (K of two MFMA halves)

// The P_hat^T tile of a group, staged by global_load_lds_dwordx4 from the
// bf16 hi/lo parts of the transposed P_hat, which k_lapply writes in 16-row
// tiles [m_pad / 16][hi, lo][rank][16] (groups start on 16-row boundaries):
// one load instruction per (part, rank tile u) copies 1 KB of contiguous
// source, the 32 ranks x two 8-row halves; lane l fetches rank 32u + l / 2,
// half (l % 2) ^ (l / 16 % 2), which makes the operand reads (lane (g, li):
// rank 32u + li, half g) conflict-free.
template <int RP>
struct LQXSmem {
  uint16_t p[2][2][RP * LQX_G];      // [stage][hi, lo][rank tile][1 KB as above]
};

__device__ __forceinline__ int lqx_slot(int li, int g) { return 2 * li + (g ^ ((li >> 3) & 1)); }

// A tiles of the right product (TILES instances, stored fp32 A): each wave's
// 16-row group of its 32*CPL columns comes into LDS by global_load_lds_dwordx4
// in whole lines.  A row is 8*CPL chunks of 16 bytes; one instruction fills a
// 1 KB slot with 8/CPL rows (lane l: row l / (8 CPL), chunk l % (8 CPL)).
// Slots are 1152 bytes apart, so at CPL = 1 (one 128-byte row per half-wave
// of an operand read) rows e and 8 + e fall in opposite halves of the banks.
constexpr int LQX_SLOT = 1024 + 128;
// stages of A per wave at rank 128 (two groups ahead; two 8-wave blocks per
// compute unit)
constexpr int LQX_AST = 3;
template <int RP>
struct LQXTile {
  static constexpr int CPL = lq_cpl(RP);
  static constexpr int RPI = 8 / CPL;                 // rows per load instruction
  static constexpr int NI = LQX_G / RPI;              // slots per group
  static constexpr int BYTES = NI * LQX_SLOT;         // one stage of one wave
  // stages per wave: at rank 128 the A tiles run LQX_AST - 1 groups ahead
  static constexpr int AST = RP >= 128 ? LQX_AST : 2;
};

// Rows r0 .. r0+15 (clamped to r_last) of columns cw .. cw + 32 CPL - 1
// (chunks past the last column read the row's last chunk instead; those
// columns are never stored).
template <int RP>
__device__ __forceinline__ void lqx_tile_issue(const Desc& d, int r0, int r_last, int cw, uint8_t* dst) {
  using T = LQXTile<RP>;
  constexpr int CH = 8 * T::CPL;
  const int lane = threadIdx.x & 63;
  const int rr = lane / CH, ch = lane % CH;
  const int c = min(cw + 4 * ch, d.n - 4);
#pragma unroll
  for (int q = 0; q < T::NI; ++q) {
    const int row = min(r0 + q * T::RPI + rr, r_last);
    __builtin_amdgcn_global_load_lds((gvoid_t*)(d.err_out + (int64_t)row * d.lde_out + c),
                                     (lvoid_t*)(dst + q * LQX_SLOT), 16, 0, 0);
  }
}

// a[e][x] = A[row 8g + e of the group][column CPL li + x of the wave]
template <int RP>
__device__ __forceinline__ void lqx_tile_read(const uint8_t* src, int li, int g,
                                              float (&a)[8][LQXTile<RP>::CPL]) {
  using T = LQXTile<RP>;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int r = 8 * g + e;
    const float* p = (const float*)(src + (r / T::RPI) * LQX_SLOT + (r % T::RPI) * (128 * T::CPL)) +
                     T::CPL * li;
    ld_f<T::CPL>(p, a[e]);
  }
}

template <int DT, int RP, int SA, bool TILES, bool RM = false>
__device__ __forceinline__ void lqx_body(const Desc& d, int b, LQXSmem<RP>& sm, uint8_t* tiles) {
  static_assert(!(TILES && RM), "the row map runs on the register form");
  constexpr int NU = RP / 32, CPL = lq_cpl(RP), BC = lq_block_cols(RP, true);
  constexpr int NW = lqx_waves(RP);
  constexpr int NLD = 2 * NU;                         // P tile load instructions per group
  const bool vec = d.vec != 0;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
  const int col_tiles = (d.n + BC - 1) / BC;
  const int ct = b % col_tiles, s = b / col_tiles;
  const int cw = ct * BC + wave * 32 * CPL;
  const int col = cw + CPL * li;
  const int r_lo = s * d.q_rows, r_hi = min(d.m, r_lo + d.q_rows);
  const int ngrp = (r_hi - r_lo + LQX_G - 1) / LQX_G;
  const uint16_t* ptb = (const uint16_t*)d.phat_t;

  f16v acc[CPL][NU];
#pragma unroll
  for (int x = 0; x < CPL; ++x)
#pragma unroll
    for (int u = 0; u < NU; ++u) acc[x][u] = f16v{};

  // this wave's share of the P tile loads of group grp (rows past r_hi are
  // multiplied by the zero rows of A)
  auto p_issue = [&](int grp, int stage) {
    const int r0 = r_lo + LQX_G * grp;   // a multiple of 16
    const int rk = lane >> 1, h = (lane & 1) ^ ((lane >> 4) & 1);
#pragma unroll
    for (int j = wave; j < NLD; j += NW) {
      const int part = j / NU, u = j % NU;
      const uint16_t* src = ptb + (((int64_t)(r0 >> 4) * 2 + part) * RP + 32 * u + rk) * 16 + 8 * h;
      __builtin_amdgcn_global_load_lds((gvoid_t*)src, (lvoid_t*)(&sm.p[stage][part][32 * u * LQX_G]),
                                       16, 0, 0);
    }
  };
  auto a_fetch = [&](int grp, RawA<DT, SA, CPL>* x) {
    const int r0 = r_lo + LQX_G * grp;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int row = r0 + 8 * g + e;
      x[e] = rawa_load<DT, SA, CPL, RM>(d, vec, row < r_hi ? row : d.m, col, d.n);
    }
  };

  auto mfma_group = [&](const bf16x8 (&ah)[NU], const bf16x8 (&al)[NU], int x, const bf16x8& bh,
                        const bf16x8& bl) {
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      acc[x][u] = mfma32bf(ah[u], bh, acc[x][u]);
      acc[x][u] = mfma32bf(ah[u], bl, acc[x][u]);
      acc[x][u] = mfma32bf(al[u], bh, acc[x][u]);
    }
  };
  const int so = lqx_slot(li, g) * 8;   // this lane's P operand, in bf16 elements

  if constexpr (TILES) {
    // Per group: wait for this group's A tile and P share, barrier (every
    // wave's share of the P tile is in; every wave is done with the other P
    // stage), read the operands, issue the next group's P share and the A
    // tile AST - 1 groups ahead, run the products.  Loads complete in order:
    // with AST > 2 the A tile issued after the P share this group waits for
    // (group grp + AST - 2) may still be in flight at the wait.
    static_assert(SA == SA_SAVED, "A tiles hold the stored fp32 A");
    using T = LQXTile<RP>;
    constexpr int AST = T::AST;
    uint8_t* const wt = tiles + wave * AST * T::BYTES;
    const int r_last = r_hi - 1;
    if (ngrp > 0) p_issue(0, 0);
#pragma unroll
    for (int y = 0; y + 1 < AST; ++y)
      if (y < ngrp) lqx_tile_issue<RP>(d, r_lo + LQX_G * y, r_last, cw, wt + y * T::BYTES);
    int st_cur = 0;                         // A stage of group grp
    for (int grp = 0; grp < ngrp; ++grp) {
      const int r0 = r_lo + LQX_G * grp;
      if (AST > 2 && grp > 0 && grp + AST - 2 < ngrp) {
        static_assert(T::NI <= 15, "vmcnt immediate");
        asm volatile("s_waitcnt vmcnt(%0)" :: "n"(T::NI) : "memory");
      } else {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      }
      // A bare barrier: every wave has waited for its own share above and
      // has consumed its earlier LDS reads, and a fence here would wait for
      // the A tile still in flight.
      asm volatile("s_barrier" ::: "memory");
      bf16x8 ah[NU], al[NU];
      float av[8][CPL];
      if constexpr (AST > 2) {
        // The operand reads as inline assembly: the compiler cannot tell that
        // the A tile in flight targets another stage and would wait for it
        // before any LDS read.
        static_assert(NU == 4 && CPL == 1, "assembly reads are written for rank 128");
        const uint32_t pa = (uint32_t)(size_t)(lvoid_t*)(&sm.p[grp & 1][0][so]);
        const uint32_t aa = (uint32_t)(size_t)(lvoid_t*)(wt + st_cur * T::BYTES + g * LQX_SLOT + 4 * li);
        constexpr int PB = RP * LQX_G * 2;   // bytes of one part (hi or lo) of a P stage
        constexpr int UB = 32 * LQX_G * 2;   // bytes of one rank tile of a part
        asm volatile(
            "ds_read_b128 %0, %16 offset:%18\n\t"
            "ds_read_b128 %1, %16 offset:%19\n\t"
            "ds_read_b128 %2, %16 offset:%20\n\t"
            "ds_read_b128 %3, %16 offset:%21\n\t"
            "ds_read_b128 %4, %16 offset:%22\n\t"
            "ds_read_b128 %5, %16 offset:%23\n\t"
            "ds_read_b128 %6, %16 offset:%24\n\t"
            "ds_read_b128 %7, %16 offset:%25\n\t"
            "ds_read_b32 %8, %17 offset:0\n\t"
            "ds_read_b32 %9, %17 offset:128\n\t"
            "ds_read_b32 %10, %17 offset:256\n\t"
            "ds_read_b32 %11, %17 offset:384\n\t"
            "ds_read_b32 %12, %17 offset:512\n\t"
            "ds_read_b32 %13, %17 offset:640\n\t"
            "ds_read_b32 %14, %17 offset:768\n\t"
            "ds_read_b32 %15, %17 offset:896\n\t"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(ah[0]), "=&v"(ah[1]), "=&v"(ah[2]), "=&v"(ah[3]),
              "=&v"(al[0]), "=&v"(al[1]), "=&v"(al[2]), "=&v"(al[3]),
              "=&v"(av[0][0]), "=&v"(av[1][0]), "=&v"(av[2][0]), "=&v"(av[3][0]),
              "=&v"(av[4][0]), "=&v"(av[5][0]), "=&v"(av[6][0]), "=&v"(av[7][0])
            : "v"(pa), "v"(aa), "n"(0), "n"(UB), "n"(2 * UB), "n"(3 * UB),
              "n"(PB), "n"(PB + UB), "n"(PB + 2 * UB), "n"(PB + 3 * UB)
            : "memory");
      } else {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          ah[u] = *(const bf16x8*)(&sm.p[grp & 1][0][32 * u * LQX_G + so]);
          al[u] = *(const bf16x8*)(&sm.p[grp & 1][1][32 * u * LQX_G + so]);
        }
        lqx_tile_read<RP>(wt + st_cur * T::BYTES, li, g, av);
      }
      const int st_new = st_cur == 0 ? AST - 1 : st_cur - 1;   // stage of group grp + AST - 1
      if (grp + 1 < ngrp) p_issue(grp + 1, (grp + 1) & 1);
      if (grp + AST - 1 < ngrp)
        lqx_tile_issue<RP>(d, r0 + LQX_G * (AST - 1), r_last, cw, wt + st_new * T::BYTES);
      st_cur = st_cur + 1 == AST ? 0 : st_cur + 1;
      const int nvalid = r_hi - r0 - 8 * g;   // rows of this lane's half inside the split
#pragma unroll
      for (int x = 0; x < CPL; ++x) {
        bf16x8 bh, bl;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float v = e < nvalid ? av[e][x] : 0.f;
          const __bf16 hv = (__bf16)v;
          bh[e] = hv;
          bl[e] = (__bf16)(v - (float)hv);
        }
        mfma_group(ah, al, x, bh, bl);
      }
    }
  } else {
    RawA<DT, SA, CPL> cur[8], nxt[8];
    if (ngrp > 0) {
      p_issue(0, 0);
      a_fetch(0, cur);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();

    for (int grp = 0; grp < ngrp; ++grp) {
      const bool more = grp + 1 < ngrp;
      // operands of this group first, then the next group's loads
      bf16x8 ah[NU], al[NU];
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        ah[u] = *(const bf16x8*)(&sm.p[grp & 1][0][32 * u * LQX_G + so]);
        al[u] = *(const bf16x8*)(&sm.p[grp & 1][1][32 * u * LQX_G + so]);
      }
      if (more) {
        a_fetch(grp + 1, nxt);
        p_issue(grp + 1, (grp + 1) & 1);
      }
#pragma unroll
      for (int x = 0; x < CPL; ++x) {
        bf16x8 bh, bl;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float v = rawa_val<DT, SA, CPL>(cur[e], x);
          const __bf16 hv = (__bf16)v;
          bh[e] = hv;
          bl[e] = (__bf16)(v - (float)hv);
        }
        mfma_group(ah, al, x, bh, bl);
      }
      // the next group's A and P tile are in before anyone reads them
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      if (more) {
#pragma unroll
        for (int e = 0; e < 8; ++e) cur[e] = nxt[e];
      }
      __syncthreads();
    }
  }

  // acc[x][u][4q + w] = Q[col + x][rank 32u + 8q + 4g + w] (this split)
#pragma unroll
  for (int x = 0; x < CPL; ++x) {
    const int c = col + x;
    if (c < d.n) {
      float* dst = d.qpart + ((int64_t)s * d.n + c) * RP;
#pragma unroll
      for (int u = 0; u < NU; ++u)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *(float4*)(dst + 32 * u + 8 * q + 4 * g) =
              make_float4(acc[x][u][4 * q], acc[x][u][4 * q + 1], acc[x][u][4 * q + 2], acc[x][u][4 * q + 3]);
    }
  }
}

template <int DT, int RP, int SA, bool TILES, bool RM = false>
__global__ __launch_bounds__(lqx_waves(RP) * kWave) void k_lqx(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) LQXSmem<RP> sm;
  __shared__ __attribute__((aligned(16)))
  uint8_t tiles[TILES ? lqx_waves(RP) * LQXTile<RP>::AST * LQXTile<RP>::BYTES : 16];
#define B_(d, b) lqx_body<DT, RP, SA, TILES, RM>(d, b, sm, tiles)
  OCC_DISPATCH_X(K_PASS_Q, B_)
#undef B_
}

// -------------------------------------------------------------------------
// Epilogue of the reconstruction passes (k_ml, k_mlx).  The products leave
// each 32 x 32 tile of M_hat in the 32x32 MFMA layout: lane (g, li) holds
// column li of rows mf32_row(v, g), so stores straight from it cover each
// row in 128-byte pieces of 4-byte accesses.  Each tile goes through LDS
// instead, and each lane then takes 16-byte pieces of rows: the stored A is
// read, and M_hat and err written, with 16-byte accesses when the rows are
// 16-byte aligned (d.vec).  The values are unchanged; only which lane
// stores which element.
// -------------------------------------------------------------------------
constexpr int LE_PITCH = 32 + 4;          // LDS row pitch (floats), 16-byte skew per row
constexpr int LE_RPI = kWave / 8;         // rows per wave instruction (8 lanes x 16 bytes a row)
constexpr int LE_IT = 32 / LE_RPI;        // instructions per 32 x 32 tile

// A (the stored fp32 A, compact rows) for this lane's pieces of the tiles
// of columns cw + 32 c, c < NCT
template <int NCT>
__device__ __forceinline__ void lm_epi_load(const Desc& d, bool vec, int row0, int r_hi, int cw,
                                            f4v (&a4)[NCT][LE_IT]) {
  const int lane = threadIdx.x & 63;
  const int rr = lane >> 3;
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    const int col = cw + 32 * c + 4 * (lane & 7);
#pragma unroll
    for (int it = 0; it < LE_IT; ++it) {
      const int row = row0 + it * LE_RPI + rr;
      const float* src = d.err_out + (int64_t)row * d.lde_out + col;
      f4v v = f4v{0.f, 0.f, 0.f, 0.f};
      if (row < r_hi) {
        if (vec && col + 4 <= d.n) {
          v = *(const f4v*)src;
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (col + j < d.n) v[j] = src[j];
        }
      }
      a4[c][it] = v;
    }
  }
}

// The tiles acc[c][v] = M_hat[row0 + mf32_row(v, g)][cw + 32 c + li], one
// at a time through LDS (ep: this wave's 32 x LE_PITCH floats), then M_hat
// and err = A - M_hat stored by rows, nontemporal.
template <int NCT, bool WM, bool WE, bool OUTBF, bool RM>
__device__ __forceinline__ void lm_epi_store(const Desc& d, bool vec, int row0, int r_hi, int cw,
                                             const f16v (&acc)[NCT], const f4v (&a4)[NCT][LE_IT],
                                             float* ep) {
  typedef float nt4 __attribute__((ext_vector_type(4)));
  typedef uint32_t nu2 __attribute__((ext_vector_type(2)));
  const int lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
  const int rr = lane >> 3, cq = lane & 7;
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
#pragma unroll
    for (int v = 0; v < 16; ++v) ep[mf32_row(v, g) * LE_PITCH + li] = acc[c][v];
    // the tile is written and read by this wave only; LDS keeps a wave's
    // operations in order, and the wait also orders them for the compiler
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    const int col = cw + 32 * c + 4 * cq;
    const bool vec_col = vec && col + 4 <= d.n;
#pragma unroll
    for (int it = 0; it < LE_IT; ++it) {
      const int tr = it * LE_RPI + rr;
      const int row = row0 + tr;
      const f4v mh = *(const f4v*)(ep + tr * LE_PITCH + 4 * cq);
      if (row >= r_hi || col >= d.n) continue;
      const int64_t pr = prow<RM>(d, row);
      float e[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) e[j] = WE ? a4[c][it][j] - mh[j] : 0.f;
      float* eo = RM ? d.err_fin + pr * d.lde_fin + col : d.err_out + pr * d.lde_out + col;
      if (vec_col) {
        if (WM && OUTBF)
          __builtin_nontemporal_store(nu2{bf16_pack2(mh[0], mh[1]), bf16_pack2(mh[2], mh[3])},
                                      (nu2*)((uint16_t*)d.Mhat + pr * d.ldh + col));
        else if (WM)
          __builtin_nontemporal_store(nt4{mh[0], mh[1], mh[2], mh[3]}, (nt4*)(d.Mhat + pr * d.ldh + col));
        if (WE) __builtin_nontemporal_store(nt4{e[0], e[1], e[2], e[3]}, (nt4*)eo);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (col + j < d.n) {
            if (WM) store_mhat1<OUTBF>(d, pr * d.ldh + col + j, mh[j]);
            if (WE) eo[j] = e[j];
          }
        }
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

// The same outputs stored straight from the MFMA layout (4-byte accesses,
// 128-byte pieces of rows), with A read the same way beforehand (av).
// Measured faster than the LDS epilogue at padded rank 32 (two tiles per
// wave) and for the bf16 reconstruction at rank 128.
template <int NCT>
__device__ __forceinline__ void lm_direct_load(const Desc& d, int row0, int cw, float (&av)[NCT][16]) {
  const int lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
#pragma unroll
  for (int c = 0; c < NCT; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = row0 + mf32_row(v, g), col = cw + 32 * c + li;
      av[c][v] = (row < d.m && col < d.n) ? d.err_out[(int64_t)row * d.lde_out + col] : 0.f;
    }
}

template <int NCT, bool WM, bool WE, bool OUTBF, bool RM>
__device__ __forceinline__ void lm_direct_store(const Desc& d, int row0, int r_hi, int cw,
                                                const f16v (&acc)[NCT], const float (&av)[NCT][16]) {
  const int lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    const int col = cw + 32 * c + li;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = row0 + mf32_row(v, g);
      if (row < r_hi && col < d.n) {
        const float mh = acc[c][v];
        const int64_t pr = prow<RM>(d, row);
        if (WM) {
          if constexpr (OUTBF) __builtin_nontemporal_store(bf16_rne(mh), (uint16_t*)d.Mhat + pr * d.ldh + col);
          else __builtin_nontemporal_store(mh, d.Mhat + pr * d.ldh + col);
        }
        if (WE)
          __builtin_nontemporal_store(av[c][v] - mh, RM ? d.err_fin + pr * d.lde_fin + col
                                                        : d.err_out + pr * d.lde_out + col);
      }
    }
  }
}

// -------------------------------------------------------------------------
// k_ml: M_hat = P_hat Q^T, err = A - M_hat for one column tile and d.mr rows.
// SRC 0: P_hat from phat_t, Q from qpad (fused step).  SRC 1: the caller's P
// (m x r) and Q (n x r), zero past rank r (stand-alone decompression; the
// same products, so both give bitwise the same M_hat).
// -------------------------------------------------------------------------
template <int RP>
struct LMSmem {
  float p[2][RP][32];   // P_hat tile, transposed: [rank][row]
  float ep[lm_lds_epilogue(RP) ? kBlock / kWave : 0][32 * LE_PITCH];   // epilogue tile per wave
};

template <int RP, int SRC>
__device__ __forceinline__ void lm_stage_direct(const Desc& d, int row0, float (*dst)[32]) {
  for (int idx = threadIdx.x; idx < RP * 32; idx += kBlock) {
    const int k = idx >> 5, i = idx & 31;
    const int row = row0 + i;
    dst[k][i] = (row < d.m && k < d.r) ? d.P[(int64_t)row * d.r + k] : 0.f;
  }
}

template <int DT, int RP, int SA, int SRC, bool WM, bool WE, bool OUTBF = false, bool RM = false>
__device__ __forceinline__ void lm_body(const Desc& d, int b, LMSmem<RP>& sm) {
  static_assert(!WE || SA == SA_SAVED, "the residual is formed from the stored A");
  constexpr int NCT = lm_tiles(RP), KP = RP / 2, BC = lm_block_cols(RP);
  constexpr bool EPI = lm_lds_epilogue(RP);
  const bool vec = d.vec != 0;
  constexpr int SF = RP * 8 / kBlock;   // float4s per thread per P_hat tile
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
  const int t = threadIdx.x;
  const int col_tiles = (d.n + BC - 1) / BC;
  const int ct = b % col_tiles, rb = b / col_tiles;
  const int r_lo = rb * d.mr, r_hi = min(d.m, r_lo + d.mr);
  const int ntile = (r_hi - r_lo + 31) / 32;
  const int cw = ct * BC + wave * 32 * NCT;

  float qv[NCT][KP];
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    const int col = cw + 32 * c + li;
#pragma unroll
    for (int kp = 0; kp < KP; ++kp) {
      const int k = 2 * kp + g;
      float v = 0.f;
      if (SRC == 0) {
        if (col < d.n_pad) v = d.qpad[(int64_t)col * RP + k];
      } else {
        if (col < d.n && k < d.r) v = d.Q[(int64_t)col * d.r + k];
      }
      qv[c][kp] = v;
    }
  }

  f4v pr[SF > 0 ? SF : 1];
  if (SRC == 0) {
#pragma unroll
    for (int x = 0; x < SF; ++x) {
      const int f = t + kBlock * x, k = f >> 3, part = f & 7;
      pr[x] = *(const f4v*)(d.phat_t + (int64_t)k * d.m_pad + r_lo + 4 * part);
      *(f4v*)(&sm.p[0][k][4 * part]) = pr[x];
    }
  } else {
    lm_stage_direct<RP, SRC>(d, r_lo, sm.p[0]);
  }
  __syncthreads();

  for (int tile = 0; tile < ntile; ++tile) {
    const int row0 = r_lo + 32 * tile;
    const bool more = tile + 1 < ntile;
    if (SRC == 0 && more) {
#pragma unroll
      for (int x = 0; x < SF; ++x) {
        const int f = t + kBlock * x, k = f >> 3, part = f & 7;
        pr[x] = *(const f4v*)(d.phat_t + (int64_t)k * d.m_pad + row0 + 32 + 4 * part);
      }
    }
    // A for this tile's outputs (issued before the products to hide latency)
    f4v a4[EPI ? NCT : 1][LE_IT];
    float av[EPI ? 1 : NCT][16];
    if (WE) {
      if constexpr (EPI) lm_epi_load<NCT>(d, vec, row0, r_hi, cw, a4);
      else lm_direct_load<NCT>(d, row0, cw, av);
    }
    f16v acc[NCT];
#pragma unroll
    for (int c = 0; c < NCT; ++c) acc[c] = f16v{};
    const float* pa = &sm.p[tile & 1][g][li];
#pragma unroll
    for (int kp = 0; kp < KP; ++kp) {
      const float a = pa[2 * kp * 32];
#pragma unroll
      for (int c = 0; c < NCT; ++c) acc[c] = mfma32(a, qv[c][kp], acc[c]);
    }
    if constexpr (EPI) lm_epi_store<NCT, WM, WE, OUTBF, RM>(d, vec, row0, r_hi, cw, acc, a4, sm.ep[wave]);
    else lm_direct_store<NCT, WM, WE, OUTBF, RM>(d, row0, r_hi, cw, acc, av);
    if (more) {
      if (SRC == 0) {
#pragma unroll
        for (int x = 0; x < SF; ++x) {
          const int f = t + kBlock * x, k = f >> 3, part = f & 7;
          *(f4v*)(&sm.p[(tile + 1) & 1][k][4 * part]) = pr[x];
        }
      } else {
        lm_stage_direct<RP, SRC>(d, row0 + 32, sm.p[(tile + 1) & 1]);
      }
    }
    __syncthreads();
  }
}

template <int DT, int RP, int SA, int SRC, bool WM, bool WE, bool OUTBF = false, bool RM = false>
__global__ __launch_bounds__(kBlock) void k_ml(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) LMSmem<RP> sm;
#define B_(d, b) lm_body<DT, RP, SA, SRC, WM, WE, OUTBF, RM>(d, b, sm)
  OCC_DISPATCH_X(K_MHAT, B_)
#undef B_
}

// -------------------------------------------------------------------------
// k_mlx: the reconstruction pass for bf16 M on the bf16 matrix cores with
// split operands (as the products of k_lp X3): M_hat = P_hat Q^T accumulated
// in fp32 as P_hi Q_hi + P_hi Q_lo + P_lo Q_hi on v_mfma_f32_32x32x16_bf16,
// 16 ranks per K-step s, with
//   A operand  P_hat: lane (g, li) supplies row li of the 32-row tile, ranks
//              16 s + 8 g .. + 7, from an LDS tile of bf16 hi/lo rows staged
//              from P_hat (SRC 0: the workspace copy; SRC 1: the caller's P,
//              zero past rank r);
//   B operand  Q^T: lane (g, li) supplies the same ranks of its column
//              cw + 32 c + li, split once into bf16 hi/lo registers;
// so acc[c][v] = M_hat[row0 + mf32_row(v, g)][cw + 32 c + li], the layout of
// k_ml, and err = A - M_hat is formed and stored straight from it.  Rounding both
// factors to two bf16 parts leaves about 2^-16 of |M_hat| per element, far
// inside bf16 input precision; at rank 128 the pass needs 3/16 of the
// matrix-core cycles of the fp32 form and is bound by memory instead.
// -------------------------------------------------------------------------
template <int RP>
struct LMXSmem {
  uint16_t p[2][2][32 * (RP + 8)];   // [stage][hi, lo][row][rank], pitch RP + 8
};

template <int RP, int SRC>
__device__ __forceinline__ void lmx_fetch(const Desc& d, int row0, f4v* pr) {
  constexpr int SF = RP * 8 / kBlock;   // float4s of a 32 x RP tile per thread
#pragma unroll
  for (int x = 0; x < SF; ++x) {
    const int f = threadIdx.x + kBlock * x;
    const int i = f / (RP / 4), k = 4 * (f % (RP / 4));
    const int row = row0 + i;
    f4v v = f4v{0.f, 0.f, 0.f, 0.f};
    if (row < d.m) {
      if (SRC == 0) {
        v = *(const f4v*)(d.phat + (int64_t)row * RP + k);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (k + e < d.r) v[e] = d.P[(int64_t)row * d.r + k + e];
      }
    }
    pr[x] = v;
  }
}

template <int RP>
__device__ __forceinline__ void lmx_stage(const f4v* pr, uint16_t (*dst)[32 * (RP + 8)]) {
  constexpr int SF = RP * 8 / kBlock;
#pragma unroll
  for (int x = 0; x < SF; ++x) {
    const int f = threadIdx.x + kBlock * x;
    const int i = f / (RP / 4), k = 4 * (f % (RP / 4));
    uint16_t hi[4], lo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const __bf16 h = (__bf16)pr[x][e];
      hi[e] = bf16_bits(h);
      lo[e] = bf16_bits((__bf16)(pr[x][e] - (float)h));
    }
    const int off = i * (RP + 8) + k;
    *(uint2*)(&dst[0][off]) = make_uint2(hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16));
    *(uint2*)(&dst[1][off]) = make_uint2(lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16));
  }
}

template <int RP, int SRC, bool WM, bool WE, bool OUTBF = false, bool RM = false>
__device__ __forceinline__ void lmx_body(const Desc& d, int b, LMXSmem<RP>& sm) {
  constexpr int NCT = lm_tiles(RP), KS = RP / 16, BC = lm_block_cols(RP);
  constexpr int SF = RP * 8 / kBlock;
  constexpr int PT = RP + 8;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int li = lane & 31, g = lane >> 5;
  const int col_tiles = (d.n + BC - 1) / BC;
  const int ct = b % col_tiles, rb = b / col_tiles;
  const int r_lo = rb * d.mr, r_hi = min(d.m, r_lo + d.mr);
  const int ntile = (r_hi - r_lo + 31) / 32;
  const int cw = ct * BC + wave * 32 * NCT;

  // Q^T operands: ranks 16 s + 8 g .. + 7 of column cw + 32 c + li
  bf16x8 bh[NCT][KS], bl[NCT][KS];
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    const int col = cw + 32 * c + li;
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = 16 * s2 + 8 * g + e;
        float v = 0.f;
        if (SRC == 0) {
          if (col < d.n_pad) v = d.qpad[(int64_t)col * RP + k];
        } else {
          if (col < d.n && k < d.r) v = d.Q[(int64_t)col * d.r + k];
        }
        const __bf16 h = (__bf16)v;
        bh[c][s2][e] = h;
        bl[c][s2][e] = (__bf16)(v - (float)h);
      }
    }
  }

  f4v pr[SF];
  lmx_fetch<RP, SRC>(d, r_lo, pr);
  lmx_stage<RP>(pr, sm.p[0]);
  __syncthreads();

  for (int tile = 0; tile < ntile; ++tile) {
    const int row0 = r_lo + 32 * tile;
    const bool more = tile + 1 < ntile;
    if (more) lmx_fetch<RP, SRC>(d, row0 + 32, pr);
    // A for this tile's outputs (issued before the products to hide latency)
    float av[NCT][16];
    if (WE) lm_direct_load<NCT>(d, row0, cw, av);
    f16v acc[NCT];
#pragma unroll
    for (int c = 0; c < NCT; ++c) acc[c] = f16v{};
    const uint16_t* ph = &sm.p[tile & 1][0][li * PT + 8 * g];
    const uint16_t* pl = &sm.p[tile & 1][1][li * PT + 8 * g];
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      const bf16x8 ah = *(const bf16x8*)(ph + 16 * s2);
      const bf16x8 al = *(const bf16x8*)(pl + 16 * s2);
#pragma unroll
      for (int c = 0; c < NCT; ++c) {
        acc[c] = mfma32bf(ah, bh[c][s2], acc[c]);
        acc[c] = mfma32bf(ah, bl[c][s2], acc[c]);
        acc[c] = mfma32bf(al, bh[c][s2], acc[c]);
      }
    }
    lm_direct_store<NCT, WM, WE, OUTBF, RM>(d, row0, r_hi, cw, acc, av);
    if (more) lmx_stage<RP>(pr, sm.p[(tile + 1) & 1]);
    __syncthreads();
  }
}

template <int RP, int SRC, bool WM, bool WE, bool OUTBF = false, bool RM = false>
__global__ __launch_bounds__(kBlock) void k_mlx(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) LMXSmem<RP> sm;
#define B_(d, b) lmx_body<RP, SRC, WM, WE, OUTBF, RM>(d, b, sm)
  OCC_DISPATCH_X(K_MHAT, B_)
#undef B_
}

}  // namespace occ
