// HIP kernels of liboptcc for gfx950 (CDNA4): shared helpers and the small
// kernels common to both rank paths (Q padding, Gram-partial sums, Q
// reduction, stand-alone reconstruction and error update).
//
// Streaming kernels read the error-fed input A = M + err_prev straight from
// HBM (M as bf16 or fp32, err_prev fp32).  Sums run in a fixed order, so
// every result is deterministic and the fused and unfused entry points agree
// bitwise.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.hpp"

namespace occ {

typedef const __attribute__((address_space(4))) float* cfloat_p;
typedef const __attribute__((address_space(4))) double* cdouble_p;

__device__ __forceinline__ cfloat_p as_const(const float* p) { return (cfloat_p)(uintptr_t)p; }
__device__ __forceinline__ cdouble_p as_const(const double* p) { return (cdouble_p)(uintptr_t)p; }

enum { DT_F32 = 0, DT_BF16 = 1 };
enum : uint32_t { FLAG_NONFINITE = 1u, FLAG_RANK_DEFICIENT = 2u, FLAG_BAD_ROWS = 4u };

// Index of this thread's wave in its block, as a wave-uniform (SGPR) value so
// that addresses derived from it qualify for scalar loads.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// bf16 bit pattern of an fp32 value, rounded to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t bf16_rne(float v) {
  return __builtin_bit_cast(uint16_t, (__bf16)v);
}

__device__ __forceinline__ uint32_t bf16_pack2(float lo, float hi) {
  return (uint32_t)bf16_rne(lo) | ((uint32_t)bf16_rne(hi) << 16);
}

// One element of M_hat at offset `off` (elements): fp32, or bf16 when OUTBF.
template <bool OUTBF, class D>
__device__ __forceinline__ void store_mhat1(const D& d, int64_t off, float v) {
  if constexpr (OUTBF) ((uint16_t*)d.Mhat)[off] = bf16_rne(v);
  else d.Mhat[off] = v;
}

// Element (row, col) of M as fp32 (exact widening for bf16).
template <int DT>
__device__ __forceinline__ float m_elem(const Desc& d, int64_t off) {
  if (DT == DT_F32) return ((const float*)d.M)[off];
  const uint16_t h = ((const uint16_t*)d.M)[off];
  return __uint_as_float((uint32_t)h << 16);
}

// Row of M, err and M_hat that holds row `row` (< d.m) of the compressed
// matrix: the same row, or with RM (row-sparse step) the row the validated
// row list names.
template <bool RM>
__device__ __forceinline__ int64_t prow(const Desc& d, int row) {
  if constexpr (RM) return (int64_t)d.rmap[row];
  else return (int64_t)row;
}

// A[row, col..col+3] = M + err_prev for columns < c_hi (zero beyond, and for
// rows >= m).  VEC requires 16-byte aligned fp32 rows (8-byte for bf16 M),
// i.e. aligned bases, ld % 4 == 0 and col % 4 == 0.
template <int DT, bool VEC, bool RM = false>
__device__ __forceinline__ void load_a4(const Desc& d, int row, int col, int c_hi, float a[4]) {
  a[0] = a[1] = a[2] = a[3] = 0.f;
  if (row >= d.m || col >= c_hi) return;
  const int64_t pr = prow<RM>(d, row);
  const int64_t mo = pr * d.ldm + col;
  const int64_t eo = pr * d.lde_in + col;
  if (VEC && col + 4 <= c_hi) {
    if (DT == DT_F32) {
      const float4 v = *(const float4*)((const float*)d.M + mo);
      a[0] = v.x; a[1] = v.y; a[2] = v.z; a[3] = v.w;
    } else {
      const uint2 v = *(const uint2*)((const uint16_t*)d.M + mo);
      a[0] = bf16_lo(v.x); a[1] = bf16_hi(v.x); a[2] = bf16_lo(v.y); a[3] = bf16_hi(v.y);
    }
    if (d.err_in) {
      const float4 e = *(const float4*)(d.err_in + eo);
      a[0] = a[0] + e.x; a[1] = a[1] + e.y; a[2] = a[2] + e.z; a[3] = a[3] + e.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (col + j < c_hi) {
        float v = m_elem<DT>(d, mo + j);
        if (d.err_in) v = v + d.err_in[eo + j];
        a[j] = v;
      }
    }
  }
}

// Single element of A (column bound n).
template <int DT>
__device__ __forceinline__ float load_a1(const Desc& d, int row, int col) {
  if (row >= d.m || col >= d.n) return 0.f;
  float v = m_elem<DT>(d, (int64_t)row * d.ldm + col);
  if (d.err_in) v = v + d.err_in[(int64_t)row * d.lde_in + col];
  return v;
}

// Block -> matrix lookup for batched launches: the last matrix whose first
// block of this kernel kind is <= b.
__device__ __forceinline__ int find_matrix(const Desc* __restrict__ table, int count, int kind,
                                           int b) {
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (table[mid].blk[kind] <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Dispatch helpers: run BODY(d, local_block) on the matrix owning block B
// of kind KIND (this block, for OCC_DISPATCH).
#define OCC_DISPATCH_AT(KIND, BODY, B)                                  \
  if (count == 1) {                                                     \
    BODY(single, (B));                                                  \
  } else {                                                              \
    const int j_ = find_matrix(table, count, KIND, (B));                \
    const Desc& d_ = table[j_];                                         \
    BODY(d_, (B) - d_.blk[KIND]);                                       \
  }

#define OCC_DISPATCH(KIND, BODY) OCC_DISPATCH_AT(KIND, BODY, (int)blockIdx.x)

#define OCC_KARGS const Desc* __restrict__ table, int count, Desc single

// Tile index of a block of a kernel whose neighbouring tiles share an operand
// slice (the Q columns of a left-product split, the P_hat rows of a
// right-product split or reconstruction row block).  Workgroups are dealt to
// the 8 XCDs round-robin (workgroup b to XCD b % 8), each XCD with its own L2;
// renumbering so that XCD x takes the contiguous tile range
// [x G8 / 8, (x + 1) G8 / 8) (G8 = the grid rounded down to a multiple of 8;
// the last G - G8 blocks keep their index) keeps the tiles that run on one
// XCD on few slices.  A bijection of [0, G): results do not change.
__device__ __forceinline__ int xcd_tile() {
  const int g8 = (int)gridDim.x & ~7, b = (int)blockIdx.x;
  return b < g8 ? (b & 7) * (g8 >> 3) + (b >> 3) : b;
}

#define OCC_DISPATCH_X(KIND, BODY)                                      \
  if (count == 1) {                                                     \
    BODY(single, xcd_tile());                                           \
  } else {                                                              \
    const int v_ = xcd_tile();                                          \
    const int j_ = find_matrix(table, count, KIND, v_);                 \
    const Desc& d_ = table[j_];                                         \
    BODY(d_, v_ - d_.blk[KIND]);                                        \
  }

// ---------------------------------------------------------------------------
// Warm-start Q -> padded layout qpad[n_pad][rp] (zeros beyond n and rank).
// ---------------------------------------------------------------------------
template <int RP>
__device__ __forceinline__ void qpad_body(const Desc& d, int b) {
  const int64_t idx = (int64_t)b * kBlock + threadIdx.x;
  if (idx >= (int64_t)d.n_pad * RP) return;
  const int c = (int)(idx / RP), k = (int)(idx % RP);
  d.qpad[idx] = (c < d.n && k < d.r) ? d.Q[(int64_t)c * d.r + k] : 0.f;
}

template <int RP>
__global__ __launch_bounds__(kBlock) void k_qpad(OCC_KARGS) {
#define B_(d, b) qpad_body<RP>(d, b)
  OCC_DISPATCH(K_QPAD, B_)
#undef B_
}

// gsum[k][l] = sum_b gpart[b][k][l] for k <= l (fixed order), zero below the
// diagonal (the Gram partials hold the upper triangle only).  MODE 1: second
// CholeskyQR pass, skipped unless the first pass asked for it.  A block
// takes GS_ENT entries; GS_SL threads per entry sum interleaved slices of
// the partials with their loads issued in batches of 8, and the slices are
// added in slice order.
constexpr int GS_SL = 8;
constexpr int GS_ENT = kBlock / GS_SL;

template <int RP, int MODE>
__device__ __forceinline__ void gsum_body(const Desc& d, int b) {
  if (MODE == 1 && !d.info[0]) return;
  __shared__ double part[GS_SL][GS_ENT];
  const int sl = threadIdx.x / GS_ENT, el = threadIdx.x % GS_ENT;
  const int idx = b * GS_ENT + el;
  const int k = idx / RP, l = idx % RP;
  const bool upper = idx < RP * RP && k <= l;
  double s = 0.0;
  if (upper) {
    for (int g0 = sl; g0 < d.ng; g0 += 8 * GS_SL) {
      double v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int g = g0 + GS_SL * u;
        v[u] = (g < d.ng) ? d.gpart[(int64_t)g * RP * RP + idx] : 0.0;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (g0 + GS_SL * u < d.ng) s = (g0 + GS_SL * u == sl) ? v[u] : s + v[u];
    }
  }
  part[sl][el] = s;
  __syncthreads();
  if (sl == 0 && idx < RP * RP) {
    double tot = 0.0;
    if (upper) {
      tot = part[0][el];
      for (int x = 1; x < GS_SL && x < d.ng; ++x) tot += part[x][el];
    }
    d.gsum[idx] = tot;
  }
}

template <int RP, int MODE>
__global__ __launch_bounds__(kBlock) void k_gsum(OCC_KARGS) {
#define B_(d, b) gsum_body<RP, MODE>(d, b)
  OCC_DISPATCH(K_GSUM, B_)
#undef B_
}

// ---------------------------------------------------------------------------
// Pivot rules shared by the Cholesky kernels: a pivot <= kPivotTol * max diag(G)
// marks its column dependent; a second CholeskyQR pass runs when the
// surviving diagonal of the Cholesky factor spans more than kSecondPassCond.
// ---------------------------------------------------------------------------
constexpr double kPivotTol = 1e-12;
constexpr double kSecondPassCond = 1e3;

// ---------------------------------------------------------------------------
// Large-rank path: Q padding (k_qpadl) and the Q reduction (k_qredl) over
// column tiles.  Both write qpad (n_pad x RP) and, when M is bf16, Q as
// two bf16 parts hi = bf16(v), lo = bf16(v - hi) (v - hi - lo is below
// 2^-16 |v|) in qbf, transposed so that the left product stages 32 columns
// of a rank row with 16-byte copies: rank k goes to row (k % NU) * 32 + k / NU,
// NU = RP / 32, the order in which that kernel's lanes read them.  The
// transpose goes through LDS, so each qbf row is written in 16-byte chunks.
// k_qpadl covers all n_pad columns (zeros past n) in 32-column tiles;
// k_qredl sums the row-split partials (fixed order, 16 loads in flight per
// element) for the n real columns, in tiles of d.qr_cols columns (8 or 32),
// and also writes the caller's Q.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint16_t bf16_bits(__bf16 h) { return __builtin_bit_cast(uint16_t, h); }

constexpr int QT_COLS = 32;                 // columns per block, at most

template <int RP>
struct QTSmem {
  uint16_t t[2][RP * QT_COLS];
};

template <int RP, bool REDUCE>
__device__ __forceinline__ void qtile_body(const Desc& d, int b, QTSmem<RP>& sm) {
  constexpr int NU = RP / 32;
  const int QT_P = REDUCE ? d.qr_cols : QT_COLS;   // columns of this tile = LDS pitch (bf16)
  const int QT_CH = QT_P / 8;                      // 16-byte chunks of a transposed rank row
  const int c0 = b * QT_P;
  const int c_end = REDUCE ? d.n : d.n_pad;
  for (int e = threadIdx.x; e < QT_P * RP; e += kBlock) {
    const int c = c0 + e / RP, k = e % RP;
    if (c >= c_end) continue;
    const int64_t idx = (int64_t)c * RP + k;
    float v;
    if (REDUCE) {
      // fixed order; loads issued in batches of 16
      v = 0.f;
      for (int s0 = 0; s0 < d.sq; s0 += 16) {
        float p[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) p[u] = (s0 + u < d.sq) ? d.qpart[(int64_t)(s0 + u) * d.n * RP + idx] : 0.f;
#pragma unroll
        for (int u = 0; u < 16; ++u)
          if (s0 + u < d.sq) v = (s0 + u == 0) ? p[u] : v + p[u];
      }
      if (k < d.r) d.Q[(int64_t)c * d.r + k] = v;
    } else {
      v = (c < d.n && k < d.r) ? d.Q[(int64_t)c * d.r + k] : 0.f;
    }
    d.qpad[idx] = v;
    if (d.qbf) {
      const int prow = (k % NU) * 32 + k / NU;
      const __bf16 hi = (__bf16)v;
      sm.t[0][prow * QT_P + (c - c0)] = bf16_bits(hi);
      sm.t[1][prow * QT_P + (c - c0)] = bf16_bits((__bf16)(v - (float)hi));
    }
  }
  if (!d.qbf) return;
  __syncthreads();
  // 2 x RP rows of QT_COLS columns, QT_CH 16-byte chunks each
  for (int f = threadIdx.x; f < 2 * RP * QT_CH; f += kBlock) {
    const int h = f / (RP * QT_CH), prow = (f / QT_CH) % RP, part = f % QT_CH;
    const int c = c0 + 8 * part;
    if (c >= c_end) continue;
    if (c + 8 <= c_end) {
      *(uint4*)(d.qbf + ((int64_t)h * RP + prow) * d.n_pad + c) = *(const uint4*)(&sm.t[h][prow * QT_P + 8 * part]);
    } else {
      for (int j = 0; j < 8 && c + j < c_end; ++j)
        d.qbf[((int64_t)h * RP + prow) * d.n_pad + c + j] = sm.t[h][prow * QT_P + 8 * part + j];
    }
  }
}

template <int RP>
__global__ __launch_bounds__(kBlock) void k_qpadl(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) QTSmem<RP> sm;
#define B_(d, b) qtile_body<RP, false>(d, b, sm)
  OCC_DISPATCH(K_QPAD, B_)
#undef B_
}

template <int RP>
__global__ __launch_bounds__(kBlock) void k_qredl(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) QTSmem<RP> sm;
#define B_(d, b) qtile_body<RP, true>(d, b, sm)
  OCC_DISPATCH(K_QRED, B_)
#undef B_
}

// ---------------------------------------------------------------------------
// Stand-alone error update: err_new = (M + err_prev) - M_hat, elementwise,
// same operation order as the fused pass.
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(kBlock) void k_err_update(Desc d) {
  const int64_t total = (int64_t)d.m * d.n;
  for (int64_t idx = (int64_t)blockIdx.x * kBlock + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * kBlock) {
    const int i = (int)(idx / d.n), c = (int)(idx % d.n);
    const float a = load_a1<DT>(d, i, c);
    const float mh = d.Mhat[(int64_t)i * d.ldh + c];
    d.err_out[(int64_t)i * d.lde_out + c] = a - mh;
  }
}

// Copy descriptor chunks passed by value into the workspace table (12
// descriptors, 3.3 KB of kernel arguments per launch).
constexpr int kTableChunk = 12;
struct TableChunk {
  Desc d[kTableChunk];
};

__global__ void k_write_table(Desc* dst, TableChunk src, int n) {
  const int words = (int)(sizeof(Desc) / 4) * n;
  const uint32_t* s = (const uint32_t*)&src;
  uint32_t* o = (uint32_t*)dst;
  for (int w = threadIdx.x; w < words; w += blockDim.x) o[w] = s[w];
}

__global__ void k_zero_words(uint32_t* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0u;
}

// Row list of the row-sparse step: rows[0 .. n) copied to dst, each index
// clamped into [0, m_rows) so that no kernel can address outside M, err or
// M_hat; an index out of range, or not larger than the one before it (the
// list must be strictly increasing), raises FLAG_BAD_ROWS.  The streaming
// kernels read the row map from the copy only.
__global__ __launch_bounds__(kBlock) void k_rows_check(const int32_t* rows, int64_t n,
                                                       int32_t m_rows, int32_t* dst,
                                                       uint32_t* flags) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kBlock) {
    const int32_t v = rows[i];
    bad = bad || v < 0 || v >= m_rows || (i > 0 && v <= rows[i - 1]);
    dst[i] = v < 0 ? 0 : (v >= m_rows ? m_rows - 1 : v);
  }
  if (bad) atomicOr(flags, FLAG_BAD_ROWS);
}

// Row-sparse step with an empty row list: A is zero, so P_hat = 0 and
// Q = A^T P_hat = 0 (the dense step on an all-zero matrix gives the same and
// flags the rank deficiency).
__global__ __launch_bounds__(kBlock) void k_rows_empty(float* Q, int64_t n, uint32_t* flags) {
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kBlock)
    Q[i] = 0.f;
  if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(flags, FLAG_RANK_DEFICIENT);
}

}  // namespace occ
