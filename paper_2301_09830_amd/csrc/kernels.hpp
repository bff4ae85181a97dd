// HIP kernels of liboptcc for gfx950 (CDNA4), vector-ALU path.
//
// Every streaming kernel reads the error-fed input A = M + err_prev straight
// from HBM (M as bf16 or fp32, err_prev fp32) and never materialises A.
// Products use explicit fmaf in a fixed order, so every result is
// deterministic and the fused and unfused entry points agree bitwise.
//
// Operands that are the same for every lane of a wave (rows of Q in the left
// product, rows of P_hat in the right product and in the reconstruction) are
// read through the constant address space, which the compiler turns into
// scalar loads: the value sits in an SGPR and feeds v_fmac directly, so the
// small-rank products need no cross-lane reduction and no LDS traffic for
// the factor.
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
enum : uint32_t { FLAG_NONFINITE = 1u, FLAG_RANK_DEFICIENT = 2u };

// Index of this thread's wave in its block, as a wave-uniform (SGPR) value so
// that addresses derived from it qualify for scalar loads.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Element (row, col) of M as fp32 (exact widening for bf16).
template <int DT>
__device__ __forceinline__ float m_elem(const Desc& d, int64_t off) {
  if (DT == DT_F32) return ((const float*)d.M)[off];
  const uint16_t h = ((const uint16_t*)d.M)[off];
  return __uint_as_float((uint32_t)h << 16);
}

// A[row, col..col+3] = M + err_prev for columns < c_hi (zero beyond, and for
// rows >= m).  VEC requires 16-byte aligned fp32 rows (8-byte for bf16 M),
// i.e. aligned bases, ld % 4 == 0 and col % 4 == 0.
template <int DT, bool VEC>
__device__ __forceinline__ void load_a4(const Desc& d, int row, int col, int c_hi, float a[4]) {
  a[0] = a[1] = a[2] = a[3] = 0.f;
  if (row >= d.m || col >= c_hi) return;
  const int64_t mo = (int64_t)row * d.ldm + col;
  const int64_t eo = (int64_t)row * d.lde_in + col;
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

// Dispatch helper: runs BODY(d, local_block) on the matrix owning this block.
#define OCC_DISPATCH(KIND, BODY)                                        \
  if (count == 1) {                                                     \
    BODY(single, (int)blockIdx.x);                                      \
  } else {                                                              \
    const int j_ = find_matrix(table, count, KIND, (int)blockIdx.x);    \
    const Desc& d_ = table[j_];                                         \
    BODY(d_, (int)blockIdx.x - d_.blk[KIND]);                           \
  }

#define OCC_KARGS const Desc* __restrict__ table, int count, Desc single

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

// ---------------------------------------------------------------------------
// Left product, split over columns: ppart[s][i][k] = sum_{c in split s} A[i,c] Q[c,k].
// A block owns 64 rows; each wave takes 32-column sub-tiles in turn, stages
// the 64x32 tile of A through LDS so that each lane holds one row, and
// accumulates its row of P with Q rows broadcast from SGPRs.
// ---------------------------------------------------------------------------
template <int DT, bool VEC, int RP>
__device__ __forceinline__ void pass_p_body(const Desc& d, int b, float* lds) {
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int row_tiles = (d.m + PP_ROWS - 1) / PP_ROWS;
  const int tile = b % row_tiles, split = b / row_tiles;
  const int row0 = tile * PP_ROWS;
  const int c_lo = split * d.p_cols;
  const int c_hi = min(d.n, c_lo + d.p_cols);
  const int nsub = (c_hi - c_lo + PP_SUB - 1) / PP_SUB;
  const int rounds = (nsub + 3) / 4;
  float* my = lds + wave * (PP_ROWS * PP_PITCH);
  const int lr = lane >> 3, lc = (lane & 7) * 4;

  float acc[RP];
#pragma unroll
  for (int k = 0; k < RP; ++k) acc[k] = 0.f;

  for (int rd = 0; rd < rounds; ++rd) {
    const int sub = rd * 4 + wave;
    const int col0 = c_lo + sub * PP_SUB;
    const bool active = sub < nsub;
    if (active) {
#pragma unroll
      for (int it = 0; it < PP_ROWS / 8; ++it) {
        const int r = it * 8 + lr;
        float a[4];
        load_a4<DT, VEC>(d, row0 + r, col0 + lc, c_hi, a);
        *(float4*)(my + r * PP_PITCH + lc) = make_float4(a[0], a[1], a[2], a[3]);
      }
    }
    __syncthreads();
    if (active) {
      float a[PP_SUB];
#pragma unroll
      for (int j = 0; j < PP_SUB / 4; ++j) {
        const float4 v = *(const float4*)(my + lane * PP_PITCH + 4 * j);
        a[4 * j] = v.x; a[4 * j + 1] = v.y; a[4 * j + 2] = v.z; a[4 * j + 3] = v.w;
      }
      // qpad has n_pad (multiple of 32) zero-padded rows, so the whole
      // sub-tile is in bounds; columns past c_hi carry a == 0.
      const cfloat_p q = as_const(d.qpad) + (int64_t)col0 * RP;
#pragma unroll
      for (int c = 0; c < PP_SUB; ++c) {
#pragma unroll
        for (int k = 0; k < RP; ++k) acc[k] = fmaf(a[c], q[c * RP + k], acc[k]);
      }
    }
    __syncthreads();
  }

  // Sum the four waves' partial rows (fixed order) and store the split.
  constexpr int CH = RP < 16 ? RP : 16;
#pragma unroll
  for (int kc = 0; kc < RP; kc += CH) {
#pragma unroll
    for (int k = 0; k < CH; ++k) lds[(wave * 64 + lane) * (CH + 1) + k] = acc[kc + k];
    __syncthreads();
    if (wave == 0 && row0 + lane < d.m) {
      float* dst = d.ppart + ((int64_t)split * d.m + row0 + lane) * RP + kc;
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        float s = lds[lane * (CH + 1) + k];
        s = s + lds[(64 + lane) * (CH + 1) + k];
        s = s + lds[(128 + lane) * (CH + 1) + k];
        s = s + lds[(192 + lane) * (CH + 1) + k];
        dst[k] = s;
      }
    }
    __syncthreads();
  }
}

template <int DT, bool VEC, int RP>
__global__ __launch_bounds__(kBlock) void k_pass_p(OCC_KARGS) {
  __shared__ __attribute__((aligned(16))) float lds[4 * PP_ROWS * PP_PITCH];
#define B_(d, b) pass_p_body<DT, VEC, RP>(d, b, lds)
  OCC_DISPATCH(K_PASS_P, B_)
#undef B_
}

// ---------------------------------------------------------------------------
// Gram partials in fp64.  Mode 0 (first CholeskyQR pass): P = sum of the
// column-split partials, stored to praw (fp32); Gram of P.  Mode 1 (second
// pass): rows of P T1 computed in fp64 from praw; Gram of those.
// Rows of a G_ROWS block are staged 64 at a time in LDS as doubles; thread
// work items are 4x4 tiles of the upper triangle, replicated over row groups.
// ---------------------------------------------------------------------------
template <int RP>
struct GramShape {
  static constexpr int NB = RP / 4;                      // 4-wide blocks per side
  static constexpr int NUP = NB * (NB + 1) / 2;          // upper-triangular tiles
  static constexpr int GROUPS = NUP >= kBlock ? 1 : kBlock / NUP;
  static constexpr int TPT = (NUP + kBlock - 1) / kBlock;  // tiles per thread (GROUPS == 1)
};

__device__ __forceinline__ void tile_coords(int p, int nb, int& kb, int& lb) {
  // p-th tile of the upper triangle in row-major order (kb <= lb)
  kb = 0;
  int rem = p;
  while (rem >= nb - kb) { rem -= nb - kb; ++kb; }
  lb = kb + rem;
}

template <int RP, int MODE>
__device__ __forceinline__ void gram_body(const Desc& d, int b, double* lds) {
  using S = GramShape<RP>;
  const int t = threadIdx.x;
  const int r_lo = b * G_ROWS;
  const int r_hi = min(d.m, r_lo + G_ROWS);
  double* rows = lds;                       // [64][RP]
  const int group = S::GROUPS > 1 ? t / S::NUP : 0;
  const int pidx = S::GROUPS > 1 ? t % S::NUP : t;
  const bool worker = S::GROUPS > 1 ? (group < S::GROUPS) : true;

  double acc[S::TPT][4][4];
  int kbs[S::TPT], lbs[S::TPT];
#pragma unroll
  for (int u = 0; u < S::TPT; ++u) {
    const int p = pidx + u * kBlock;
    if (p < S::NUP) tile_coords(p, S::NB, kbs[u], lbs[u]); else { kbs[u] = -1; lbs[u] = -1; }
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y) acc[u][x][y] = 0.0;
  }

  for (int c0 = r_lo; c0 < r_hi; c0 += 64) {
    const int nr = min(64, r_hi - c0);
    for (int idx = t; idx < 64 * RP; idx += kBlock) {
      const int i = idx / RP, k = idx % RP;
      double v = 0.0;
      if (i < nr) {
        const int64_t row = c0 + i;
        if (MODE == 0) {
          float s = d.ppart[row * RP + k];
          for (int sp = 1; sp < d.sp; ++sp) s = s + d.ppart[((int64_t)sp * d.m + row) * RP + k];
          d.praw[row * RP + k] = s;
          v = (double)s;
        } else {
          const float* pr = d.praw + row * RP;
          for (int l = 0; l <= k; ++l) v = fma((double)pr[l], d.t1[l * RP + k], v);
        }
      }
      rows[i * RP + k] = v;
    }
    __syncthreads();
    if (worker) {
      for (int i = group; i < nr; i += S::GROUPS) {
        const double* row = rows + i * RP;
#pragma unroll
        for (int u = 0; u < S::TPT; ++u) {
          if (kbs[u] < 0) continue;
          double x[4], y[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) { x[q] = row[kbs[u] * 4 + q]; y[q] = row[lbs[u] * 4 + q]; }
#pragma unroll
          for (int p = 0; p < 4; ++p)
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[u][p][q] = fma(x[p], y[q], acc[u][p][q]);
        }
      }
    }
    __syncthreads();
  }

  // Combine row groups (fixed order) and store the full symmetric partial.
  double* gp = d.gpart + (int64_t)b * RP * RP;
  if (S::GROUPS == 1) {
#pragma unroll
    for (int u = 0; u < S::TPT; ++u) {
      if (kbs[u] < 0) continue;
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int k = kbs[u] * 4 + p, l = lbs[u] * 4 + q;
          gp[k * RP + l] = acc[u][p][q];
          gp[l * RP + k] = acc[u][p][q];
        }
    }
  } else {
    double* red = lds;  // [GROUPS][NUP][16]
    if (worker) {
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) red[((int64_t)group * S::NUP + pidx) * 16 + p * 4 + q] = acc[0][p][q];
    }
    __syncthreads();
    for (int idx = t; idx < S::NUP * 16; idx += kBlock) {
      const int p = idx / 16, e = idx % 16;
      double s = red[p * 16 + e];
      for (int g = 1; g < S::GROUPS; ++g) s += red[((int64_t)g * S::NUP + p) * 16 + e];
      int kb, lb;
      tile_coords(p, S::NB, kb, lb);
      const int k = kb * 4 + e / 4, l = lb * 4 + e % 4;
      gp[k * RP + l] = s;
      gp[l * RP + k] = s;
    }
  }
}

template <int RP>
constexpr int gram_lds_doubles() {
  using S = GramShape<RP>;
  constexpr int a = 64 * RP;
  constexpr int b = S::GROUPS > 1 ? S::GROUPS * S::NUP * 16 : 0;
  return a > b ? a : b;
}

template <int RP, int MODE>
__global__ __launch_bounds__(kBlock) void k_gram(OCC_KARGS) {
  __shared__ double lds[gram_lds_doubles<RP>()];
  if (MODE == 1) {
    // second CholeskyQR pass only when the first one asked for it
    const uint32_t need = (count == 1) ? single.info[0]
                                       : table[find_matrix(table, count, K_GRAM2, blockIdx.x)].info[0];
    if (!need) return;
  }
#define B_(d, b) gram_body<RP, MODE>(d, b, lds)
  OCC_DISPATCH(MODE == 0 ? K_PGRAM : K_GRAM2, B_)
#undef B_
}

// gsum[k][l] = sum_b gpart[b][k][l], fixed order.
template <int RP, int MODE>
__device__ __forceinline__ void gsum_body(const Desc& d, int b) {
  if (MODE == 1 && !d.info[0]) return;
  const int idx = b * kBlock + threadIdx.x;
  if (idx >= RP * RP) return;
  double s = d.gpart[idx];
  for (int g = 1; g < d.ng; ++g) s += d.gpart[(int64_t)g * RP * RP + idx];
  d.gsum[idx] = s;
}

template <int RP, int MODE>
__global__ __launch_bounds__(kBlock) void k_gsum(OCC_KARGS) {
#define B_(d, b) gsum_body<RP, MODE>(d, b)
  OCC_DISPATCH(K_GSUM, B_)
#undef B_
}

// ---------------------------------------------------------------------------
// Cholesky of the r x r Gram (fp64, in LDS, packed lower triangle), one block
// per matrix.  Pivot rule: a pivot <= 1e-12 * max diag(G) marks the column
// dependent (its column of P_hat becomes zero; later columns ignore it).
// Then X = L^-1 restricted to the independent rows, T = X^T (upper).
//   MODE 0: T1 = T; decide whether a second pass is needed; if not, Tm = T1.
//   MODE 1: Tm = T1 * T2 (only when the second pass ran).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int pk(int i, int k) { return i * (i + 1) / 2 + k; }

constexpr double kPivotTol = 1e-12;
constexpr double kSecondPassCond = 1e3;  // diag(L) ratio above which CholeskyQR2 runs

template <int RP, int MODE>
__device__ __forceinline__ void chol_body(const Desc& d, uint32_t* flags, double* L, double* X,
                                          int* def) {
  const int t = threadIdx.x;
  if (MODE == 1 && !d.info[0]) return;
  const int r = d.r;
  for (int idx = t; idx < RP * (RP + 1) / 2; idx += kBlock) {
    int i = 0;
    while ((i + 1) * (i + 2) / 2 <= idx) ++i;
    const int k = idx - i * (i + 1) / 2;
    L[idx] = d.gsum[i * RP + k];
  }
  __shared__ double s_maxdiag;
  __shared__ int s_nonfinite;
  __syncthreads();
  if (t == 0) {
    double mx = 0.0;
    int nf = 0;
    for (int j = 0; j < RP; ++j) {
      const double g = L[pk(j, j)];
      if (!isfinite(g)) nf = 1;
      if (g > mx) mx = g;
    }
    s_maxdiag = mx;
    s_nonfinite = nf;
    if (nf && flags) atomicOr(flags, FLAG_NONFINITE);
  }
  __syncthreads();
  const double thr = kPivotTol * s_maxdiag;
  for (int j = 0; j < RP; ++j) {
    const double piv = L[pk(j, j)];
    const bool dep = (j >= r) || (piv <= thr);
    __syncthreads();
    if (t == 0) {
      def[j] = dep ? 1 : 0;
      if (dep && j < r && flags) atomicOr(flags, FLAG_RANK_DEFICIENT);
      L[pk(j, j)] = dep ? 1.0 : sqrt(piv);
    }
    const double ljj = dep ? 1.0 : sqrt(piv);
    for (int i = j + 1 + t; i < RP; i += kBlock) L[pk(i, j)] = dep ? 0.0 : L[pk(i, j)] / ljj;
    __syncthreads();
    // trailing update of the lower triangle: L[i][l] -= L[i][j] L[l][j], j < l <= i
    const int nt = RP - j - 1;
    for (int idx = t; idx < nt * (nt + 1) / 2; idx += kBlock) {
      int ii = 0;
      while ((ii + 1) * (ii + 2) / 2 <= idx) ++ii;
      const int ll = idx - ii * (ii + 1) / 2;
      const int i = j + 1 + ii, l = j + 1 + ll;
      L[pk(i, l)] -= L[pk(i, j)] * L[pk(l, j)];
    }
    __syncthreads();
  }
  // X = L^-1 (lower), columns in parallel; dependent rows are zero.
  for (int c = t; c < RP; c += kBlock) {
    for (int i = c; i < RP; ++i) {
      double x = 0.0;
      if (!def[i]) {
        double s = (i == c) ? 1.0 : 0.0;
        for (int k = c; k < i; ++k) s -= L[pk(i, k)] * X[pk(k, c)];
        x = s / L[pk(i, i)];
      }
      X[pk(i, c)] = x;
    }
  }
  __syncthreads();
  if (MODE == 0) {
    // T1 = X^T; decide whether the first pass lost orthogonality
    for (int idx = t; idx < RP * RP; idx += kBlock) {
      const int l = idx / RP, k = idx % RP;       // T1[l][k] = X[k][l] for l <= k
      const double v = (l <= k) ? X[pk(k, l)] : 0.0;
      d.t1[idx] = v;
    }
    __shared__ uint32_t s_need;
    if (t == 0) {
      double dmax = 0.0, dmin = 1e308;
      for (int j = 0; j < r; ++j) {
        if (def[j]) continue;
        const double v = L[pk(j, j)];
        dmax = v > dmax ? v : dmax;
        dmin = v < dmin ? v : dmin;
      }
      const uint32_t need = (dmax > 0.0 && dmax > kSecondPassCond * dmin) ? 1u : 0u;
      s_need = need;
      d.info[0] = need;
    }
    __syncthreads();
    if (!s_need) {
      for (int idx = t; idx < RP * RP; idx += kBlock) {
        const int l = idx / RP, k = idx % RP;
        d.tm[idx] = (l <= k) ? X[pk(k, l)] : 0.0;
      }
    }
  } else {
    // Tm = T1 T2 with T2 = X^T: Tm[l][k] = sum_{l <= p <= k} T1[l][p] X[k][p]
    for (int idx = t; idx < RP * RP; idx += kBlock) {
      const int l = idx / RP, k = idx % RP;
      double s = 0.0;
      if (l <= k)
        for (int p = l; p <= k; ++p) s = fma(d.t1[l * RP + p], X[pk(k, p)], s);
      d.tm[idx] = s;
    }
  }
}

template <int RP, int MODE>
__global__ __launch_bounds__(kBlock) void k_chol(OCC_KARGS, uint32_t* flags) {
  __shared__ double L[RP * (RP + 1) / 2];
  __shared__ double X[RP * (RP + 1) / 2];
  __shared__ int def[RP];
  if (count == 1) chol_body<RP, MODE>(single, flags, L, X, def);
  else chol_body<RP, MODE>(table[blockIdx.x], flags, L, X, def);
}

// ---------------------------------------------------------------------------
// P_hat = P Tm (fp64 arithmetic, fp32 result) -> phat[m][rp] and caller's P.
// ---------------------------------------------------------------------------
template <int RP>
__device__ __forceinline__ void apply_body(const Desc& d, int b, double* tm) {
  for (int idx = threadIdx.x; idx < RP * RP; idx += kBlock) tm[idx] = d.tm[idx];
  __syncthreads();
  const int row0 = b * 64;
  for (int idx = threadIdx.x; idx < 64 * RP; idx += kBlock) {
    const int i = row0 + idx / RP, k = idx % RP;
    if (i >= d.m) continue;
    const float* pr = d.praw + (int64_t)i * RP;
    double s = 0.0;
    for (int l = 0; l <= k; ++l) s = fma((double)pr[l], tm[l * RP + k], s);
    const float v = (float)s;
    d.phat[(int64_t)i * RP + k] = v;
    if (k < d.r) d.P[(int64_t)i * d.r + k] = v;
  }
}

template <int RP>
constexpr int apply_lds_doubles() { return RP * RP; }

template <int RP>
__global__ __launch_bounds__(kBlock) void k_apply(OCC_KARGS) {
  __shared__ double tm[apply_lds_doubles<RP>()];
#define B_(d, b) apply_body<RP>(d, b, tm)
  OCC_DISPATCH(K_APPLY, B_)
#undef B_
}

// ---------------------------------------------------------------------------
// Right product, split over rows: qpart[s][c][k] = sum_{i in split s} A[i,c] P_hat[i,k].
// Each lane owns CPL consecutive columns; the four waves of a block take
// interleaved rows of the split; rows of P_hat come from SGPRs.
// ---------------------------------------------------------------------------
template <int DT, bool VEC, int RP>
__device__ __forceinline__ void pass_q_body(const Desc& d, int b, float* lds) {
  constexpr int CPL = cols_per_lane(RP);
  constexpr int RC = q_rank_chunk(RP);
  constexpr int NRC = RP / RC;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int col_tiles = (d.n + 64 * CPL - 1) / (64 * CPL);
  const int rc = b % NRC;
  const int rest = b / NRC;
  const int ct = rest % col_tiles, s = rest / col_tiles;
  const int c0 = ct * 64 * CPL + lane * CPL;
  const int r_lo = s * d.q_rows;
  const int r_hi = min(d.m, r_lo + d.q_rows);

  float acc[CPL][RC];
#pragma unroll
  for (int j = 0; j < CPL; ++j)
#pragma unroll
    for (int k = 0; k < RC; ++k) acc[j][k] = 0.f;

  for (int i = r_lo + wave; i < r_hi; i += 4) {
    float a[CPL];
    if (CPL == 4) {
      load_a4<DT, VEC>(d, i, c0, d.n, a);
    } else {
      a[0] = load_a1<DT>(d, i, c0);
    }
    const cfloat_p ph = as_const(d.phat) + (int64_t)i * RP + rc * RC;
#pragma unroll
    for (int k = 0; k < RC; ++k) {
      const float p = ph[k];
#pragma unroll
      for (int j = 0; j < CPL; ++j) acc[j][k] = fmaf(a[j], p, acc[j][k]);
    }
  }
  // fixed-order sum of the four waves, through LDS [4][64*CPL][RC+1]
  constexpr int PITCH = RC + 1;
#pragma unroll
  for (int j = 0; j < CPL; ++j)
#pragma unroll
    for (int k = 0; k < RC; ++k) lds[((wave * 64 + lane) * CPL + j) * PITCH + k] = acc[j][k];
  __syncthreads();
  for (int idx = threadIdx.x; idx < 64 * CPL * RC; idx += kBlock) {
    const int cl = idx / RC, k = idx % RC;
    const int col = ct * 64 * CPL + cl;
    if (col >= d.n) continue;
    float v = lds[(0 * 64 * CPL + cl) * PITCH + k];
    v = v + lds[(1 * 64 * CPL + cl) * PITCH + k];
    v = v + lds[(2 * 64 * CPL + cl) * PITCH + k];
    v = v + lds[(3 * 64 * CPL + cl) * PITCH + k];
    d.qpart[((int64_t)s * d.n + col) * RP + rc * RC + k] = v;
  }
}

template <int RP>
constexpr int pass_q_lds_floats() { return 4 * 64 * cols_per_lane(RP) * (q_rank_chunk(RP) + 1); }

template <int DT, bool VEC, int RP>
__global__ __launch_bounds__(kBlock) void k_pass_q(OCC_KARGS) {
  __shared__ float lds[pass_q_lds_floats<RP>()];
#define B_(d, b) pass_q_body<DT, VEC, RP>(d, b, lds)
  OCC_DISPATCH(K_PASS_Q, B_)
#undef B_
}

// Q[c][k] = sum_s qpart[s][c][k] (fixed order) -> caller's Q and qpad.
template <int RP>
__device__ __forceinline__ void qred_body(const Desc& d, int b) {
  const int64_t idx = (int64_t)b * kBlock + threadIdx.x;
  if (idx >= (int64_t)d.n * RP) return;
  const int c = (int)(idx / RP), k = (int)(idx % RP);
  float v = d.qpart[idx];
  for (int s = 1; s < d.sq; ++s) v = v + d.qpart[(int64_t)s * d.n * RP + idx];
  d.qpad[idx] = v;
  if (k < d.r) d.Q[(int64_t)c * d.r + k] = v;
}

template <int RP>
__global__ __launch_bounds__(kBlock) void k_qred(OCC_KARGS) {
#define B_(d, b) qred_body<RP>(d, b)
  OCC_DISPATCH(K_QRED, B_)
#undef B_
}

// ---------------------------------------------------------------------------
// Reconstruction and residual in one pass:
//   M_hat[i,c] = sum_k P_hat[i,k] Q[c,k]  (k ascending, fmaf from 0)
//   err[i,c]   = (M[i,c] + err_prev[i,c]) - M_hat[i,c]
// Each lane owns CPL columns and keeps their Q rows in VGPRs; rows of P_hat
// come from SGPRs.  SRC selects where the factors come from:
//   0: the workspace's padded phat/qpad (fused step)
//   1: the caller's P (m x r) and Q (n x r) (stand-alone decompression)
// ---------------------------------------------------------------------------
template <int DT, bool VEC, int RP, int SRC, bool WRITE_MHAT, bool WRITE_ERR>
__device__ __forceinline__ void mhat_body(const Desc& d, int b) {
  constexpr int CPL = cols_per_lane(RP);
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int col_tiles = (d.n + 64 * CPL - 1) / (64 * CPL);
  const int ct = b % col_tiles, rb = b / col_tiles;
  const int c0 = ct * 64 * CPL + lane * CPL;
  const int r_lo = rb * MH_ROWS;
  const int r_hi = min(d.m, r_lo + MH_ROWS);

  float q[CPL][RP];
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const int c = c0 + j;
#pragma unroll
    for (int k = 0; k < RP; ++k) {
      float v = 0.f;
      if (c < d.n) {
        if (SRC == 0) v = d.qpad[(int64_t)c * RP + k];
        else if (k < d.r) v = d.Q[(int64_t)c * d.r + k];
      }
      q[j][k] = v;
    }
  }

  for (int i = r_lo + wave; i < r_hi; i += 4) {
    float ph[RP];
    if (SRC == 0) {
      const cfloat_p p = as_const(d.phat) + (int64_t)i * RP;
#pragma unroll
      for (int k = 0; k < RP; ++k) ph[k] = p[k];
    } else {
      const cfloat_p p = as_const(d.P) + (int64_t)i * d.r;
#pragma unroll
      for (int k = 0; k < RP; ++k) ph[k] = (k < d.r) ? p[k] : 0.f;
    }
    float mh[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < RP; ++k) s = fmaf(ph[k], q[j][k], s);
      mh[j] = s;
    }
    if (WRITE_MHAT) {
      const int64_t ho = (int64_t)i * d.ldh + c0;
      if (CPL == 4 && VEC && c0 + 4 <= d.n) {
        *(float4*)(d.Mhat + ho) = make_float4(mh[0], mh[1 % CPL], mh[2 % CPL], mh[3 % CPL]);
      } else {
#pragma unroll
        for (int j = 0; j < CPL; ++j) if (c0 + j < d.n) d.Mhat[ho + j] = mh[j];
      }
    }
    if (WRITE_ERR) {
      float a[CPL];
      if (CPL == 4) load_a4<DT, VEC>(d, i, c0, d.n, a);
      else a[0] = load_a1<DT>(d, i, c0);
      float e[CPL];
#pragma unroll
      for (int j = 0; j < CPL; ++j) e[j] = a[j] - mh[j];
      const int64_t eo = (int64_t)i * d.lde_out + c0;
      if (CPL == 4 && VEC && c0 + 4 <= d.n) {
        *(float4*)(d.err_out + eo) = make_float4(e[0], e[1 % CPL], e[2 % CPL], e[3 % CPL]);
      } else {
#pragma unroll
        for (int j = 0; j < CPL; ++j) if (c0 + j < d.n) d.err_out[eo + j] = e[j];
      }
    }
  }
}

template <int DT, bool VEC, int RP, int SRC, bool WRITE_MHAT, bool WRITE_ERR>
__global__ __launch_bounds__(kBlock) void k_mhat(OCC_KARGS) {
#define B_(d, b) mhat_body<DT, VEC, RP, SRC, WRITE_MHAT, WRITE_ERR>(d, b)
  OCC_DISPATCH(K_MHAT, B_)
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

// Copy descriptor chunks passed by value into the workspace table.
constexpr int kTableChunk = 4;
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

}  // namespace occ
